"""DFloat11 CPU oracle: ctypes access to ``df11_oracle.c``.

TEST INFRASTRUCTURE ONLY.  The test-suite, the smoke check and the
benchmark's CPU-baseline leg are the only callers.  The product library never
imports this package, and this package never imports the product library.

Each wrapper mirrors one C function of ``df11_oracle.c``; the C file cites the
passage of the paper each step follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "df11_oracle.c")
_LIB = os.path.join(_HERE, "libdf11_oracle.so")

_u8p = ctypes.POINTER(ctypes.c_uint8)
_u16p = ctypes.POINTER(ctypes.c_uint16)
_u32p = ctypes.POINTER(ctypes.c_uint32)
_u64p = ctypes.POINTER(ctypes.c_uint64)
_uintp = ctypes.POINTER(ctypes.c_uint)

_lib = None


def build() -> str:
    """Compile the oracle with gcc (plain C99, -O2, no vector tricks needed)."""
    cmd = ["gcc", "-std=c99", "-O2", "-fPIC", "-shared", "-Wall", "-Wextra", _SRC, "-o", _LIB]
    subprocess.run(cmd, check=True)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    sig = {
        "dfo_histogram": [_u16p, ctypes.c_uint64, _u64p],
        "dfo_huffman_lengths": [_u64p, _uintp],
        "dfo_package_merge": [_u64p, ctypes.c_uint, _uintp],
        "dfo_code_lengths": [_u64p, ctypes.c_uint, _u8p],
        "dfo_canonical_codes": [_u8p, _u32p],
        "dfo_layout": [ctypes.c_uint64, ctypes.c_uint, ctypes.c_uint, _u64p, _u64p, _u64p, _u64p],
        "dfo_encode": [_u16p, ctypes.c_uint64, _u8p, _u32p, _u8p, ctypes.c_uint64, _u8p, _u64p],
        "dfo_metadata": [_u16p, ctypes.c_uint64, _u8p, ctypes.c_uint, ctypes.c_uint, _u8p,
                         ctypes.c_uint64, _u32p, ctypes.c_uint64],
        "dfo_pack_gaps": [_u8p, ctypes.c_uint64, _u8p, ctypes.c_uint64],
        "dfo_decode_prefix": [ctypes.c_uint64, ctypes.c_uint, _u8p, ctypes.POINTER(ctypes.c_int),
                              _uintp],
        "dfo_decode_serial": [_u8p, ctypes.c_uint64, _u8p, ctypes.c_uint64, _u8p, _u16p],
        "dfo_decode_blocks": [_u8p, ctypes.c_uint64, _u8p, ctypes.c_uint64, _u8p, ctypes.c_uint,
                              ctypes.c_uint, _u8p, _u32p, ctypes.c_uint64, ctypes.c_uint64, _u16p],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    _lib = lib
    return lib


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError(f"{what} failed with code {rc}")


def _ptr(a: np.ndarray, typ):
    return a.ctypes.data_as(typ)


def _as_u16(w) -> np.ndarray:
    a = np.ascontiguousarray(w)
    if a.dtype != np.uint16:
        a = a.view(np.uint16) if a.dtype.itemsize == 2 else a.astype(np.uint16)
    return a.reshape(-1)


def histogram(w) -> np.ndarray:
    w = _as_u16(w)
    c = np.zeros(256, np.uint64)
    _check(_load().dfo_histogram(_ptr(w, _u16p), w.size, _ptr(c, _u64p)), "histogram")
    return c


def huffman_lengths(counts):
    """Unconstrained Huffman lengths (may exceed 32).  Returns (lengths, max)."""
    c = np.ascontiguousarray(counts, dtype=np.uint64)
    l = np.zeros(256, np.uint32)
    depth = _load().dfo_huffman_lengths(_ptr(c, _u64p), _ptr(l, _uintp))
    return l, int(depth)


def package_merge(counts, max_len: int) -> np.ndarray:
    c = np.ascontiguousarray(counts, dtype=np.uint64)
    l = np.zeros(256, np.uint32)
    _check(_load().dfo_package_merge(_ptr(c, _u64p), max_len, _ptr(l, _uintp)), "package_merge")
    return l


def code_lengths(counts, max_len: int = 32) -> np.ndarray:
    c = np.ascontiguousarray(counts, dtype=np.uint64)
    l = np.zeros(256, np.uint8)
    _check(_load().dfo_code_lengths(_ptr(c, _u64p), max_len, _ptr(l, _u8p)), "code_lengths")
    return l


def canonical_codes(lengths) -> np.ndarray:
    l = np.ascontiguousarray(lengths, dtype=np.uint8)
    codes = np.zeros(256, np.uint32)
    _check(_load().dfo_canonical_codes(_ptr(l, _u8p), _ptr(codes, _u32p)), "canonical_codes")
    return codes


def layout(total_bits: int, n_bytes: int = 8, threads: int = 256) -> dict:
    out = [ctypes.c_uint64() for _ in range(4)]
    _check(_load().dfo_layout(total_bits, n_bytes, threads, *[ctypes.byref(o) for o in out]),
           "layout")
    keys = ("num_chunks", "num_blocks", "exp_bytes", "gap_bytes")
    return {k: int(o.value) for k, o in zip(keys, out)}


def encode(w, lengths, codes, exp_cap: int):
    w = _as_u16(w)
    l = np.ascontiguousarray(lengths, dtype=np.uint8)
    c = np.ascontiguousarray(codes, dtype=np.uint32)
    exp = np.zeros(max(exp_cap, 1), np.uint8)
    sm = np.zeros(max(w.size, 1), np.uint8)
    tb = ctypes.c_uint64()
    _check(_load().dfo_encode(_ptr(w, _u16p), w.size, _ptr(l, _u8p), _ptr(c, _u32p),
                              _ptr(exp, _u8p), exp_cap, _ptr(sm, _u8p), ctypes.byref(tb)),
           "encode")
    return exp[:exp_cap], sm[:w.size], int(tb.value)


def metadata(w, lengths, n_bytes: int, threads: int, total_bits: int):
    """Unpacked Gaps (one byte per slot, B*T+1 slots) and BlockOutputPos (B+1)."""
    w = _as_u16(w)
    l = np.ascontiguousarray(lengths, dtype=np.uint8)
    lay = layout(total_bits, n_bytes, threads)
    slots = lay["num_blocks"] * threads + 1
    gaps = np.zeros(slots, np.uint8)
    bp = np.zeros(lay["num_blocks"] + 1, np.uint32)
    _check(_load().dfo_metadata(_ptr(w, _u16p), w.size, _ptr(l, _u8p), n_bytes, threads,
                                _ptr(gaps, _u8p), slots, _ptr(bp, _u32p), bp.size), "metadata")
    return gaps, bp


def pack_gaps(gaps, packed_bytes: int) -> np.ndarray:
    g = np.ascontiguousarray(gaps, dtype=np.uint8)
    out = np.zeros(max(packed_bytes, 1), np.uint8)
    _check(_load().dfo_pack_gaps(_ptr(g, _u8p), g.size, _ptr(out, _u8p), packed_bytes),
           "pack_gaps")
    return out[:packed_bytes]


def decode_prefix(pattern: int, nbits: int, lengths):
    """First symbol of a bit pattern (its first bit is bit nbits-1).  (sym, len)."""
    l = np.ascontiguousarray(lengths, dtype=np.uint8)
    s = ctypes.c_int()
    n = ctypes.c_uint()
    rc = _load().dfo_decode_prefix(pattern, nbits, _ptr(l, _u8p), ctypes.byref(s), ctypes.byref(n))
    if rc != 0:
        return None
    return int(s.value), int(n.value)


def decode_serial(exp, total_bits: int, sm, n: int, lengths) -> np.ndarray:
    e = np.ascontiguousarray(exp, dtype=np.uint8)
    m = np.ascontiguousarray(sm, dtype=np.uint8)
    l = np.ascontiguousarray(lengths, dtype=np.uint8)
    out = np.zeros(max(n, 1), np.uint16)
    _check(_load().dfo_decode_serial(_ptr(e, _u8p), total_bits, _ptr(m, _u8p), n, _ptr(l, _u8p),
                                     _ptr(out, _u16p)), "decode_serial")
    return out[:n]


def decode_blocks(exp, total_bits: int, sm, n: int, lengths, n_bytes: int, threads: int, gaps,
                  block_pos, first_block: int, num_blocks: int, out: np.ndarray | None = None):
    e = np.ascontiguousarray(exp, dtype=np.uint8)
    m = np.ascontiguousarray(sm, dtype=np.uint8)
    l = np.ascontiguousarray(lengths, dtype=np.uint8)
    g = np.ascontiguousarray(gaps, dtype=np.uint8)
    bp = np.ascontiguousarray(block_pos, dtype=np.uint32)
    if out is None:
        out = np.zeros(max(n, 1), np.uint16)
    _check(_load().dfo_decode_blocks(_ptr(e, _u8p), total_bits, _ptr(m, _u8p), n, _ptr(l, _u8p),
                                     n_bytes, threads, _ptr(g, _u8p), _ptr(bp, _u32p),
                                     first_block, num_blocks, _ptr(out, _u16p)), "decode_blocks")
    return out[:n]


def compress(w, max_len: int = 32, n_bytes: int = 8, threads: int = 256) -> dict:
    """Whole format, step by step: histogram, lengths, codes, encode, metadata."""
    w = _as_u16(w)
    counts = histogram(w)
    lengths = code_lengths(counts, max_len)
    codes = canonical_codes(lengths)
    total_bits = int(sum(int(counts[s]) * int(lengths[s]) for s in range(256)))
    lay = layout(total_bits, n_bytes, threads)
    exp, sm, tb = encode(w, lengths, codes, lay["exp_bytes"])
    assert tb == total_bits
    gaps, bp = metadata(w, lengths, n_bytes, threads, total_bits)
    packed = pack_gaps(gaps, lay["gap_bytes"])
    return dict(counts=counts, lengths=lengths, codes=codes, total_bits=total_bits, exp=exp,
                sm=sm, gaps=gaps, gaps_packed=packed, block_pos=bp, n=w.size, n_bytes=n_bytes,
                threads=threads, **lay)


# ------------------------------------------------------------ matrix products
def bf16_to_f64(bits) -> np.ndarray:
    """BF16 bit patterns -> float64: a BF16 value is the float32 whose upper 16
    bits are the pattern and whose lower 16 bits are zero."""
    b = np.ascontiguousarray(bits)
    if b.dtype != np.uint16:
        b = b.view(np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def linear(x_bits, w_bits) -> np.ndarray:
    """Y = X W^T in float64 for BF16 X (tokens x k) and W (rows x k): the
    product the decompressed weights feed (Sec. 2.3.3), with every BF16 product
    exact and the sums rounded only at float64 precision."""
    x = bf16_to_f64(x_bits)
    w = bf16_to_f64(w_bits)
    return x @ w.T
