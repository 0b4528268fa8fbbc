"""Thin ctypes binding of libdf11.so (the C ABI declared in include/df11.h).

Argument marshalling only: every step of encoding runs in the library's C++
host code and every step of decoding in its HIP kernels.  PyTorch supplies
device memory and the current HIP stream; nothing here computes.  When the
library is missing, import fails loudly -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdf11.so")

DF11_OK = 0
ERRORS = {
    -1: "DF11_E_INVALID_ARG", -2: "DF11_E_CAP_INFEASIBLE", -3: "DF11_E_BUFFER_TOO_SMALL",
    -4: "DF11_E_CORRUPT", -5: "DF11_E_HIP", -6: "DF11_E_UNSUPPORTED",
}

# every function include/df11.h declares
EXPORTS = (
    "df11_build_codebook", "df11_codebook_from_counts", "df11_default_layout",
    "df11_encoded_sizes", "df11_encode",
    "df11_build_tables", "df11_validate", "df11_decode_block", "df11_decode_launch_shape",
    "df11_gemm_workspace_bytes", "df11_block_gemm", "df11_block_forward",
    "df11_block_forward_noalloc", "df11_gemv_workspace_bytes", "df11_block_gemv", "df11_strerror",
    "df11_build_hlut_tables", "df11_decode_block_hlut",
)

MAX_MATRICES = 8  # DF11_MAX_MATRICES
MAX_TOKENS = 64   # DF11_MAX_TOKENS
STATIC_SCRATCH_BYTES = 32 << 20  # DF11_STATIC_SCRATCH_BYTES


class Codebook(ctypes.Structure):
    _fields_ = [("max_code_len", ctypes.c_uint32), ("num_symbols", ctypes.c_uint32),
                ("count", ctypes.c_uint64 * 256), ("len", ctypes.c_uint8 * 256),
                ("code", ctypes.c_uint32 * 256)]

    @property
    def lengths(self) -> np.ndarray:
        return np.frombuffer(bytes(self.len), np.uint8).copy()

    @property
    def codes(self) -> np.ndarray:
        return np.array(self.code[:], np.uint32)

    @property
    def counts(self) -> np.ndarray:
        return np.array(self.count[:], np.uint64)


class Layout(ctypes.Structure):
    _fields_ = [("bytes_per_thread", ctypes.c_uint32), ("threads_per_block", ctypes.c_uint32),
                ("lut_bits", ctypes.c_uint32)]


class Sizes(ctypes.Structure):
    _fields_ = [("n_elems", ctypes.c_uint64), ("total_bits", ctypes.c_uint64),
                ("num_chunks", ctypes.c_uint64), ("num_blocks", ctypes.c_uint64),
                ("exp_bytes", ctypes.c_uint64), ("sm_bytes", ctypes.c_uint64),
                ("gap_bytes", ctypes.c_uint64), ("block_pos_bytes", ctypes.c_uint64),
                ("table_bytes", ctypes.c_uint64), ("max_elems_per_block", ctypes.c_uint32),
                ("max_code_len", ctypes.c_uint32)]

    def as_dict(self) -> dict:
        return {k: int(getattr(self, k)) for k, _ in self._fields_}


class Stream(ctypes.Structure):
    _fields_ = [("exp", ctypes.c_void_p), ("sm", ctypes.c_void_p), ("gaps", ctypes.c_void_p),
                ("block_pos", ctypes.c_void_p), ("tables", ctypes.c_void_p), ("sizes", Sizes),
                ("layout", Layout)]


class Matrix(ctypes.Structure):
    _fields_ = [("offset", ctypes.c_uint64), ("rows", ctypes.c_uint32), ("cols", ctypes.c_uint32)]


# bytes per thread, threads per block, table index bits, where no weight count
# is at hand: the layout of large streams (128-chunk blocks, decoded one per
# wavefront, two chunks per lane).  encode() takes default_layout(n).
DEFAULT_LAYOUT = (8, 128, 11)
# The fused decode-and-multiply path decodes 64-chunk blocks only.
FUSED_LAYOUT = (8, 64, 11)

_lib = None


class DF11Error(RuntimeError):
    def __init__(self, rc: int, what: str):
        super().__init__(f"{what}: {ERRORS.get(rc, rc)} ({rc})")
        self.rc = rc


def lib():
    """The loaded libdf11.so; raises when it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(there is no fallback decoder)")
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    vp = ctypes.c_void_p
    u64 = ctypes.c_uint64
    sig = {
        "df11_build_codebook": [vp, u64, ctypes.c_uint32, P(Codebook)],
        "df11_codebook_from_counts": [vp, ctypes.c_uint32, P(Codebook)],
        "df11_default_layout": [u64, P(Layout)],
        "df11_encoded_sizes": [P(Codebook), P(Layout), P(Sizes)],
        "df11_encode": [vp, u64, P(Codebook), P(Layout), vp, u64, vp, u64, vp, u64, vp, u64,
                        P(Sizes)],
        "df11_build_tables": [P(Codebook), ctypes.c_uint32, vp, u64],
        "df11_validate": [P(Stream)],
        "df11_decode_block": [P(Stream), vp, vp],
        "df11_decode_launch_shape": [P(Stream), P(ctypes.c_uint32), P(ctypes.c_uint32),
                                     P(ctypes.c_uint32)],
        "df11_gemm_workspace_bytes": [P(Matrix), ctypes.c_uint32, ctypes.c_uint32, P(u64)],
        "df11_block_gemm": [vp, u64, P(Matrix), ctypes.c_uint32, P(vp), ctypes.c_uint32, P(vp),
                            vp, u64, vp],
        "df11_block_forward": [P(Stream), vp, P(Matrix), ctypes.c_uint32, P(vp), ctypes.c_uint32,
                               P(vp), vp, u64, vp],
        "df11_block_forward_noalloc": [P(Stream), vp, P(Matrix), ctypes.c_uint32, P(vp),
                                       ctypes.c_uint32, P(vp), vp],
        "df11_gemv_workspace_bytes": [P(Stream), P(Matrix), ctypes.c_uint32, P(u64)],
        "df11_block_gemv": [P(Stream), P(Matrix), ctypes.c_uint32, P(vp), P(vp), vp, u64, vp],
        "df11_build_hlut_tables": [P(Codebook), ctypes.c_uint32, vp, u64, P(ctypes.c_uint32)],
        "df11_decode_block_hlut": [P(Stream), vp, ctypes.c_uint32, vp, vp],
    }
    for name, args in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    L.df11_strerror.argtypes = [ctypes.c_int]
    L.df11_strerror.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(rc: int, what: str):
    if rc != DF11_OK:
        raise DF11Error(rc, what)


def _u16(w) -> np.ndarray:
    a = np.ascontiguousarray(w)
    if a.dtype != np.uint16:
        a = a.view(np.uint16)
    return a.reshape(-1)


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data) if a.size else ctypes.c_void_p(0)


def make_layout(bytes_per_thread=None, threads_per_block=None, lut_bits=None) -> Layout:
    n, T, K = DEFAULT_LAYOUT
    return Layout(bytes_per_thread or n, threads_per_block or T, lut_bits or K)


def default_layout(n: int) -> Layout:
    """The library's layout for a stream of n weights (df11_default_layout)."""
    lay = Layout()
    _check(lib().df11_default_layout(int(n), ctypes.byref(lay)), "df11_default_layout")
    return lay


# ---------------------------------------------------------------- host side
def build_codebook(w, max_code_len: int = 32) -> Codebook:
    w = _u16(w)
    cb = Codebook()
    _check(lib().df11_build_codebook(_ptr(w), w.size, max_code_len, ctypes.byref(cb)),
           "df11_build_codebook")
    return cb


def codebook_from_counts(counts, max_code_len: int = 32) -> Codebook:
    c = np.ascontiguousarray(counts, dtype=np.uint64)
    cb = Codebook()
    _check(lib().df11_codebook_from_counts(_ptr(c), max_code_len, ctypes.byref(cb)),
           "df11_codebook_from_counts")
    return cb


def encoded_sizes(cb: Codebook, layout: Layout) -> Sizes:
    s = Sizes()
    _check(lib().df11_encoded_sizes(ctypes.byref(cb), ctypes.byref(layout), ctypes.byref(s)),
           "df11_encoded_sizes")
    return s


def build_tables(cb: Codebook, lut_bits: int) -> np.ndarray:
    lay = Layout(8, 256, lut_bits)
    nbytes = encoded_sizes(cb, lay).table_bytes
    t = np.zeros(nbytes, np.uint8)
    _check(lib().df11_build_tables(ctypes.byref(cb), lut_bits, _ptr(t), t.size),
           "df11_build_tables")
    return t


@dataclass
class HostStream:
    """One encoded stream in host memory (numpy arrays)."""
    exp: np.ndarray
    sm: np.ndarray  # n_elems bytes + zero padding (sizes.sm_bytes)
    gaps: np.ndarray
    block_pos: np.ndarray
    tables: np.ndarray
    sizes: Sizes
    layout: Layout
    codebook: Codebook

    def struct(self) -> Stream:
        return Stream(_ptr(self.exp).value, _ptr(self.sm).value, _ptr(self.gaps).value,
                      _ptr(self.block_pos).value, _ptr(self.tables).value, self.sizes,
                      self.layout)

    @property
    def compressed_bytes(self) -> int:
        """Bytes the decoder reads: exact stream + sign/mantissa + gaps + positions + tables."""
        z = self.sizes
        return int((z.total_bits + 7) // 8 + z.n_elems + z.gap_bytes + z.block_pos_bytes +
                   z.table_bytes)


def encode(w, cb: Codebook | None = None, layout: Layout | None = None,
           max_code_len: int = 32) -> HostStream:
    """Code book (unless given), stream, metadata and tables for BF16 bit patterns."""
    w = _u16(w)
    layout = layout or default_layout(w.size)
    if cb is None:
        cb = build_codebook(w, max_code_len)
    z = encoded_sizes(cb, layout)
    exp = np.empty(z.exp_bytes, np.uint8)
    sm = np.empty(z.sm_bytes, np.uint8)
    gaps = np.empty(z.gap_bytes, np.uint8)
    bp = np.empty(z.num_blocks + 1, np.uint32)
    out = Sizes()
    _check(lib().df11_encode(_ptr(w), w.size, ctypes.byref(cb), ctypes.byref(layout), _ptr(exp),
                             exp.size, _ptr(sm), sm.size, _ptr(gaps), gaps.size, _ptr(bp),
                             bp.nbytes, ctypes.byref(out)), "df11_encode")
    tables = build_tables(cb, layout.lut_bits)
    return HostStream(exp, sm, gaps, bp, tables, out, layout, cb)


def validate(hs: HostStream) -> int:
    """0 when consistent, else the negative status (no exception)."""
    st = hs.struct()
    return int(lib().df11_validate(ctypes.byref(st)))


def strerror(rc: int) -> str:
    return lib().df11_strerror(rc).decode()


# ---------------------------------------------------------------- device side
class DeviceStream:
    """A stream resident in device memory (torch uint8/int32 tensors)."""

    def __init__(self, hs: HostStream, device="cuda"):
        import torch
        dev = torch.device(device)
        if dev.type != "cuda":
            raise ValueError(f"a device stream lives in GPU memory, not on {dev}")
        self.exp = torch.from_numpy(hs.exp).to(dev)
        self.sm = torch.from_numpy(hs.sm).to(dev)
        self.gaps = torch.from_numpy(hs.gaps).to(dev)
        self.block_pos = torch.from_numpy(hs.block_pos.view(np.int32)).to(dev)
        self.tables = torch.from_numpy(hs.tables).to(dev)
        self.sizes = Sizes.from_buffer_copy(hs.sizes)
        self.layout = Layout.from_buffer_copy(hs.layout)
        self.device = self.exp.device  # with its index
        self._st = Stream(self.exp.data_ptr(), self.sm.data_ptr(), self.gaps.data_ptr(),
                          self.block_pos.data_ptr(), self.tables.data_ptr(), self.sizes,
                          self.layout)

    @property
    def n_elems(self) -> int:
        return int(self.sizes.n_elems)

    def struct(self) -> Stream:
        return self._st

    def nbytes(self) -> int:
        return sum(t.numel() * t.element_size()
                   for t in (self.exp, self.sm, self.gaps, self.block_pos, self.tables))


def to_device(hs: HostStream, device="cuda") -> DeviceStream:
    return DeviceStream(hs, device)


def launch_shape(ds: DeviceStream):
    g, b, l = ctypes.c_uint32(), ctypes.c_uint32(), ctypes.c_uint32()
    _check(lib().df11_decode_launch_shape(ctypes.byref(ds.struct()), ctypes.byref(g),
                                          ctypes.byref(b), ctypes.byref(l)),
           "df11_decode_launch_shape")
    return int(g.value), int(b.value), int(l.value)


def _on_device(t, device, what: str):
    """The library dereferences these pointers on the GPU: a host tensor or
    one on another GPU would fault there, so it is refused here."""
    if t.device != device:
        raise ValueError(f"{what} must be on {device}, not {t.device}")


def decode_block(ds: DeviceStream, out=None, stream=None):
    """Decode into ``out`` (a bfloat16 device tensor of n_elems, 16-byte aligned;
    allocated when None) on ``stream`` (default: torch's current stream)."""
    import torch
    n = ds.n_elems
    if out is None:
        out = torch.empty(n, dtype=torch.bfloat16, device=ds.device)
    if out.numel() < n or out.element_size() != 2 or not out.is_contiguous():
        raise ValueError("out must be a contiguous 2-byte tensor with n_elems elements")
    _on_device(out, ds.device, "out")
    if stream is None:
        stream = torch.cuda.current_stream(ds.device)
    handle = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    _check(lib().df11_decode_block(ctypes.byref(ds.struct()), ctypes.c_void_p(out.data_ptr()),
                                   ctypes.c_void_p(handle)), "df11_decode_block")
    return out


# ------------------------------------------------------- decode-then-GEMM driver
def _mats(mats) -> "ctypes.Array":
    arr = (Matrix * len(mats))()
    for i, (off, rows, cols) in enumerate(mats):
        arr[i] = Matrix(int(off), int(rows), int(cols))
    return arr


def gemm_workspace_bytes(mats, tokens: int) -> int:
    """Workspace bytes block_gemm / block_forward need (mats: (offset, rows, cols))."""
    m = _mats(mats)
    out = ctypes.c_uint64()
    _check(lib().df11_gemm_workspace_bytes(m, len(mats), int(tokens), ctypes.byref(out)),
           "df11_gemm_workspace_bytes")
    return int(out.value)


def _gemm_marshal(mats, xs, ys, workspace, device):
    if not (len(mats) == len(xs) == len(ys)) or not mats:
        raise ValueError("one activation and one output tensor per matrix")
    tokens = int(xs[0].shape[0])
    for (off, rows, cols), x, y in zip(mats, xs, ys):
        if tuple(x.shape) != (tokens, cols) or x.element_size() != 2 or not x.is_contiguous():
            raise ValueError("x[m] must be a contiguous bf16 tensor of shape (tokens, cols)")
        if tuple(y.shape) != (tokens, rows) or y.element_size() != 4 or not y.is_contiguous():
            raise ValueError("y[m] must be a contiguous fp32 tensor of shape (tokens, rows)")
        _on_device(x, device, "x[m]")
        _on_device(y, device, "y[m]")
    if workspace is not None:
        _on_device(workspace, device, "workspace")
    xp = (ctypes.c_void_p * len(xs))(*[x.data_ptr() for x in xs])
    yp = (ctypes.c_void_p * len(ys))(*[y.data_ptr() for y in ys])
    ws_ptr = workspace.data_ptr() if workspace is not None else 0
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    return _mats(mats), xp, yp, tokens, ws_ptr, ws_bytes


def _handle(stream, device):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def block_gemm(weights, mats, xs, ys, workspace=None, stream=None):
    """ys[m] = xs[m] @ W_m^T for the matrices (offset, rows, cols) of the BF16
    block ``weights`` (device tensor), fp32 results written into ys."""
    if weights.element_size() != 2 or not weights.is_contiguous():
        raise ValueError("weights must be a contiguous bf16 tensor")
    if weights.device.type != "cuda":
        raise ValueError(f"weights must be on a GPU, not {weights.device}")
    m, xp, yp, tokens, ws_ptr, ws_bytes = _gemm_marshal(mats, xs, ys, workspace, weights.device)
    _check(lib().df11_block_gemm(ctypes.c_void_p(weights.data_ptr()), weights.numel(), m,
                                 len(mats), xp, tokens, yp, ctypes.c_void_p(ws_ptr), ws_bytes,
                                 ctypes.c_void_p(_handle(stream, weights.device))),
           "df11_block_gemm")
    return ys


def block_forward(ds: DeviceStream, weights_out, mats, xs, ys, workspace=None, stream=None):
    """Decode ``ds`` into ``weights_out`` (bf16 device tensor of n_elems), then
    block_gemm on it, all on one stream."""
    if (weights_out.numel() < ds.n_elems or weights_out.element_size() != 2 or
            not weights_out.is_contiguous()):
        raise ValueError("weights_out must be a contiguous 2-byte tensor with n_elems elements")
    _on_device(weights_out, ds.device, "weights_out")
    m, xp, yp, tokens, ws_ptr, ws_bytes = _gemm_marshal(mats, xs, ys, workspace, ds.device)
    _check(lib().df11_block_forward(ctypes.byref(ds.struct()),
                                    ctypes.c_void_p(weights_out.data_ptr()), m, len(mats), xp,
                                    tokens, yp, ctypes.c_void_p(ws_ptr), ws_bytes,
                                    ctypes.c_void_p(_handle(stream, ds.device))),
           "df11_block_forward")
    return ys


def block_forward_noalloc(ds: DeviceStream, weights_out, mats, xs, ys, stream=None):
    """block_forward with the partial sums in the library's fixed per-GPU
    array (no workspace, no device allocation by the library).  Calls that
    overlap on one GPU race on that array."""
    if (weights_out.numel() < ds.n_elems or weights_out.element_size() != 2 or
            not weights_out.is_contiguous()):
        raise ValueError("weights_out must be a contiguous 2-byte tensor with n_elems elements")
    _on_device(weights_out, ds.device, "weights_out")
    m, xp, yp, tokens, _, _ = _gemm_marshal(mats, xs, ys, None, ds.device)
    _check(lib().df11_block_forward_noalloc(ctypes.byref(ds.struct()),
                                            ctypes.c_void_p(weights_out.data_ptr()), m,
                                            len(mats), xp, tokens, yp,
                                            ctypes.c_void_p(_handle(stream, ds.device))),
           "df11_block_forward_noalloc")
    return ys


# ------------------------------------------------ fused decode-and-multiply
def gemv_workspace_bytes(ds: DeviceStream, mats) -> int:
    """Workspace bytes block_gemv needs for this stream and these matrices."""
    out = ctypes.c_uint64()
    _check(lib().df11_gemv_workspace_bytes(ctypes.byref(ds.struct()), _mats(mats), len(mats),
                                           ctypes.byref(out)),
           "df11_gemv_workspace_bytes")
    return int(out.value)


def block_gemv(ds: DeviceStream, mats, xs, ys, workspace=None, stream=None):
    """ys[m][r] = sum_k xs[m][k] * W_m[r][k] for one token, with the weights of
    ``ds`` decoded on chip (never written out).  xs[m]: bf16 (cols,) or
    (1, cols); ys[m]: fp32 (rows,) or (1, rows).  ``ds`` must be encoded in
    FUSED_LAYOUT (64 chunks per block)."""
    import torch
    if not (len(mats) == len(xs) == len(ys)) or not mats:
        raise ValueError("one activation and one output tensor per matrix")
    for (off, rows, cols), x, y in zip(mats, xs, ys):
        if x.numel() != cols or x.element_size() != 2 or not x.is_contiguous():
            raise ValueError("x[m] must be a contiguous bf16 tensor of cols elements")
        if y.numel() != rows or y.element_size() != 4 or not y.is_contiguous():
            raise ValueError("y[m] must be a contiguous fp32 tensor of rows elements")
        _on_device(x, ds.device, "x[m]")
        _on_device(y, ds.device, "y[m]")
    if workspace is None:
        workspace = torch.empty(max(gemv_workspace_bytes(ds, mats) // 4, 4), dtype=torch.float32,
                                device=ds.device)
        # the kernels run on `stream`: the caching allocator must not hand this
        # memory out again before that stream has finished with it
        s = torch.cuda.current_stream(ds.device) if stream is None else stream
        if not hasattr(s, "cuda_stream"):
            s = torch.cuda.ExternalStream(int(s), device=ds.device)
        workspace.record_stream(s)
    _on_device(workspace, ds.device, "workspace")
    xp = (ctypes.c_void_p * len(xs))(*[x.data_ptr() for x in xs])
    yp = (ctypes.c_void_p * len(ys))(*[y.data_ptr() for y in ys])
    _check(lib().df11_block_gemv(ctypes.byref(ds.struct()), _mats(mats), len(mats), xp, yp,
                                 ctypes.c_void_p(workspace.data_ptr()),
                                 workspace.numel() * workspace.element_size(),
                                 ctypes.c_void_p(_handle(stream, ds.device))),
           "df11_block_gemv")
    return ys


# ------------------------------------ the paper's decoder (ablation)
HLUT_MAX_BYTES = 18 * 256  # DF11_HLUT_MAX_BYTES


def build_hlut_tables(cb: Codebook, level_bits: int = 8):
    """(tables, k): the paper's hierarchical lookup tables LUT_1..LUT_k
    (2**level_bits bytes each) followed by CodeLengths[256]."""
    k = ctypes.c_uint32()
    buf = np.zeros(HLUT_MAX_BYTES if level_bits == 8 else (17 << level_bits) + 256, np.uint8)
    rc = lib().df11_build_hlut_tables(ctypes.byref(cb), level_bits, _ptr(buf), buf.size,
                                      ctypes.byref(k))
    _check(rc, "df11_build_hlut_tables")
    return buf[:(int(k.value) << level_bits) + 256].copy(), int(k.value)


class DeviceHlut:
    """The paper's tables for one stream, in device memory."""

    def __init__(self, hs: HostStream, device="cuda"):
        import torch
        tabs, self.k = build_hlut_tables(hs.codebook, 8)
        self.tables = torch.from_numpy(tabs).to(torch.device(device))


def decode_block_hlut(ds: DeviceStream, hl: DeviceHlut, out=None, stream=None):
    """Decode ``ds`` with the paper's kernel and tables ``hl`` into ``out``."""
    import torch
    n = ds.n_elems
    if out is None:
        out = torch.empty(n, dtype=torch.bfloat16, device=ds.device)
    if out.numel() < n or out.element_size() != 2 or not out.is_contiguous():
        raise ValueError("out must be a contiguous 2-byte tensor with n_elems elements")
    _on_device(out, ds.device, "out")
    _on_device(hl.tables, ds.device, "tables")
    _check(lib().df11_decode_block_hlut(ctypes.byref(ds.struct()),
                                        ctypes.c_void_p(hl.tables.data_ptr()), hl.k,
                                        ctypes.c_void_p(out.data_ptr()),
                                        ctypes.c_void_p(_handle(stream, ds.device))),
           "df11_decode_block_hlut")
    return out
