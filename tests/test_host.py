"""Host half of the library (libdf11.so, no GPU needed) against the oracle:
code books, byte-identical streams and metadata, decode tables read off the
oracle's tree walk, a CPU model of the decoder's table walk, validation of
corrupted streams, and the exported C ABI."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2504_11651_amd import codec, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def stream_cases():
    return {
        "empty": lambda: np.zeros(0, np.uint16),
        "one": lambda: np.array([0xBF80], np.uint16),
        "two": lambda: np.array([0x3F80, 0x0001], np.uint16),
        "single_symbol": lambda: (np.arange(3000, dtype=np.uint16) & 0x807F) | (100 << 7),
        "gauss_small": lambda: synth.gaussian(9_999, 0.02, 1),
        "gauss": lambda: synth.gaussian(300_001, 0.02, 2),
        "gauss_wide": lambda: synth.gaussian(100_000, 5.0, 3),
        "special": lambda: synth.special_values(40_000),
        "patterns": synth.all_bf16_patterns,
        "fib24": lambda: synth.fibonacci_exponents(24),
        "heavy": lambda: synth.heavy_tailed_block(200_000, 1),
    }


LAYOUTS = [(8, 64, 12), (8, 256, 12), (8, 1024, 10), (16, 128, 8), (4, 64, 11)]


@pytest.mark.parametrize("case", sorted(stream_cases()))
@pytest.mark.parametrize("lay", LAYOUTS, ids=lambda l: "n%d_T%d_K%d" % l)
def test_stream_identical_to_oracle(case, lay):
    n_bytes, T, K = lay
    w = stream_cases()[case]()
    hs = codec.encode(w, layout=codec.make_layout(n_bytes, T, K))
    st = oracle.compress(w, 32, n_bytes, T)
    assert np.array_equal(hs.codebook.lengths, st["lengths"])
    assert np.array_equal(hs.codebook.codes, st["codes"])
    assert hs.sizes.total_bits == st["total_bits"]
    assert hs.sizes.num_chunks == st["num_chunks"] and hs.sizes.num_blocks == st["num_blocks"]
    assert np.array_equal(hs.exp, st["exp"])
    assert np.array_equal(hs.sm[:w.size], st["sm"])
    assert hs.sm.size == ((w.size + 15) // 16) * 16 + 16 and not hs.sm[w.size:].any()
    assert np.array_equal(hs.gaps, st["gaps_packed"])
    assert np.array_equal(hs.block_pos, st["block_pos"])
    bp = st["block_pos"].astype(np.int64)
    assert hs.sizes.max_elems_per_block == (int(np.diff(bp).max()) if bp.size > 1 else 0)
    assert codec.validate(hs) == 0
    # the oracle decodes the library's stream back to the input
    out = oracle.decode_serial(hs.exp, hs.sizes.total_bits, hs.sm, w.size, hs.codebook.lengths)
    assert np.array_equal(out, w)


@pytest.mark.parametrize("cap", [9, 12, 16, 20, 32])
def test_capped_codebook_matches_oracle(cap):
    fib = [1, 1]
    while len(fib) < 40:
        fib.append(fib[-1] + fib[-2])
    counts = np.zeros(256, np.uint64)
    counts[80:120] = fib
    cb = codec.codebook_from_counts(counts, cap)
    ol = oracle.code_lengths(counts, cap)
    assert cb.lengths.max() == cap
    # independent package-merge implementations, same tie rule: same lengths
    assert np.array_equal(cb.lengths, ol)
    assert np.array_equal(cb.codes, oracle.canonical_codes(ol))


def test_codebook_random_histograms_match_oracle():
    rng = np.random.default_rng(0)
    for trial in range(200):
        m = int(rng.integers(1, 257))
        counts = np.zeros(256, np.uint64)
        hi = [3, 100, 10**9][trial % 3]
        counts[rng.choice(256, size=m, replace=False)] = rng.integers(1, hi + 1, size=m)
        for cap in (32, 12):
            if cap < 32 and (1 << cap) < m:
                continue
            cb = codec.codebook_from_counts(counts, cap)
            assert np.array_equal(cb.lengths, oracle.code_lengths(counts, cap)), (trial, cap)


def test_cap_errors():
    counts = np.ones(256, np.uint64)
    with pytest.raises(codec.DF11Error) as e:
        codec.codebook_from_counts(counts, 7)
    assert e.value.rc == -2
    with pytest.raises(codec.DF11Error):
        codec.codebook_from_counts(counts, 33)


# ---------------------------------------------------------------- decode tables
def parse_tables(blob: np.ndarray):
    hdr = blob[:16].view(np.uint32)
    K = int(hdr[1])
    ent = blob[16:16 + (8 << K)].view(np.uint32).reshape(-1, 2)
    esc = blob[16 + (8 << K):]
    lj = esc[:132].view(np.uint32)
    off = esc[132:264].view(np.uint32)
    sorted_syms = esc[264:520]
    return int(hdr[0]), K, int(hdr[2]), ent, lj, off, sorted_syms


@pytest.mark.parametrize("K", [8, 10, 12])
@pytest.mark.parametrize("case", ["gauss", "fib24", "special"])
def test_table_entries_match_oracle_tree_walk(K, case):
    w = stream_cases()[case]()
    cb = codec.build_codebook(w)
    magic, k, maxlen, ent, lj, off, srt = parse_tables(codec.build_tables(cb, K))
    assert magic == 0x544C4644 and k == K and maxlen == cb.max_code_len
    lengths = cb.lengths
    rng = np.random.default_rng(K)
    xs = range(1 << K) if K <= 10 else rng.choice(1 << K, size=1500, replace=False)
    for x in xs:
        x = int(x)
        # window bit j is stream bit j: the K-bit pattern read first-bit-first
        bits = "".join(str((x >> j) & 1) for j in range(K))
        syms, pos, mask = [], 0, 0
        while len(syms) < 4 and pos < K:
            r = oracle.decode_prefix(int(bits[pos:], 2), K - pos, lengths)
            if r is None:
                break
            syms.append(r[0])
            mask |= 1 << pos
            pos += r[1]
        lo, meta = int(ent[x, 0]), int(ent[x, 1])
        if not syms:
            assert meta == 0 and lo == 0
            continue
        assert meta & 0xFF == pos and (meta >> 8) & 0xFF == len(syms) and meta >> 16 == mask
        assert [(lo >> (8 * i)) & 0xFF for i in range(len(syms))] == syms
        assert lo >> (8 * len(syms)) == 0


def test_long_code_escape_tables():
    # every code longer than K must be decodable from lj_last/offset/sorted
    fib = [1, 1]
    while len(fib) < 40:
        fib.append(fib[-1] + fib[-2])
    counts = np.zeros(256, np.uint64)
    counts[80:120] = fib
    cb = codec.codebook_from_counts(counts, 32)
    K = 10
    _, _, maxlen, ent, lj, off, srt = parse_tables(codec.build_tables(cb, K))
    for s in range(80, 120):
        L = int(cb.lengths[s])
        if L <= K:
            continue
        v = (int(cb.codes[s]) << (32 - L)) | ((1 << (32 - L)) - 1 if L < 32 else 0)
        ll = K + 1
        while ll < maxlen and v > int(lj[ll]):
            ll += 1
        assert ll == L
        idx = ((v >> (32 - ll)) + int(off[ll])) & 0xFFFFFFFF & 255
        assert int(srt[idx]) == s


def kernel_model_decode(hs: codec.HostStream) -> np.ndarray:
    """Pure-Python model of the GPU decoder's per-chunk table walk (phase 1
    count with the start-mask correction, phase 2 writes including the codes
    a lookup decodes past the chunk end).  Test-only; n = 8 layouts."""
    z = hs.sizes
    _, K, maxlen, ent, lj, off, srt = parse_tables(hs.tables)
    T = hs.layout.threads_per_block
    exp = hs.exp
    gbits = "".join(format(int(b), "08b") for b in hs.gaps)
    C, B = int(z.num_chunks), int(z.num_blocks)
    out_exp = {}
    for b in range(B):
        counts, starts, ends = [], [], []
        for t in range(T):
            c = b * T + t
            g0 = int(gbits[5 * c:5 * c + 5], 2)
            g1 = int(gbits[5 * c + 5:5 * c + 10], 2)
            if c >= C:
                starts.append(0), ends.append(0), counts.append(0)
                continue
            start = g0
            end = 64 + g1 if c + 1 < C else int(z.total_bits) - 64 * c
            chunk = int.from_bytes(exp[8 * c:8 * c + 12].tobytes(), "big")  # 96 bits
            cnt, p, last_p, last_meta = 0, start, 0, 0
            while p < end:
                win = (chunk >> (96 - p - 32)) & 0xFFFFFFFF  # MSB-first 32 bits at p
                x = int("".join(str((win >> (31 - j)) & 1) for j in range(K))[::-1], 2)
                lo, meta = int(ent[x, 0]), int(ent[x, 1])
                if meta == 0:
                    L = K + 1
                    while L < maxlen and win > int(lj[L]):
                        L += 1
                    lo = int(srt[((win >> (32 - L)) + int(off[L])) & 0xFFFFFFFF & 255])
                    meta = L | (1 << 8) | (1 << 16)
                last_p, last_meta = p, meta
                p += meta & 0xFF
                cnt += (meta >> 8) & 0xFF
            cnt -= bin((last_meta >> 16) >> min(end - last_p, 31)).count("1")
            counts.append(cnt), starts.append(start), ends.append(end)
        pos = int(hs.block_pos[b])
        assert sum(counts) == int(hs.block_pos[b + 1]) - pos
        for t in range(T):
            c = b * T + t
            if c >= C:
                continue
            chunk = int.from_bytes(exp[8 * c:8 * c + 12].tobytes(), "big")
            p, o = starts[t], pos + sum(counts[:t])
            while p < ends[t]:
                win = (chunk >> (96 - p - 32)) & 0xFFFFFFFF
                x = int("".join(str((win >> (31 - j)) & 1) for j in range(K))[::-1], 2)
                lo, meta = int(ent[x, 0]), int(ent[x, 1])
                if meta == 0:
                    L = K + 1
                    while L < maxlen and win > int(lj[L]):
                        L += 1
                    lo = int(srt[((win >> (32 - L)) + int(off[L])) & 0xFFFFFFFF & 255])
                    meta = L | (1 << 8) | (1 << 16)
                for k in range((meta >> 8) & 0xFF):
                    e = (lo >> (8 * k)) & 0xFF
                    prev = out_exp.get(o + k)
                    assert prev is None or prev == e  # overlapping writes agree
                    out_exp[o + k] = e
                o += (meta >> 8) & 0xFF
                p += meta & 0xFF
    n = int(z.n_elems)
    e = np.array([out_exp[i] for i in range(n)], np.uint16)
    sm = hs.sm[:n].astype(np.uint16)
    return ((sm & 0x80) << 8) | (e << 7) | (sm & 0x7F)


@pytest.mark.parametrize("case,lay", [("gauss_small", (8, 64, 12)), ("special", (8, 64, 9)),
                                      ("fib24", (8, 64, 8)), ("two", (8, 64, 12)),
                                      ("single_symbol", (8, 128, 10))])
def test_kernel_table_walk_model(case, lay):
    w = stream_cases()[case]()
    if w.size > 12_000:
        w = w[:12_000]
    hs = codec.encode(w, layout=codec.make_layout(*lay))
    assert np.array_equal(kernel_model_decode(hs), w)


# ---------------------------------------------------------------- validation
def _fresh():
    w = synth.gaussian(60_000, 0.02, 9)
    return codec.encode(w, layout=codec.make_layout(8, 64, 12))


def test_validate_rejects_corruption():
    hs = _fresh()
    assert codec.validate(hs) == 0
    hs.block_pos[3] = hs.block_pos[2] - 1
    assert codec.validate(hs) == -4
    hs = _fresh()
    hs.block_pos[-1] += 1
    assert codec.validate(hs) == -4
    hs = _fresh()
    hs.sizes.max_elems_per_block += 1
    assert codec.validate(hs) == -4
    hs = _fresh()
    hs.sizes.exp_bytes -= 1
    assert codec.validate(hs) == -4
    hs = _fresh()
    hs.tables[0] ^= 1
    assert codec.validate(hs) == -4
    hs = _fresh()
    ent = hs.tables[16:].view(np.uint32)
    ent[1] = (ent[1] & ~np.uint32(0xFF)) | np.uint32(0)  # bits consumed 0
    assert codec.validate(hs) == -4
    hs = _fresh()  # a gap past the code-length cap
    hs.gaps[0] |= 0xF8
    assert codec.validate(hs) == -4


def _table_words(hs):
    """(entries as uint32 pairs, lj_last[33], offset[33], sorted[256]) views
    into the stream's table blob (layout of df11_tables.h)."""
    K = int(hs.layout.lut_bits)
    body = hs.tables[16:]
    ent = body[:8 << K].view(np.uint32)
    esc = body[8 << K:(8 << K) + 264].view(np.uint32)
    return ent, esc[:33], esc[33:66], body[(8 << K) + 264:(8 << K) + 264 + 256]


@pytest.mark.parametrize("what", ["entry_exponent", "entry_meta", "lj_last", "lj_last_top",
                                  "offset", "sorted_swap", "sorted_dup", "sorted_tail",
                                  "padding"])
def test_validate_rejects_corrupt_tables(what):
    """The table blob must be the canonical tables of a complete prefix code
    (Kraft sum 1): any single corrupted entry, length boundary, offset or
    symbol is refused."""
    hs = _fresh()
    assert codec.validate(hs) == 0
    ent, lj, off, srt = _table_words(hs)
    L = int(hs.sizes.max_code_len)
    if what == "entry_exponent":
        ent[2 * 7] ^= 1 << 8           # second exponent of entry 7
    elif what == "entry_meta":
        ent[2 * 100 + 1] ^= 1 << 16    # code-start mask of entry 100
    elif what == "lj_last":
        lj[3] -= 1 << 29               # length-3 codes end one code earlier
    elif what == "lj_last_top":
        lj[L] -= 1 << (32 - L)         # the longest length loses a code: Kraft < 1
    elif what == "offset":
        off[4] += 1
    elif what == "sorted_swap":
        srt[0], srt[1] = srt[1], srt[0]
    elif what == "sorted_dup":
        srt[1] = srt[0]
    elif what == "sorted_tail":
        srt[255] = 1                   # past the used symbols: must stay zero
    elif what == "padding":
        hs.tables[-1] = 0x5A
    assert codec.validate(hs) == -4


def test_validate_accepts_valid_books():
    """Complete codes of every shape validate: one symbol (a 1-bit code),
    two symbols, all 65,536 BF16 patterns (256 symbols), a 32-bit code."""
    cases = [np.full(1000, 0x3F80, np.uint16), np.array([0x3F80, 0x4000] * 50, np.uint16),
             synth.all_bf16_patterns()]
    counts = np.array([1 << (31 - i) if i < 31 else 1 for i in range(32)] + [1], np.uint64)
    geo = np.repeat((np.arange(33, dtype=np.uint16) + 60) << 7, counts.astype(np.int64) // (1 << 12) + 1)
    cases.append(geo)
    for w in cases:
        for K in (8, 11, 12):
            hs = codec.encode(w, layout=codec.make_layout(8, 64, K))
            assert codec.validate(hs) == 0


def test_encode_rejects_mismatched_codebook():
    w = synth.gaussian(10_000, 0.02, 1)
    cb = codec.build_codebook(synth.gaussian(10_000, 0.02, 2))
    with pytest.raises(codec.DF11Error):
        codec.encode(w, cb=cb)


def test_encode_buffer_too_small():
    w = synth.gaussian(1000, 0.02, 1)
    cb = codec.build_codebook(w)
    lay = codec.make_layout()
    z = codec.encoded_sizes(cb, lay)
    buf = np.zeros(z.exp_bytes - 1, np.uint8)
    rc = codec.lib().df11_encode(w.ctypes.data, w.size, ctypes.byref(cb), ctypes.byref(lay),
                                 buf.ctypes.data, buf.size, np.zeros(1000, np.uint8).ctypes.data,
                                 1000, np.zeros(z.gap_bytes, np.uint8).ctypes.data, z.gap_bytes,
                                 np.zeros(z.num_blocks + 1, np.uint32).ctypes.data,
                                 4 * (z.num_blocks + 1), ctypes.byref(codec.Sizes()))
    assert rc == -3


def test_bad_layouts_rejected():
    cb = codec.build_codebook(synth.gaussian(1000, 0.02, 1))
    for lay in [(8, 100, 12), (8, 2048, 12), (8, 256, 13), (8, 256, 7), (2, 256, 12)]:
        with pytest.raises(codec.DF11Error):
            codec.encoded_sizes(cb, codec.make_layout(*lay))


# ---------------------------------------------------------------- the C ABI
def test_library_exports_every_declared_symbol():
    header = open(os.path.join(ROOT, "include", "df11.h")).read()
    declared = set(re.findall(r"^(?:int|const char \*)\s*(df11_\w+)\(", header, re.M))
    assert declared == set(codec.EXPORTS)
    L = codec.lib()
    for name in declared:
        assert hasattr(L, name)
    assert codec.strerror(-4) == "corrupt stream"


def test_decode_rejects_bad_descriptors_without_launching():
    hs = _fresh()
    st = hs.struct()
    st.layout.bytes_per_thread = 16
    assert codec.lib().df11_decode_block(ctypes.byref(st), None, None) == -6
    st = hs.struct()
    st.layout.threads_per_block = 192
    assert codec.lib().df11_decode_block(ctypes.byref(st), None, None) == -6
    assert codec.lib().df11_decode_block(None, None, None) == -1
    st = hs.struct()
    st.sizes.n_elems = 0  # nothing to do: no launch, ok
    assert codec.lib().df11_decode_block(ctypes.byref(st), None, None) == 0


def test_size_limits_of_32_bit_positions():
    # BlockOutputPos entries are 32-bit: a stream of more than 2^32 - 1
    # weights is refused when sized, and a descriptor claiming one is
    # refused by the decoder before anything is launched
    counts = np.zeros(256, np.uint64)
    counts[120], counts[121] = 2 ** 31, 2 ** 31  # 2^32 weights
    cb = codec.codebook_from_counts(counts)
    with pytest.raises(codec.DF11Error) as e:
        codec.encoded_sizes(cb, codec.make_layout())
    assert e.value.rc == -1
    counts[121] -= 1  # 2^32 - 1 weights: allowed
    z = codec.encoded_sizes(codec.codebook_from_counts(counts), codec.make_layout())
    assert z.n_elems == 2 ** 32 - 1
    st = _fresh().struct()
    st.sizes.n_elems = 2 ** 32
    assert codec.lib().df11_decode_block(ctypes.byref(st), None, None) == -1
