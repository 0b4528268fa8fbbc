"""Pins for the CPU oracle: each test checks it against something other than
itself -- the paper's printed example, closed forms, textbook bounds, exact
optimisation by brute force or by an independent dynamic program, and direct
pure-Python restatements of the format's definitions on tiny inputs."""
import functools
import json
import math
import os

import numpy as np
import pytest

import oracle
from paper_2504_11651_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- helpers
def entropy_bits(counts) -> float:
    c = np.asarray(counts, dtype=np.float64)
    p = c[c > 0] / c.sum()
    return float(-(p * np.log2(p)).sum())


def cost(counts, lengths) -> int:
    return int(sum(int(c) * int(l) for c, l in zip(counts, lengths)))


def kraft_scaled(lengths) -> int:
    """sum 2^(32-l) over used symbols, exact integers (== 2^32 for a full tree)."""
    return sum(1 << (32 - int(l)) for l in lengths if l)


def optimal_cost_dp(counts, max_len):
    """Exact minimum of sum c_i*l_i over prefix codes with l_i <= max_len.

    Independent of Huffman and package-merge: some optimal code gives the
    more frequent symbol the shorter (or equal) length, so sort counts in
    descending order and decide, depth by depth, how many of the next symbols
    become leaves; the free nodes at the next depth are twice the nodes that
    were not used as leaves."""
    c = sorted((int(x) for x in counts if x), reverse=True)
    m = len(c)
    if m == 0:
        return 0
    if m == 1:
        return c[0]  # one symbol: code length 1 (stated reading)
    suffix = [0] * (m + 1)
    for i in range(m - 1, -1, -1):
        suffix[i] = suffix[i + 1] + c[i]

    @functools.lru_cache(maxsize=None)
    def f(d, i, a):
        if i == m:
            return 0
        if d > max_len or a == 0:
            return math.inf
        best = math.inf
        for k in range(0, min(a, m - i) + 1):
            here = d * (suffix[i] - suffix[i + k])
            rest_nodes = min(2 * (a - k), m - i - k)
            if i + k < m and rest_nodes == 0:
                continue
            best = min(best, here + f(d + 1, i + k, rest_nodes))
        return best

    return f(1, 0, 2)


def brute_force_cost(counts, max_len):
    """Minimum over every length vector in [1, min(max_len, m-1)]^m with
    Kraft sum <= 1 (vectorised enumeration)."""
    used = [int(x) for x in counts if x]
    m = len(used)
    if m == 1:
        return used[0]
    top = min(max_len, m - 1)
    best = None
    rng1 = np.arange(1, top + 1, dtype=np.int64)
    for first in range(1, top + 1):  # chunk over the first coordinate
        rest = np.stack(np.meshgrid(*([rng1] * (m - 1)), indexing="ij"), -1).reshape(-1, m - 1)
        grids = np.concatenate([np.full((rest.shape[0], 1), first, np.int64), rest], 1)
        kraft = (np.int64(1) << (np.int64(top) - grids)).sum(1)
        ok = kraft <= (1 << top)
        if ok.any():
            c = int((grids[ok] @ np.array(used, np.int64)).min())
            best = c if best is None else min(best, c)
    return best


# ---------------------------------------------------------------- paper example
def test_paper_worked_example_codes_and_flat_lut():
    g = json.load(open(os.path.join(GOLDEN, "paper_lut_example.json")))
    names = g["symbols"]
    sym = {nm: 120 + i for i, nm in enumerate(names)}  # increasing exponent values
    counts = np.zeros(256, np.uint64)
    for nm, c in zip(names, (8, 2, 2, 2, 1, 1)):
        counts[sym[nm]] = c
    lengths = oracle.code_lengths(counts, 32)
    for nm, l in g["code_lengths"].items():
        assert lengths[sym[nm]] == l
    codes = oracle.canonical_codes(lengths)
    stated = dict(g["codes_stated"], **g["codes_from_two_level_tables"])
    for nm, bits in stated.items():
        assert format(int(codes[sym[nm]]), f"0{len(bits)}b") == bits
    # flat 4-bit LUT read off the oracle's tree walk
    inv = {v: k for k, v in sym.items()}
    for idx, nm in g["flat_lut_entries_stated"].items():
        s, _ = oracle.decode_prefix(int(idx), g["flat_lut_L"], lengths)
        assert inv[s] == nm
    # two-level 2-bit tables: prefix + 2 bits
    for prefix, table in (("", "LUT0"), ("10", "LUT1"), ("11", "LUT2")):
        for two, target in g["two_level_tables"][table].items():
            if target.startswith("->"):
                continue
            pat = prefix + two
            s, l = oracle.decode_prefix(int(pat, 2), len(pat), lengths)
            assert inv[s] == target and l <= len(pat)
    # dyadic: the mean code length equals the entropy (2.125 bits)
    assert cost(counts, lengths) / counts.sum() == pytest.approx(entropy_bits(counts), abs=0)
    assert entropy_bits(counts) == pytest.approx(2.125)


def test_bitstream_is_msb_first():
    # A=0, B=100 (worked example) -> stream "0100..." -> first byte 0x40
    counts = np.zeros(256, np.uint64)
    for s, c in zip(range(120, 126), (8, 2, 2, 2, 1, 1)):
        counts[s] = c
    lengths = oracle.code_lengths(counts)
    codes = oracle.canonical_codes(lengths)
    w = np.array([120 << 7, (121 << 7) | 0x8000 | 0x25], np.uint16)  # A, then -B with mantissa
    exp, sm, tb = oracle.encode(w, lengths, codes, 16)
    assert tb == 4
    assert exp[0] == 0x40 and not exp[1:].any()
    assert list(sm) == [0x00, 0xA5]  # sign to bit 7, mantissa bits 6..0 (Algorithm 1)


# ---------------------------------------------------------------- closed forms
@pytest.mark.parametrize("K", [2, 5, 17, 32])
def test_geometric_counts_give_unary_lengths(K):
    # counts 2^(K-1), ..., 2, 1, 1 -> lengths 1, 2, ..., K, K
    counts = np.zeros(256, np.uint64)
    for i in range(K):
        counts[i] = 1 << (K - 1 - i)
    counts[K] = 1
    lengths = oracle.code_lengths(counts, 32)
    assert list(lengths[:K + 1]) == list(range(1, K + 1)) + [K]
    assert kraft_scaled(lengths) == 1 << 32


@pytest.mark.parametrize("seed", range(6))
def test_dyadic_lengths_are_minus_log2_p(seed):
    rng = np.random.default_rng(seed)
    # random full binary tree -> leaf depths; counts 2^(D - depth) are dyadic
    depths = [0]
    while len(depths) < 2 + seed * 5:
        i = int(rng.integers(len(depths)))
        d = depths.pop(i)
        depths += [d + 1, d + 1]
    D = max(depths)
    counts = np.zeros(256, np.uint64)
    syms = rng.choice(256, size=len(depths), replace=False)
    for s, d in zip(syms, depths):
        counts[s] = 1 << (D - d)
    lengths = oracle.code_lengths(counts, 32)
    for s, d in zip(syms, depths):
        assert lengths[s] == d
    assert cost(counts, lengths) / counts.sum() == pytest.approx(entropy_bits(counts), abs=1e-12)


def test_single_and_empty_alphabets():
    counts = np.zeros(256, np.uint64)
    assert not oracle.code_lengths(counts).any()
    counts[77] = 1000
    lengths = oracle.code_lengths(counts)
    assert lengths[77] == 1 and lengths.sum() == 1
    assert oracle.canonical_codes(lengths)[77] == 0


# ---------------------------------------------------------------- optimality
@pytest.mark.parametrize("m", [2, 3, 4, 5, 6, 7, 8])
def test_huffman_is_optimal_brute_force(m):
    rng = np.random.default_rng(100 + m)
    trials = {7: 6, 8: 2}.get(m, 25)
    for trial in range(trials):
        hi = 4 if trial % 2 else 1000  # small ranges force ties
        c = rng.integers(1, hi + 1, size=m)
        counts = np.zeros(256, np.uint64)
        syms = rng.choice(256, size=m, replace=False)
        counts[syms] = c
        lengths = oracle.code_lengths(counts, 32)
        assert cost(counts, lengths) == brute_force_cost(counts, 32)
        assert kraft_scaled(lengths) == 1 << 32


@pytest.mark.parametrize("m,cap", [(5, 3), (6, 3), (7, 3), (8, 3), (8, 4), (7, 4)])
def test_capped_code_is_optimal_brute_force(m, cap):
    rng = np.random.default_rng(200 + 10 * m + cap)
    for trial in range(4):
        # steep counts so plain Huffman is deeper than the cap
        c = (rng.integers(1, 3, size=m) * (2.0 ** (2 * np.arange(m)))).astype(np.uint64)
        counts = np.zeros(256, np.uint64)
        counts[rng.choice(256, size=m, replace=False)] = c
        lengths = oracle.code_lengths(counts, cap)
        assert lengths.max() <= cap
        assert cost(counts, lengths) == brute_force_cost(counts, cap)
        assert cost(counts, lengths) == optimal_cost_dp(counts, cap)


@pytest.mark.parametrize("m", [12, 40, 96])
def test_huffman_cost_matches_exact_dp(m):
    rng = np.random.default_rng(m)
    counts = np.zeros(256, np.uint64)
    counts[rng.choice(256, size=m, replace=False)] = rng.integers(1, 10**6, size=m)
    lengths = oracle.code_lengths(counts, 32)
    assert lengths.max() <= 32
    # counts below 2^20 keep any optimal tree far shallower than 32 levels
    assert cost(counts, lengths) == optimal_cost_dp(counts, 32)


def test_fibonacci_counts_cap_binds_and_stays_optimal():
    fib = [1, 1]
    while len(fib) < 40:
        fib.append(fib[-1] + fib[-2])
    counts = np.zeros(256, np.uint64)
    counts[80:120] = fib
    free, depth = oracle.huffman_lengths(counts)
    assert depth == 39  # unconstrained tree is 39 deep
    lengths = oracle.code_lengths(counts, 32)
    assert lengths.max() == 32
    assert kraft_scaled(lengths) == 1 << 32
    assert cost(counts, lengths) == optimal_cost_dp(counts, 32)
    assert cost(counts, lengths) >= cost(counts, free)
    # same exact optimum under other caps
    for cap in (6, 10, 20, 31):
        l2 = oracle.code_lengths(counts, cap)
        assert l2.max() <= cap and kraft_scaled(l2) == 1 << 32
        assert cost(counts, l2) == optimal_cost_dp(counts, cap)


def test_cap_infeasible_is_an_error():
    counts = np.ones(256, np.uint64)
    with pytest.raises(oracle.OracleError):
        oracle.code_lengths(counts, 7)  # 2^7 < 256 symbols
    assert oracle.code_lengths(counts, 8).max() == 8


# ---------------------------------------------------------------- entropy bound
@pytest.mark.parametrize("kind", ["gauss", "gauss_wide", "special", "patterns"])
def test_entropy_bound(kind):
    w = {"gauss": lambda: synth.gaussian(200_000, 0.02, 3),
         "gauss_wide": lambda: synth.gaussian(200_000, 3.0, 4),
         "special": lambda: synth.special_values(50_000),
         "patterns": synth.all_bf16_patterns}[kind]()
    counts = oracle.histogram(w)
    lengths = oracle.code_lengths(counts, 32)
    H = entropy_bits(counts)
    Lbar = cost(counts, lengths) / counts.sum()
    assert H - 1e-12 <= Lbar < H + 1


@pytest.mark.parametrize("config", ["matrix_4096", "llama3_8b_block", "heavy_tailed_block",
                                    "llama31_70b_block"])
def test_kraft_and_entropy_bound_on_workload_histograms(config):
    """Pins P2 and P3 on the histograms of the four decode workloads (Sec. 2.1,
    Huffman optimality): the code is a complete prefix code (Kraft sum 1,
    exact in integers) and its mean length is within one bit of the
    exponent entropy."""
    w = {"matrix_4096": synth.matrix_4096,
         "llama3_8b_block": lambda: synth.llama3_8b_block()[0],
         "heavy_tailed_block": synth.heavy_tailed_block,
         "llama31_70b_block": lambda: synth.llama31_70b_block()[0]}[config]()
    counts = oracle.histogram(w)
    assert int(counts.sum()) == w.size
    del w
    lengths = oracle.code_lengths(counts, 32)
    assert kraft_scaled(lengths) == 1 << 32
    assert lengths.max() <= 32 and all((lengths > 0) == (counts > 0))
    H = entropy_bits(counts)
    Lbar = cost(counts, lengths) / counts.sum()
    assert H - 1e-12 <= Lbar < H + 1


def test_histogram_definition():
    w = synth.special_values(3000)
    ref = np.zeros(256, np.uint64)
    for x in w.tolist():
        ref[(x >> 7) & 0xFF] += 1
    assert np.array_equal(oracle.histogram(w), ref)


# ---------------------------------------------------------------- round trip
ROUND_TRIP_CASES = {
    "empty": lambda: np.zeros(0, np.uint16),
    "one": lambda: np.array([0x3F80], np.uint16),
    "two": lambda: np.array([0x3F80, 0xBC00], np.uint16),
    "single_symbol": lambda: (np.arange(5000, dtype=np.uint16) & 0x807F) | (121 << 7),
    "gauss": lambda: synth.gaussian(100_003, 0.02, 5),
    "special": lambda: synth.special_values(20_000),
    "patterns": synth.all_bf16_patterns,
    "fib22": lambda: synth.fibonacci_exponents(22),
}


@pytest.mark.parametrize("case", sorted(ROUND_TRIP_CASES))
def test_round_trip_serial(case):
    w = ROUND_TRIP_CASES[case]()
    st = oracle.compress(w, 32, 8, 256)
    out = oracle.decode_serial(st["exp"], st["total_bits"], st["sm"], w.size, st["lengths"])
    assert np.array_equal(out, w)


def test_round_trip_with_binding_cap():
    w = synth.fibonacci_exponents(22)  # unconstrained depth 21
    st = oracle.compress(w, 12, 8, 64)
    assert st["lengths"].max() == 12
    out = oracle.decode_serial(st["exp"], st["total_bits"], st["sm"], w.size, st["lengths"])
    assert np.array_equal(out, w)
    out2 = oracle.decode_blocks(st["exp"], st["total_bits"], st["sm"], w.size, st["lengths"], 8,
                                64, st["gaps"], st["block_pos"], 0, st["num_blocks"])
    assert np.array_equal(out2, w)


# ---------------------------------------------------------------- metadata
def python_metadata(w, lengths, n_bytes, T):
    """The format's definitions, restated with pure-Python loops."""
    starts, pos = [], 0
    for x in w.tolist():
        starts.append(pos)
        pos += int(lengths[(x >> 7) & 0xFF])
    total = pos
    chunk = 8 * n_bytes
    C = -(-total // chunk)
    B = -(-C // T)
    gaps = []
    for c in range(B * T + 1):
        b0 = chunk * c
        if b0 > total:
            gaps.append(0)
        else:
            gaps.append(min([s for s in starts if s >= b0] + [total]) - b0)
    bp = [sum(1 for s in starts if s < chunk * T * b) for b in range(B + 1)]
    return total, gaps, bp


@pytest.mark.parametrize("n,n_bytes,T,seed", [(0, 8, 64, 0), (1, 8, 64, 0), (3, 8, 64, 1),
                                              (777, 8, 64, 2), (5000, 8, 128, 3),
                                              (4099, 4, 64, 4), (6000, 16, 64, 5)])
def test_metadata_matches_definition(n, n_bytes, T, seed):
    w = synth.gaussian(n, 0.02, seed) if n else np.zeros(0, np.uint16)
    st = oracle.compress(w, 32, n_bytes, T)
    total, gaps, bp = python_metadata(w, st["lengths"], n_bytes, T)
    assert total == st["total_bits"]
    assert list(st["gaps"]) == gaps
    assert list(st["block_pos"]) == bp
    assert max(gaps) <= 31 and bp[0] == 0 and bp[-1] == n
    assert all(a <= b for a, b in zip(bp, bp[1:]))


def test_metadata_exact_multiple_of_chunk():
    # 64 symbols of a 2-symbol alphabet -> lengths 1 -> total bits 64 = one chunk
    w = np.array([(120 + (i % 2)) << 7 for i in range(64)], np.uint16)
    st = oracle.compress(w, 32, 8, 64)
    assert st["total_bits"] == 64 and st["num_chunks"] == 1
    total, gaps, bp = python_metadata(w, st["lengths"], 8, 64)
    assert list(st["gaps"]) == gaps and list(st["block_pos"]) == bp


def test_gap_packing_is_5bit_msb_first():
    rng = np.random.default_rng(9)
    g = rng.integers(0, 32, size=101).astype(np.uint8)
    packed = oracle.pack_gaps(g, 80)
    bits = "".join(format(int(b), "08b") for b in packed)
    assert [int(bits[5 * i:5 * i + 5], 2) for i in range(g.size)] == g.tolist()
    assert not int(bits[5 * g.size:], 2)


def test_metadata_driven_decode_of_a_block_subset():
    w = synth.gaussian(50_000, 0.02, 11)
    st = oracle.compress(w, 32, 8, 64)
    B = st["num_blocks"]
    out = np.zeros(w.size, np.uint16)
    oracle.decode_blocks(st["exp"], st["total_bits"], st["sm"], w.size, st["lengths"], 8, 64,
                         st["gaps"], st["block_pos"], 3, 4, out)
    lo, hi = st["block_pos"][3], st["block_pos"][7]
    assert np.array_equal(out[lo:hi], w[lo:hi]) and not out[:lo].any()


def test_layout_sizes():
    lay = oracle.layout(1000, 8, 64)
    assert lay == {"num_chunks": 16, "num_blocks": 1, "exp_bytes": 8 * 64 + 16,
                   "gap_bytes": 4 * (-(-5 * 65 // 32) + 2)}


@pytest.mark.parametrize("n_bytes,threads", [(4, 64), (8, 64), (8, 256), (16, 128), (8, 1024)])
def test_layout_by_enumeration(n_bytes, threads):
    """Chunk and block counts by walking the stream (a chunk exists while its
    first bit lies before total_bits; a block while its first chunk exists),
    and the padding the readers need: every chunk can be read with the 4
    bytes that follow it (Algorithm 1 reads 4 bytes past a position), and
    the two 32-bit Gaps words holding the last slot (B*T) are inside the
    buffer (Sec. 2.3.2, readings S5-S8)."""
    rng = np.random.default_rng(n_bytes * threads)
    cb = 8 * n_bytes
    sizes = [0, 1, cb - 1, cb, cb + 1, cb * threads - 1, cb * threads, cb * threads + 1]
    sizes += rng.integers(0, 40 * cb * threads, size=30).tolist()
    for total_bits in sizes:
        lay = oracle.layout(int(total_bits), n_bytes, threads)
        chunks = 0
        while cb * chunks < total_bits:
            chunks += 1
        blocks = 0
        while threads * blocks < chunks:
            blocks += 1
        assert lay["num_chunks"] == chunks and lay["num_blocks"] == blocks, total_bits
        # every chunk of every block, plus the 4 bytes after it, is inside
        assert lay["exp_bytes"] >= n_bytes * threads * blocks + 4
        assert lay["exp_bytes"] >= (total_bits + 7) // 8
        # the last slot's two words: slot B*T starts at bit 5*B*T
        last_word = (5 * blocks * threads) // 32
        assert lay["gap_bytes"] >= 4 * (last_word + 2)
        assert lay["gap_bytes"] % 4 == 0


# ---------------------------------------------------------------- plausibility
def test_gaussian_statistics_resemble_the_paper():
    """Sanity, not parity: exponent entropy near 2.6 bits, a few dozen
    exponents in use, about 11 bits per weight (Sec. 2.2, Table 1)."""
    w = synth.gaussian(1 << 20, 0.02, 12)
    counts = oracle.histogram(w)
    lengths = oracle.code_lengths(counts)
    H = entropy_bits(counts)
    assert 2.4 < H < 2.9
    assert 15 <= int((counts > 0).sum()) <= 45
    bits_per_weight = 8 + cost(counts, lengths) / counts.sum()
    assert 10.4 < bits_per_weight < 11.2


# ------------------------------------------------ matrix products (linear)
def test_bf16_to_f64_ieee_values():
    # BF16 = upper half of an IEEE binary32: values fixed by that format
    bits = np.array([0x3F80, 0xBF80, 0x4000, 0x3F00, 0x4049, 0x0000, 0x8000, 0x0001, 0x7F7F,
                     0x7F80, 0xFF80], np.uint16)
    want = [1.0, -1.0, 2.0, 0.5, 3.140625, 0.0, -0.0, 2.0 ** -133, (2 - 2 ** -7) * 2.0 ** 127,
            math.inf, -math.inf]
    got = oracle.bf16_to_f64(bits)
    for g, w in zip(got, want):
        assert g == w and math.copysign(1, g) == math.copysign(1, w)
    assert math.isnan(oracle.bf16_to_f64(np.array([0x7FC0], np.uint16))[0])


def _bits_of_small_ints(vals) -> np.ndarray:
    # small integers are exact in BF16 (8-bit significand): build their bits
    # from sign, exponent and mantissa by hand
    out = []
    for v in vals:
        v = int(v)
        if v == 0:
            out.append(0)
            continue
        s, a = (1, -v) if v < 0 else (0, v)
        e = a.bit_length() - 1
        mant = (a << (7 - e)) & 0x7F if e <= 7 else None
        assert mant is not None and (a >> e) == 1 and a == ((0x80 | mant) << e) >> 7
        out.append((s << 15) | ((e + 127) << 7) | mant)
    return np.array(out, np.uint16)


def test_linear_brute_force_exact_rationals():
    # tiny non-square shapes with distinct small-integer entries: the exact
    # result is known, and a transposed operand or swapped index changes it
    from fractions import Fraction
    rng = np.random.default_rng(3)
    for t, rows, k in [(1, 3, 2), (2, 3, 5), (3, 2, 7), (4, 5, 3)]:
        xi = rng.integers(-9, 10, size=(t, k))
        wi = rng.integers(-9, 10, size=(rows, k))
        y = oracle.linear(_bits_of_small_ints(xi.ravel()).reshape(t, k),
                          _bits_of_small_ints(wi.ravel()).reshape(rows, k))
        assert y.shape == (t, rows)
        for a in range(t):
            for r in range(rows):
                exact = sum(Fraction(int(xi[a, q])) * Fraction(int(wi[r, q])) for q in range(k))
                assert y[a, r] == float(exact)


def test_linear_identity_and_selection():
    # x = identity rows select rows of W: y[t][r] = W[r][t]
    k, rows = 6, 4
    eye = _bits_of_small_ints(np.eye(k, dtype=int).ravel()).reshape(k, k)
    wi = np.arange(rows * k).reshape(rows, k) - 11
    y = oracle.linear(eye, _bits_of_small_ints(wi.ravel()).reshape(rows, k))
    assert np.array_equal(y, wi.T.astype(np.float64))


def test_linear_error_bound_on_random_bf16():
    # float64 sums of exact BF16 products: within k * 2^-53 * sum|x w| of the
    # exact value, checked against exact integer arithmetic on scaled values
    x = synth.activations(3, 257, 9, 9)
    w = synth.gaussian(5 * 257, 0.02, 11).reshape(5, 257)
    y = oracle.linear(x, w)

    def as_int(bits):  # value * 2^150 is an integer for every finite BF16
        b = bits.astype(np.int64)
        sign = np.where(b >> 15, -1, 1)
        e, m = (b >> 7) & 0xFF, b & 0x7F
        sig = np.where(e == 0, m, m | 0x80)
        sh = np.where(e == 0, 1, e) - 1 - 7 + 150 - 127 + 1
        return [int(sg) * (int(sv) << int(s)) for sg, sv, s in zip(sign, sig, sh)]
    xs = [as_int(r) for r in x]
    ws = [as_int(r) for r in w]
    for a in range(3):
        for r in range(5):
            exact = sum(p * q for p, q in zip(xs[a], ws[r])) / 2.0 ** 300
            mag = sum(abs(p * q) for p, q in zip(xs[a], ws[r])) / 2.0 ** 300
            assert abs(y[a, r] - exact) <= 257 * 2.0 ** -53 * mag + 1e-300
