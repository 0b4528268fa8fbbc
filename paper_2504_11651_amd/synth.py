"""Seeded synthetic BF16 weights shaped like the paper's workloads.

The paper measures on trained LLM weights (Llama 3.x linear layers, LM heads),
which are not available here; these generators stand in for them with the same
shapes and with value distributions whose exponent statistics resemble trained
weights (a few dozen exponent values in use, about 2.6 bits of exponent
entropy, Sec. 2.2).  Nothing in this module knows how the codec works: it only
draws numbers and rounds them to BF16, and both the product path and the
oracle consume its output.

Seeding: every piece of every matrix has its own ``numpy`` PCG64 generator
seeded by ``SeedSequence([0, config, block, matrix, piece])`` with pieces of
2**22 elements, so the values do not depend on the thread count.  Per-matrix
standard deviations come from ``SeedSequence([0, config, block])``.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

PIECE = 1 << 22
BASE_SEED = 0

# (name, rows, cols); row-major [out, in] like nn.Linear weights
LLAMA3_8B_BLOCK = (
    ("q_proj", 4096, 4096), ("k_proj", 1024, 4096), ("v_proj", 1024, 4096),
    ("o_proj", 4096, 4096), ("gate_proj", 14336, 4096), ("up_proj", 14336, 4096),
    ("down_proj", 4096, 14336),
)
LLAMA31_70B_BLOCK = (
    ("q_proj", 8192, 8192), ("k_proj", 1024, 8192), ("v_proj", 1024, 8192),
    ("o_proj", 8192, 8192), ("gate_proj", 28672, 8192), ("up_proj", 28672, 8192),
    ("down_proj", 8192, 28672),
)


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to BF16 (round to nearest, ties to even), return uint16 bits.

    Equivalent to ``torch.Tensor.to(torch.bfloat16)`` for finite inputs."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + r) >> np.uint32(16)).astype(np.uint16)


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([BASE_SEED, *key])))


def _fill_pieces(out: np.ndarray, key: tuple, fill) -> None:
    """Fill ``out`` (uint16) piece by piece, in parallel; ``fill(rng, n)``
    returns float32 values for one piece."""
    n = out.size
    npieces = (n + PIECE - 1) // PIECE

    def work(p: int):
        lo, hi = p * PIECE, min(n, (p + 1) * PIECE)
        out[lo:hi] = f32_to_bf16_bits(fill(_rng(*key, p), hi - lo))

    if npieces <= 1:
        for p in range(npieces):
            work(p)
        return
    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(work, range(npieces)))


def _normal(sigma: float):
    def fill(rng: np.random.Generator, n: int) -> np.ndarray:
        x = np.empty(n, np.float32)
        rng.standard_normal(out=x, dtype=np.float32)
        x *= np.float32(sigma)
        return x
    return fill


def gaussian(n: int, sigma: float = 0.02, seed: int = 1) -> np.ndarray:
    """n BF16 weights ~ N(0, sigma^2) (uint16 bit patterns)."""
    out = np.empty(n, np.uint16)
    _fill_pieces(out, (100, seed, 0), _normal(sigma))
    return out


def matrix_4096(seed: int = 0) -> np.ndarray:
    """4096 x 4096 BF16 matrix ~ N(0, 0.02^2), one stream (16,777,216 weights)."""
    out = np.empty(4096 * 4096, np.uint16)
    _fill_pieces(out, (1, seed, 0), _normal(0.02))
    return out


def _block(shapes, config: int, block: int, sig_lo: float, sig_hi: float):
    sigmas = _rng(config, block).uniform(sig_lo, sig_hi, size=len(shapes))
    total = sum(r * c for _, r, c in shapes)
    out = np.empty(total, np.uint16)
    offsets = {}
    off = 0
    for m, ((name, r, c), s) in enumerate(zip(shapes, sigmas)):
        view = out[off:off + r * c]
        _fill_pieces(view, (config, block, m), _normal(float(s)))
        offsets[name] = (off, r, c, float(s))
        off += r * c
    return out, offsets


def llama3_8b_block(block: int = 0, config: int = 2):
    """One Llama-3-8B-shaped transformer block (q,k,v,o,gate,up,down concatenated,
    218,103,808 weights), sigma ~ U[0.008, 0.04] per matrix.  Returns
    (uint16 weights, {name: (offset, rows, cols, sigma)})."""
    return _block(LLAMA3_8B_BLOCK, config, block, 0.008, 0.04)


def llama31_70b_block(block: int = 0):
    """One Llama-3.1-70B-shaped block (855,638,016 weights), sigma ~ U[0.005, 0.03]."""
    return _block(LLAMA31_70B_BLOCK, 4, block, 0.005, 0.03)


LM_HEAD_ROWS, LM_HEAD_COLS = 128_256, 4096  # Llama-3.1-8B vocabulary x hidden size


def lm_head(rows: int = LM_HEAD_ROWS, cols: int = LM_HEAD_COLS, seed: int = 0) -> np.ndarray:
    """The first ``rows`` rows of an LM-head-shaped matrix (128,256 x 4096,
    row-major [vocab, hidden]) ~ N(0, 0.02^2).  Every piece is seeded on its
    own, so a prefix of rows is the same whatever ``rows`` is: the slices of
    the size sweep are prefixes of one matrix."""
    out = np.empty(rows * cols, np.uint16)
    _fill_pieces(out, (7, seed, cols), _normal(0.02))
    return out


def llama3_8b_stack_block(i: int):
    """Block i of the 32-block Llama-3-8B-shaped stack (block seeds (5, i))."""
    return _block(LLAMA3_8B_BLOCK, 5, i, 0.008, 0.04)


def activations(tokens: int, cols: int, *key: int) -> np.ndarray:
    """tokens x cols BF16 activations ~ N(0, 1), row-major (uint16 bit patterns),
    from the generator seeded by ``key``."""
    out = np.empty(tokens * cols, np.uint16)
    _fill_pieces(out, (200, *key), _normal(1.0))
    return out.reshape(tokens, cols)


def heavy_tailed_block(n: int = 218_103_808, seed: int = 0) -> np.ndarray:
    """Stress block: 0.02 * Student-t(3), then 0.01% outliers of magnitude
    2**U(0, 6) with random sign and 1% exact +0.0, at disjoint uniformly drawn
    positions."""
    nu = 3.0

    def fill(rng: np.random.Generator, k: int) -> np.ndarray:
        z = np.empty(k, np.float32)
        rng.standard_normal(out=z, dtype=np.float32)
        g = np.empty(k, np.float64)
        rng.standard_gamma(nu / 2.0, out=g)
        # Student-t: Z / sqrt(chi2_nu / nu) with chi2_nu = 2 * Gamma(nu/2)
        t = z * np.sqrt(nu / (2.0 * g)).astype(np.float32)
        return (t * np.float32(0.02)).astype(np.float32)

    out = np.empty(n, np.uint16)
    _fill_pieces(out, (3, seed, 0), fill)
    n_out = int(round(n * 1e-4))
    n_zero = int(round(n * 1e-2))
    rng = _rng(3, seed, 1)
    need = n_out + n_zero
    picked = np.empty(0, np.int64)
    while picked.size < need:
        cand = rng.integers(0, n, size=int(need * 1.1) + 16)
        allc = np.concatenate([picked, cand])
        _, first = np.unique(allc, return_index=True)
        picked = allc[np.sort(first)]
    picked = picked[:need]
    mag = np.exp2(rng.uniform(0.0, 6.0, size=n_out)).astype(np.float32)
    sgn = np.where(rng.integers(0, 2, size=n_out) == 1, np.float32(-1), np.float32(1))
    out[picked[:n_out]] = f32_to_bf16_bits(mag * sgn)
    out[picked[n_out:]] = 0
    return out


def fibonacci_exponents(terms: int = 40, first_exp: int = 80, seed: int = 0) -> np.ndarray:
    """Weights whose exponents first_exp .. first_exp+terms-1 occur F1..F_terms
    times (F1 = F2 = 1), in shuffled order, with uniform signs and mantissas.
    With 40 terms an unconstrained Huffman tree is 39 deep, so a 32-bit cap
    binds.  N = F_(terms+2) - 1 (267,914,295 for 40 terms)."""
    fib = [1, 1]
    while len(fib) < terms:
        fib.append(fib[-1] + fib[-2])
    fib = np.array(fib[:terms], np.int64)
    exps = np.repeat(np.arange(first_exp, first_exp + terms, dtype=np.uint16), fib)
    rng = _rng(6, seed, terms)
    rng.shuffle(exps)
    sm = rng.integers(0, 256, size=exps.size, dtype=np.uint16)
    return ((sm & np.uint16(0x80)) << np.uint16(8)) | (exps << np.uint16(7)) | (sm & np.uint16(0x7F))


def all_bf16_patterns() -> np.ndarray:
    """Every 16-bit pattern once: +-0, subnormals, +-Inf, every NaN payload."""
    return np.arange(65536, dtype=np.uint32).astype(np.uint16)


def special_values(n: int = 4096, seed: int = 7) -> np.ndarray:
    """Gaussian weights salted with +-0, subnormals, +-Inf, NaNs, max/min normals."""
    w = gaussian(n, 0.02, seed)
    specials = np.array([0x0000, 0x8000, 0x0001, 0x807F, 0x7F80, 0xFF80, 0x7FC0, 0xFFFF,
                         0x7F7F, 0xFF7F, 0x0080, 0x8080, 0x7F81, 0x3F80], np.uint16)
    rng = _rng(7, seed, 1)
    pos = rng.choice(n, size=min(n, 4 * specials.size), replace=False)
    w[pos] = np.resize(specials, pos.size)
    return w
