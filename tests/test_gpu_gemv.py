"""GPU parity of the fused decode-and-multiply path (df11_block_gemv): every
output against the oracle's float64 product within the fp32-accumulation
bound, against the decode-then-products driver, and run to run."""
import numpy as np
import pytest

import oracle
from paper_2504_11651_amd import codec, synth

FUSED = codec.make_layout(*codec.FUSED_LAYOUT)  # the fused kernel decodes 64-chunk blocks

from conftest import gpu_available

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]


def make_stream(shapes, seed, gaps=(), sigma=0.02, const=None):
    """shapes: [(rows, cols)]; gaps: weights left out before each matrix.
    Returns (weights, mats)."""
    parts, mats, off = [], [], 0
    for i, (r, c) in enumerate(shapes):
        g = gaps[i] if i < len(gaps) else 0
        if g:
            parts.append(synth.gaussian(g, 0.5, seed * 31 + i))  # weights of no matrix
            off += g
        if const is not None:
            parts.append(np.full(r * c, const, np.uint16))
        else:
            parts.append(synth.gaussian(r * c, sigma * (1 + i % 3), seed * 100 + i))
        mats.append((off, r, c))
        off += r * c
    return np.concatenate(parts), mats


def run_gemv(ds, mats, xs_h):
    import torch
    xs = [torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16).reshape(-1) for x in xs_h]
    ys = [torch.full((r,), float("nan"), dtype=torch.float32, device="cuda") for _, r, _ in mats]
    codec.block_gemv(ds, mats, xs, ys)
    torch.cuda.synchronize()
    return [y.cpu().numpy() for y in ys]


def check_oracle(w, mats, xs_h, ys):
    for (off, r, c), x, y in zip(mats, xs_h, ys):
        wm = w[off:off + r * c].reshape(r, c)
        ref = oracle.linear(x.reshape(1, c), wm)[0]
        mag = oracle.linear(x.reshape(1, c) & 0x7FFF, wm & 0x7FFF)[0]
        err = np.abs(y.astype(np.float64) - ref)
        assert np.all(np.isfinite(y)), "unwritten outputs"
        bad = err > c * 2.0 ** -23 * mag + 1e-30
        assert not bad.any(), f"{int(bad.sum())} outputs outside the bound"


CASES = {
    "one_matrix": dict(shapes=[(16, 2048)]),
    "two_with_gap": dict(shapes=[(24, 4096), (8, 2048)], gaps=[0, 1000]),
    "leading_gap": dict(shapes=[(16, 4096), (16, 2112)], gaps=[5000, 3]),
    "llama_like": dict(shapes=[(64, 4096), (16, 4096), (16, 4096), (64, 4096), (96, 4096),
                               (96, 4096), (64, 14336)]),
    # 1-bit codes: blocks of 4096 weights spanning three 2048-wide rows
    "one_symbol": dict(shapes=[(40, 2048), (8, 4096)], const=0x3F80),
    "heavy_gaps": dict(shapes=[(4, 2048)] * 6, gaps=[7, 4104, 8, 64, 4096 * 3 + 5, 1]),
}


@pytest.mark.parametrize("name", list(CASES))
def test_block_gemv_matches_oracle_and_driver(name):
    import torch
    kw = CASES[name]
    gaps = kw.get("gaps", ())
    # matrices must start 16-byte aligned: round the gaps up to multiples of 8
    gaps = tuple((g + 7) // 8 * 8 for g in gaps)
    w, mats = make_stream(kw["shapes"], len(name), gaps=gaps, const=kw.get("const"))
    hs = codec.encode(w, layout=FUSED)
    ds = codec.to_device(hs, "cuda")
    xs_h = [synth.activations(1, c, 55, i) for i, (_, _, c) in enumerate(mats)]
    ys = run_gemv(ds, mats, xs_h)
    check_oracle(w, mats, xs_h, ys)
    # run to run: bit-identical
    ys2 = run_gemv(ds, mats, xs_h)
    for a, b in zip(ys, ys2):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    # against decode-then-products (different summation order: to rounding);
    # that driver takes row counts that are multiples of 16 only
    if any(r % 16 for _, r, _ in mats):
        return
    xs = [torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16) for x in xs_h]
    yd = [torch.empty((1, r), dtype=torch.float32, device="cuda") for _, r, _ in mats]
    work = torch.empty(w.size, dtype=torch.bfloat16, device="cuda")
    wsb = codec.gemm_workspace_bytes(mats, 1)
    wsp = torch.empty(max(wsb // 4, 1), dtype=torch.float32, device="cuda")
    codec.block_forward(ds, work, mats, xs, yd, wsp)
    torch.cuda.synchronize()
    for (off, r, c), a, b, x in zip(mats, ys, yd, xs_h):
        wm = w[off:off + r * c].reshape(r, c)
        mag = oracle.linear(x.reshape(1, c) & 0x7FFF, wm & 0x7FFF)[0]
        assert np.all(np.abs(a - b.cpu().numpy()[0]) <= 2 * c * 2.0 ** -23 * mag + 1e-30)


def test_block_gemv_llama3_8b_block_every_output():
    """Full Llama-3-8B-shaped block: every output against the oracle's float64
    product, and against decode-then-products."""
    import torch
    w, offs = synth.llama3_8b_block()
    mats = [(off, r, c) for off, r, c, _ in offs.values()]
    ds = codec.to_device(codec.encode(w, layout=FUSED), "cuda")
    xs_h = [synth.activations(1, c, 56, i) for i, (_, _, c) in enumerate(mats)]
    ys = run_gemv(ds, mats, xs_h)
    xs = [torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16) for x in xs_h]
    yd = [torch.empty((1, r), dtype=torch.float32, device="cuda") for _, r, _ in mats]
    work = torch.empty(w.size, dtype=torch.bfloat16, device="cuda")
    wsp = torch.empty(max(codec.gemm_workspace_bytes(mats, 1) // 4, 1), dtype=torch.float32,
                      device="cuda")
    codec.block_forward(ds, work, mats, xs, yd, wsp)
    torch.cuda.synchronize()
    for (off, r, c), y, yb, x in zip(mats, ys, yd, xs_h):
        assert np.all(np.isfinite(y))
        wm = w[off:off + r * c].reshape(r, c)
        ref = oracle.linear(x, wm)[0]
        mag = oracle.linear(x & 0x7FFF, wm & 0x7FFF)[0]
        assert np.all(np.abs(y.astype(np.float64) - ref) <= c * 2.0 ** -23 * mag + 1e-30)
        yb = yb.cpu().numpy()[0]
        rel = np.linalg.norm(y - yb) / np.linalg.norm(yb)
        assert rel <= 1e-5, rel


@pytest.mark.parametrize("seed", range(24))
def test_random_streams_gemv(seed):
    """Seeded random matrix lists (2 to 64 rows, so at least 4096 weights;
    2048 to 5120 columns; gaps of weights outside every matrix) through the
    fused path: every output within the bound of the oracle's float64
    product, run to run identical."""
    rng = np.random.default_rng(800 + seed)
    k = int(rng.integers(1, 5))
    shapes = [(int(rng.integers(2, 65)), 64 * int(rng.integers(32, 81))) for _ in range(k)]
    gaps = tuple(8 * int(rng.integers(0, 700)) if rng.random() < 0.5 else 0 for _ in range(k))
    w, mats = make_stream(shapes, 900 + seed, gaps=gaps)
    ds = codec.to_device(codec.encode(w, layout=FUSED), "cuda")
    xs_h = [synth.activations(1, c, 950 + seed, i) for i, (_, _, c) in enumerate(mats)]
    ys = run_gemv(ds, mats, xs_h)
    check_oracle(w, mats, xs_h, ys)
    ys2 = run_gemv(ds, mats, xs_h)
    for a, b in zip(ys, ys2):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_gemv_on_a_side_stream_without_workspace():
    """block_gemv on a stream other than torch's current one, with the
    workspace left to the binding: the result matches the current-stream call
    bit for bit, and memory allocated while the side stream still runs does
    not disturb it."""
    import torch
    w, mats = make_stream([(48, 4096), (16, 2048)], 1234)
    ds = codec.to_device(codec.encode(w, layout=FUSED), "cuda")
    xs_h = [synth.activations(1, c, 1235, i) for i, (_, _, c) in enumerate(mats)]
    ref = run_gemv(ds, mats, xs_h)
    side = torch.cuda.Stream()
    xs = [torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16).reshape(-1) for x in xs_h]
    ys = [torch.full((r,), float("nan"), dtype=torch.float32, device="cuda") for _, r, _ in mats]
    torch.cuda.synchronize()
    for _ in range(3):
        codec.block_gemv(ds, mats, xs, ys, stream=side)
        junk = torch.full((1 << 20,), 7.0, device="cuda")  # reuses freed blocks if unprotected
        del junk
    side.synchronize()
    for a, b in zip(ys, ref):
        assert np.array_equal(a.cpu().numpy().view(np.uint32), b.view(np.uint32))
