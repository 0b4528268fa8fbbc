"""GPU parity of the decode-then-GEMM driver: df11_block_gemm against the
oracle's float64 product (every output element, within the fp32-accumulation
error bound), determinism, and df11_block_forward (decode + products) against
the same products on the uncompressed weights (bit-identical)."""
import numpy as np
import pytest

import oracle
from paper_2504_11651_amd import codec, synth

from conftest import gpu_available

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]


def make_block(shapes, seed):
    """shapes: [(rows, cols)] -> (uint16 weights, [(offset, rows, cols)])."""
    mats, off, parts = [], 0, []
    for i, (r, c) in enumerate(shapes):
        parts.append(synth.gaussian(r * c, 0.02 * (1 + i % 3), seed * 100 + i))
        mats.append((off, r, c))
        off += r * c
    return np.concatenate(parts), mats


def run_gemm(w_dev, mats, xs_host, weights_out=None, ds=None):
    import torch
    xs = [torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16) for x in xs_host]
    t = xs_host[0].shape[0]
    ys = [torch.full((t, r), float("nan"), dtype=torch.float32, device="cuda")
          for _, r, _ in mats]
    wsb = codec.gemm_workspace_bytes(mats, t)
    ws = torch.empty(max(wsb // 4, 1), dtype=torch.float32, device="cuda")
    if ds is None:
        codec.block_gemm(w_dev, mats, xs, ys, ws)
    else:
        codec.block_forward(ds, weights_out, mats, xs, ys, ws)
    torch.cuda.synchronize()
    return [y.cpu().numpy() for y in ys]


def check_against_oracle(w, mats, xs, ys):
    for (off, r, c), x, y in zip(mats, xs, ys):
        wm = w[off:off + r * c].reshape(r, c)
        ref = oracle.linear(x, wm)
        mag = oracle.linear(x & 0x7FFF, wm & 0x7FFF)  # sum of |x w|
        bound = c * 2.0 ** -23 * mag + 1e-30
        err = np.abs(y.astype(np.float64) - ref)
        assert np.all(np.isfinite(y)), "unwritten or non-finite outputs"
        bad = err > bound
        assert not bad.any(), f"{int(bad.sum())} outputs outside the bound, worst " \
                              f"{float((err / bound).max()):.3g} x bound"


SHAPES = [
    [(16, 64)],
    [(48, 320)],
    [(32, 4096)],
    [(16, 4160)],               # k ranges ending in a 64-wide partial slab
    [(64, 8192)],               # split into 8 (up to 8 tokens) or 2 k ranges
    [(64, 256), (16, 256), (16, 256), (64, 256), (128, 256), (128, 256), (64, 4352)],
]
TOKENS = [1, 2, 3, 4, 8, 9, 15, 16, 17, 32, 33, 48, 64]


@pytest.mark.parametrize("si", range(len(SHAPES)))
@pytest.mark.parametrize("tokens", TOKENS)
def test_block_gemm_matches_oracle(si, tokens):
    import torch
    w, mats = make_block(SHAPES[si], si + 1)
    xs = [synth.activations(tokens, c, 77, si, m) for m, (_, _, c) in enumerate(mats)]
    w_dev = torch.from_numpy(w.view(np.int16)).cuda().view(torch.bfloat16)
    ys = run_gemm(w_dev, mats, xs)
    check_against_oracle(w, mats, xs, ys)


def test_block_gemm_deterministic_and_address_independent():
    import torch
    w, mats = make_block(SHAPES[-1], 9)
    xs = [synth.activations(64, c, 78, m) for m, (_, _, c) in enumerate(mats)]
    a = torch.from_numpy(w.view(np.int16)).cuda().view(torch.bfloat16)
    b = torch.empty(w.size + 64, dtype=torch.bfloat16, device="cuda")[8:8 + w.size]
    b.copy_(a)
    y1 = run_gemm(a, mats, xs)
    y2 = run_gemm(a, mats, xs)
    y3 = run_gemm(b, mats, xs)
    for p, q, s in zip(y1, y2, y3):
        assert np.array_equal(p.view(np.uint32), q.view(np.uint32))
        assert np.array_equal(p.view(np.uint32), s.view(np.uint32))


@pytest.mark.parametrize("tokens", [1, 64])
def test_block_forward_bit_identical_to_uncompressed(tokens):
    import torch
    w, mats = make_block(SHAPES[-1], 5)
    hs = codec.encode(w)
    ds = codec.to_device(hs, "cuda")
    xs = [synth.activations(tokens, c, 79, m) for m, (_, _, c) in enumerate(mats)]
    work = torch.full((w.size,), 0x5A5A, dtype=torch.int16, device="cuda")
    y_dec = run_gemm(None, mats, xs, weights_out=work.view(torch.bfloat16), ds=ds)
    assert np.array_equal(work.cpu().numpy().view(np.uint16), w)
    w_dev = torch.from_numpy(w.view(np.int16)).cuda().view(torch.bfloat16)
    y_raw = run_gemm(w_dev, mats, xs)
    for p, q in zip(y_dec, y_raw):
        assert np.array_equal(p.view(np.uint32), q.view(np.uint32))
    check_against_oracle(w, mats, xs, y_dec)


def test_block_forward_rejects_before_decoding():
    import torch
    w, mats = make_block([(16, 64)], 3)
    ds = codec.to_device(codec.encode(w), "cuda")
    work = torch.full((w.size,), 0x5A5A, dtype=torch.int16, device="cuda")
    xs = [torch.zeros((1, 64), dtype=torch.bfloat16, device="cuda")]
    ys = [torch.zeros((1, 16), dtype=torch.float32, device="cuda")]
    with pytest.raises(codec.DF11Error):
        codec.block_forward(ds, work.view(torch.bfloat16), [(8, 16, 64)], xs, ys)  # past the end
    torch.cuda.synchronize()
    assert int((work == 0x5A5A).sum()) == w.size  # nothing was decoded


def test_binding_refuses_host_tensors():
    # host tensors are refused before anything is enqueued
    import torch
    w, mats = make_block([(16, 2048)], 31)
    ds = codec.to_device(codec.encode(w), "cuda")
    with pytest.raises(ValueError):
        codec.decode_block(ds, torch.empty(w.size, dtype=torch.bfloat16))
    x = torch.zeros((1, 2048), dtype=torch.bfloat16)
    y = torch.zeros((1, 16), dtype=torch.float32)
    work = torch.empty(w.size, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError):
        codec.block_forward(ds, work, mats, [x], [y.cuda()])
    with pytest.raises(ValueError):
        codec.block_forward(ds, work, mats, [x.cuda()], [y])
    with pytest.raises(ValueError):
        codec.block_gemv(ds, mats, [x.cuda().reshape(-1)], [y.reshape(-1)])
    torch.cuda.synchronize()


@pytest.mark.parametrize("seed", range(24))
def test_random_blocks_forward(seed):
    """Seeded random matrix lists and token counts through decode-then-products:
    every output within the bound of the oracle's float64 product, and bit for
    bit the products on the uncompressed weights."""
    import torch
    rng = np.random.default_rng(500 + seed)
    shapes = [(16 * int(rng.integers(1, 17)), 64 * int(rng.integers(1, 65)))
              for _ in range(int(rng.integers(1, 5)))]
    tokens = int(rng.integers(1, 65))
    w, mats = make_block(shapes, 600 + seed)
    ds = codec.to_device(codec.encode(w), "cuda")
    xs = [synth.activations(tokens, c, 700 + seed, m) for m, (_, _, c) in enumerate(mats)]
    work = torch.empty(w.size, dtype=torch.bfloat16, device="cuda")
    y_dec = run_gemm(None, mats, xs, weights_out=work, ds=ds)
    w_dev = torch.from_numpy(w.view(np.int16)).cuda().view(torch.bfloat16)
    y_raw = run_gemm(w_dev, mats, xs)
    for p, q in zip(y_dec, y_raw):
        assert np.array_equal(p.view(np.uint32), q.view(np.uint32)), f"shapes {shapes} t={tokens}"
    check_against_oracle(w, mats, xs, y_dec)
