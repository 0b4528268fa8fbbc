"""The decode and the decode-then-products driver inside a captured HIP graph
(torch.cuda.CUDAGraph): the library allocates nothing and records no memset
or host synchronisation, so a captured launch replays the same kernels.
Every replay is checked against the eager result, with eager work and
synchronisations between replays."""
import numpy as np
import pytest

import oracle
from paper_2504_11651_amd import codec, synth

from conftest import gpu_available

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]


@pytest.mark.parametrize("T", [64, 128])
def test_decode_block_replays_in_a_graph(T):
    """Both one-wavefront decoders: 64-chunk blocks and 128-chunk blocks."""
    import torch
    wa = synth.gaussian(3_000_017, 0.02, 81)
    wb = synth.gaussian(1_500_001, 0.03, 82)
    lay = codec.make_layout(8, T, 11)
    da = codec.to_device(codec.encode(wa, layout=lay), "cuda")
    db = codec.to_device(codec.encode(wb, layout=lay), "cuda")
    out_a = torch.full((wa.size,), 0x5A5A, dtype=torch.int16, device="cuda")
    out_b = torch.empty(wb.size, dtype=torch.int16, device="cuda")
    ref_a = torch.from_numpy(wa.view(np.int16)).cuda()
    ref_b = torch.from_numpy(wb.view(np.int16)).cuda()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):  # eager call first: launch shapes are cached
        codec.decode_block(da, out_a.view(torch.bfloat16))
    torch.cuda.synchronize()
    assert torch.equal(out_a, ref_a)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        codec.decode_block(da, out_a.view(torch.bfloat16))
    for rep in range(4):
        out_a.fill_(0x5A5A)                                  # eager work between replays
        codec.decode_block(db, out_b.view(torch.bfloat16))   # another stream, eagerly
        torch.cuda.synchronize()
        assert torch.equal(out_b, ref_b), f"eager decode before replay {rep}"
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out_a, ref_a), f"replay {rep}"


def test_block_forward_replays_in_a_graph():
    import torch
    shapes = [(64, 2048), (16, 2048), (128, 4096)]
    mats, off = [], 0
    for r, c in shapes:
        mats.append((off, r, c))
        off += r * c
    w = synth.gaussian(off, 0.02, 83)
    ds = codec.to_device(codec.encode(w), "cuda")
    for tokens in (1, 64):
        xs_h = [synth.activations(tokens, c, 84, m) for m, (_, _, c) in enumerate(mats)]
        xs = [torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16) for x in xs_h]
        ys = [torch.empty((tokens, r), dtype=torch.float32, device="cuda") for _, r, _ in mats]
        work = torch.empty(off, dtype=torch.bfloat16, device="cuda")
        ws = torch.empty(max(codec.gemm_workspace_bytes(mats, tokens) // 4, 1),
                         dtype=torch.float32, device="cuda")
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            codec.block_forward(ds, work, mats, xs, ys, ws)
        torch.cuda.synchronize()
        eager = [y.clone() for y in ys]
        for (o, r, c), x, y in zip(mats, xs_h, eager):
            wm = w[o:o + r * c].reshape(r, c)
            ref = oracle.linear(x, wm)
            mag = oracle.linear(x & 0x7FFF, wm & 0x7FFF)
            assert np.all(np.abs(y.cpu().numpy() - ref) <= c * 2.0 ** -23 * mag + 1e-30)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            codec.block_forward(ds, work, mats, xs, ys, ws)
        for rep in range(3):
            for y in ys:
                y.fill_(float("nan"))
            work.zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(work.view(torch.int16).cpu(),
                               torch.from_numpy(w.view(np.int16))), f"tokens {tokens} replay {rep}"
            for a, b in zip(ys, eager):
                assert torch.equal(a.view(torch.int32), b.view(torch.int32)), \
                    f"tokens {tokens} replay {rep}"


def test_block_gemv_replays_in_a_graph():
    import torch
    shapes = [(64, 2048), (16, 2048), (128, 4096)]
    mats, off = [], 0
    for r, c in shapes:
        mats.append((off, r, c))
        off += r * c
    w = synth.gaussian(off, 0.02, 85)
    ds = codec.to_device(codec.encode(w, layout=codec.make_layout(*codec.FUSED_LAYOUT)), "cuda")
    xs = [torch.from_numpy(synth.activations(1, c, 86, m).view(np.int16)).cuda()
          .view(torch.bfloat16).reshape(-1) for m, (_, _, c) in enumerate(mats)]
    ys = [torch.empty(r, dtype=torch.float32, device="cuda") for _, r, _ in mats]
    ws = torch.empty(max(codec.gemv_workspace_bytes(ds, mats) // 4, 4), dtype=torch.float32,
                     device="cuda")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        codec.block_gemv(ds, mats, xs, ys, ws)
    torch.cuda.synchronize()
    eager = [y.clone() for y in ys]
    assert all(bool(torch.isfinite(y).all()) for y in eager)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        codec.block_gemv(ds, mats, xs, ys, ws)
    for rep in range(3):
        for y in ys:
            y.fill_(float("nan"))
        ws.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(ys, eager):
            assert torch.equal(a.view(torch.int32), b.view(torch.int32)), f"replay {rep}"
