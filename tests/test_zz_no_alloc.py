"""df11_block_forward_noalloc: decode then products with the partial sums in
the library's fixed per-GPU array.  Its outputs must be bit-identical to
df11_block_forward with a caller workspace (same kernels, fixed summation
order), on two calls in a row, the second smaller than the first, and the
decoded block must equal the input.  Requests larger than the array are
refused before anything is enqueued."""
import numpy as np
import pytest

import oracle
from paper_2504_11651_amd import codec, synth

from conftest import gpu_available


def _block(shapes, seed):
    mats, off, parts = [], 0, []
    for i, (r, c) in enumerate(shapes):
        parts.append(synth.gaussian(r * c, 0.01 * (1 + i % 4), seed * 100 + i))
        mats.append((off, r, c))
        off += r * c
    return np.concatenate(parts), mats


def _run_both(w, mats, tokens, seed):
    """(decoded, ys from noalloc, ys from block_forward), all on the host."""
    import torch
    ds = codec.to_device(codec.encode(w), "cuda")
    xs = [torch.from_numpy(synth.activations(tokens, c, 41, seed, m).view(np.int16)).cuda()
          .view(torch.bfloat16) for m, (_, _, c) in enumerate(mats)]
    work = torch.empty(w.size, dtype=torch.bfloat16, device="cuda")
    ys = [torch.full((tokens, r), float("nan"), dtype=torch.float32, device="cuda")
          for _, r, _ in mats]
    codec.block_forward_noalloc(ds, work, mats, xs, ys)
    torch.cuda.synchronize()
    dec = work.view(torch.int16).cpu().numpy().view(np.uint16)
    got = [y.cpu().numpy() for y in ys]
    ws = torch.empty(max(codec.gemm_workspace_bytes(mats, tokens) // 4, 1), dtype=torch.float32,
                     device="cuda")
    ref = [torch.full_like(y, float("nan")) for y in ys]
    codec.block_forward(ds, work, mats, xs, ref, ws)
    torch.cuda.synchronize()
    return dec, got, [y.cpu().numpy() for y in ref], [x.view(torch.int16).cpu().numpy()
                                                      .view(np.uint16) for x in xs]


@pytest.mark.gpu
@pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")
def test_noalloc_matches_block_forward_two_calls():
    # call 1: the Llama-3-8B-shaped block at 64 tokens (28.3 MB of partial sums)
    w, offs = synth.llama3_8b_block(block=3)
    mats = [(o, r, c) for (o, r, c, _) in offs.values()]
    assert codec.gemm_workspace_bytes(mats, 64) > 16 << 20
    dec, got, ref, _ = _run_both(w, mats, 64, 1)
    assert np.array_equal(dec, w)
    for g, r in zip(got, ref):
        assert np.all(np.isfinite(g)), "unwritten outputs"
        assert np.array_equal(g.view(np.uint32), r.view(np.uint32))
    del w, dec, got, ref

    # call 2: a smaller block at 5 tokens; stale partial sums from call 1 are
    # still in the array and must not leak into these outputs
    w, mats = _block([(64, 2048), (32, 4160), (16, 8192)], 2)
    assert 0 < codec.gemm_workspace_bytes(mats, 5) < 1 << 20
    dec, got, ref, xs = _run_both(w, mats, 5, 2)
    assert np.array_equal(dec, w)
    for (off, r, c), g, rf, x in zip(mats, got, ref, xs):
        assert np.array_equal(g.view(np.uint32), rf.view(np.uint32))
        wm = w[off:off + r * c].reshape(r, c)
        x2 = x.reshape(5, c)
        bound = c * 2.0 ** -23 * oracle.linear(x2 & 0x7FFF, wm & 0x7FFF) + 1e-30
        assert np.all(np.abs(g.astype(np.float64) - oracle.linear(x2, wm)) <= bound)


def test_noalloc_refuses_more_than_its_array():
    """The Llama-3.1-70B block's products at 21 tokens need 33.5 MiB of
    partial sums: refused (host-side check, nothing is enqueued)."""
    import ctypes
    mats, off = [], 0
    for _, r, c in synth.LLAMA31_70B_BLOCK:
        mats.append((off, r, c))
        off += r * c
    assert codec.gemm_workspace_bytes(mats, 20) <= codec.STATIC_SCRATCH_BYTES
    assert codec.gemm_workspace_bytes(mats, 21) > codec.STATIC_SCRATCH_BYTES
    st = codec.Stream()
    st.sizes.n_elems = off
    m = codec._mats(mats)
    dummy = (ctypes.c_void_p * len(mats))(*([16] * len(mats)))
    rc = codec.lib().df11_block_forward_noalloc(ctypes.byref(st), ctypes.c_void_p(16), m,
                                                len(mats), dummy, 21, dummy, None)
    assert rc == -3  # DF11_E_BUFFER_TOO_SMALL
