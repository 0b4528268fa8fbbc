"""GPU parity at the largest stream the format allows: 2^32 - 1 weights (the
output positions are 32-bit), in the default layout (128-chunk blocks, two
chunks per lane) and in the 64-chunk layout.  Every decoded weight is
compared with the input, and the fused decode-and-multiply path (64-chunk
blocks) is checked on sampled rows of a matrix that ends just before the
stream does (the last block then reaches into weights that belong to no
matrix)."""
import numpy as np
import pytest

import oracle
from paper_2504_11651_amd import codec, synth

from conftest import gpu_available

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]

N_MAX = 2 ** 32 - 1


def _decode_all(ds, w):
    import torch
    out = torch.full((N_MAX,), 0x5A5A, dtype=torch.int16, device="cuda")
    codec.decode_block(ds, out.view(torch.bfloat16))
    torch.cuda.synchronize()
    ref = torch.from_numpy(w.view(np.int16)).cuda()
    same = out == ref
    if not bool(same.all()):
        bad = torch.nonzero(~same).flatten()[:8].cpu().tolist()
        pytest.fail(f"{int((~same).sum())} mismatches, first at {bad}")
    del out, ref, same
    torch.cuda.empty_cache()


def test_largest_stream_decodes_bit_exact():
    import torch
    print(f"generating {N_MAX} weights", flush=True)
    w = synth.gaussian(N_MAX, 0.02, 2024)
    for lay in (codec.make_layout(), codec.make_layout(*codec.FUSED_LAYOUT)):
        print(f"layout T={lay.threads_per_block}", flush=True)
        hs = codec.encode(w, layout=lay)
        assert codec.validate(hs) == 0
        assert int(hs.block_pos[-1]) == N_MAX
        ds = codec.to_device(hs, "cuda")
        del hs
        _decode_all(ds, w)
        if lay.threads_per_block != codec.FUSED_LAYOUT[1]:
            del ds
            torch.cuda.empty_cache()

    # one matrix of 4096 columns covering all but the last 4095 weights
    rows, cols = N_MAX // 4096, 4096
    mats = [(0, rows, cols)]
    x_h = synth.activations(1, cols, 57, 0)
    x = torch.from_numpy(x_h.view(np.int16)).cuda().view(torch.bfloat16).reshape(-1)
    y = torch.full((rows,), float("nan"), dtype=torch.float32, device="cuda")
    codec.block_gemv(ds, mats, [x], [y])
    torch.cuda.synchronize()
    y = y.cpu().numpy()
    assert np.all(np.isfinite(y))
    rng = np.random.default_rng(1)
    sample = np.unique(np.concatenate([[0, 1, rows - 2, rows - 1],
                                       rng.choice(rows, 60, replace=False)]))
    wm = w[:rows * cols].reshape(rows, cols)[sample]
    ref = oracle.linear(x_h, wm)[0]
    mag = oracle.linear(x_h & 0x7FFF, wm & 0x7FFF)[0]
    assert np.all(np.abs(y[sample].astype(np.float64) - ref) <= cols * 2.0 ** -23 * mag + 1e-30)
