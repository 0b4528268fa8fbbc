"""GPU parity at full workload sizes, in the launch configuration the
benchmark times (default layout: n = 8 bytes per thread, T = 64, 11-bit
table).  Every decoded weight is compared with the generator's input (a
property that holds at any size, given the oracle's pinned round trip); the
library's stream is compared byte for byte with the oracle's own stream, and
sampled blocks are decoded by the oracle and compared with the GPU output."""
import functools

import numpy as np
import pytest

import oracle
from paper_2504_11651_amd import codec, synth

from conftest import gpu_available

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]


@functools.lru_cache(maxsize=1)
def weights(name: str) -> np.ndarray:
    if name == "matrix_4096":
        return synth.matrix_4096()
    if name == "llama3_8b_block":
        return synth.llama3_8b_block()[0]
    if name == "heavy_tailed_block":
        return synth.heavy_tailed_block()
    if name == "llama31_70b_block":
        return synth.llama31_70b_block()[0]
    if name == "fibonacci_40":
        return synth.fibonacci_exponents(40)
    raise KeyError(name)


def decode_on_gpu(hs):
    import torch
    ds = codec.to_device(hs, "cuda")
    out = torch.full((ds.n_elems,), 0x5A5A, dtype=torch.int16, device="cuda")
    codec.decode_block(ds, out.view(torch.bfloat16))
    torch.cuda.synchronize()
    del ds
    return out


def check_full(w: np.ndarray, out) -> None:
    import torch
    ref = torch.from_numpy(w.view(np.int16)).to(out.device)
    same = out == ref
    if not bool(same.all()):
        bad = torch.nonzero(~same).flatten()[:8].cpu().tolist()
        pytest.fail(f"{int((~same).sum())} mismatches, first at {bad}")


def check_against_oracle_stream(w, hs, out, sample_blocks=12, seed=0):
    """Oracle's own stream == library stream; oracle block decode == GPU."""
    st = oracle.compress(w, 32, 8, hs.layout.threads_per_block)
    assert np.array_equal(st["lengths"], hs.codebook.lengths)
    assert st["total_bits"] == hs.sizes.total_bits
    assert np.array_equal(st["exp"], hs.exp)
    assert np.array_equal(st["sm"], hs.sm[:w.size])
    assert np.array_equal(st["gaps_packed"], hs.gaps)
    assert np.array_equal(st["block_pos"], hs.block_pos)
    B = st["num_blocks"]
    rng = np.random.default_rng(seed)
    blocks = sorted(set([0, B - 1] + rng.integers(0, B, size=sample_blocks).tolist()))
    got = out.view(-1)
    ref = np.zeros(w.size, np.uint16)
    for b in blocks:
        oracle.decode_blocks(st["exp"], st["total_bits"], st["sm"], w.size, st["lengths"], 8,
                             hs.layout.threads_per_block, st["gaps"], st["block_pos"], b, 1, ref)
        lo, hi = int(st["block_pos"][b]), int(st["block_pos"][b + 1])
        g = got[lo:hi].cpu().numpy().view(np.uint16)
        assert np.array_equal(g, ref[lo:hi]), f"block {b}"


@pytest.mark.parametrize("name", ["matrix_4096", "llama3_8b_block", "heavy_tailed_block"])
def test_config_bit_exact_and_oracle_stream(name):
    w = weights(name)
    hs = codec.encode(w)
    assert codec.validate(hs) == 0
    out = decode_on_gpu(hs)
    check_full(w, out)
    check_against_oracle_stream(w, hs, out)


def test_llama31_70b_block_bit_exact():
    w = weights("llama31_70b_block")
    assert w.size == 855_638_016
    hs = codec.encode(w)
    out = decode_on_gpu(hs)
    check_full(w, out)
    check_against_oracle_stream(w, hs, out, sample_blocks=8, seed=4)


def test_fibonacci_cap_binds_32_bit_codes():
    w = weights("fibonacci_40")
    hs = codec.encode(w)
    assert hs.codebook.max_code_len == 32
    out = decode_on_gpu(hs)
    check_full(w, out)


# ------------------------------------------------------------------------
# 32-block Llama-3-8B-shaped stack kept compressed on the device; per block:
# decode into one reused BF16 workspace, then the block's 7 products on the
# matrix cores at 1 and 64 tokens.
STACK_BLOCKS = 32
SAMPLE_ROWS = 32


def stack_mats():
    mats, off = [], 0
    for _, r, c in synth.LLAMA3_8B_BLOCK:
        mats.append((off, r, c))
        off += r * c
    return mats, off


@pytest.fixture(scope="module")
def stack_streams():
    streams = []
    for i in range(STACK_BLOCKS):
        w, _ = synth.llama3_8b_stack_block(i)
        hs = codec.encode(w)
        streams.append(codec.to_device(hs, "cuda"))
        del w, hs
    yield streams
    del streams


def stack_activations(i: int, tokens: int):
    """x for q, k, v, o, gate, up: one [tokens, 4096] draw; down: [tokens, 14336]."""
    x1 = synth.activations(tokens, 4096, 5, i, 1)
    x2 = synth.activations(tokens, 14336, 5, i, 2)
    return [x1] * 6 + [x2]


@pytest.mark.parametrize("tokens", [1, 64])
def test_llama3_8b_stack_decode_then_gemm(stack_streams, tokens):
    import torch
    mats, n = stack_mats()
    rng = np.random.default_rng(tokens)
    work = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    raw = torch.empty(n, dtype=torch.int16, device="cuda")
    ws = torch.empty(max(codec.gemm_workspace_bytes(mats, tokens) // 4, 1), dtype=torch.float32,
                     device="cuda")
    worst = 0.0
    for i, ds in enumerate(stack_streams):
        w, _ = synth.llama3_8b_stack_block(i)
        xs_h = stack_activations(i, tokens)
        xs = [torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16) for x in xs_h]
        y_dec = [torch.empty((tokens, r), dtype=torch.float32, device="cuda") for _, r, _ in mats]
        y_raw = [torch.empty((tokens, r), dtype=torch.float32, device="cuda") for _, r, _ in mats]
        codec.block_forward(ds, work, mats, xs, y_dec, ws)
        raw.copy_(torch.from_numpy(w.view(np.int16)))
        codec.block_gemm(raw.view(torch.bfloat16), mats, xs, y_raw, ws)
        torch.cuda.synchronize()
        # decoded weights are the weights; products bit-identical to the
        # products on the uncompressed weights
        assert torch.equal(work.view(torch.int16), raw), f"block {i}: decode differs"
        for m, (p, q) in enumerate(zip(y_dec, y_raw)):
            assert torch.equal(p.view(torch.int32), q.view(torch.int32)), f"block {i} matrix {m}"
        # sampled output features against a CPU fp32-accumulate reference
        # (relative Frobenius error <= 1e-2) and the oracle's float64 product
        for m, ((off, r, c), x) in enumerate(zip(mats, xs_h)):
            rows = np.sort(rng.choice(r, SAMPLE_ROWS, replace=False))
            wm = w[off:off + r * c].reshape(r, c)[rows]
            y = y_dec[m][:, torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
            ref32 = (oracle.bf16_to_f64(x).astype(np.float32) @
                     oracle.bf16_to_f64(wm).astype(np.float32).T).astype(np.float64)
            rel = np.linalg.norm(y - ref32) / np.linalg.norm(ref32)
            assert rel <= 1e-2, f"block {i} matrix {m}: relative error {rel}"
            worst = max(worst, rel)
            ref = oracle.linear(x, wm)
            mag = oracle.linear(x & 0x7FFF, wm & 0x7FFF)
            assert np.all(np.abs(y - ref) <= c * 2.0 ** -23 * mag + 1e-30), f"block {i} matrix {m}"
    print(f"tokens={tokens}: worst relative Frobenius error vs fp32 reference {worst:.3g}")


@pytest.mark.parametrize("tokens", [1, 64])
def test_llama3_8b_stack_block0_every_output(stack_streams, tokens):
    """Every output of one full stack block (block 0, all 7 matrices) against
    the oracle's float64 product, within the fp32-accumulation bound
    k * 2^-23 * sum |x w|, at 1 and 64 tokens (the split-k layouts the
    products use at both token counts)."""
    import torch
    mats, n = stack_mats()
    w, _ = synth.llama3_8b_stack_block(0)
    xs_h = stack_activations(0, tokens)
    xs = [torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16) for x in xs_h]
    ys = [torch.full((tokens, r), float("nan"), dtype=torch.float32, device="cuda")
          for _, r, _ in mats]
    work = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(max(codec.gemm_workspace_bytes(mats, tokens) // 4, 1), dtype=torch.float32,
                     device="cuda")
    codec.block_forward(stack_streams[0], work, mats, xs, ys, ws)
    torch.cuda.synchronize()
    for m, ((off, r, c), x, y) in enumerate(zip(mats, xs_h, ys)):
        wm = w[off:off + r * c].reshape(r, c)
        got = y.cpu().numpy().astype(np.float64)
        assert np.all(np.isfinite(got)), f"matrix {m}: unwritten outputs"
        ref = oracle.linear(x, wm)
        mag = oracle.linear(x & 0x7FFF, wm & 0x7FFF)
        bad = np.abs(got - ref) > c * 2.0 ** -23 * mag + 1e-30
        assert not bad.any(), f"matrix {m}: {int(bad.sum())} of {got.size} outputs outside the bound"
