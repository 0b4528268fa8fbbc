"""GPU parity of the paper's kernel on gfx950 (df11_decode_block_hlut, the
ablation beside df11_decode_block): every decoded weight equals the input
(and, for small inputs, the oracle's bit-serial decode of the same stream),
on edge cases, seeded random streams at every supported T, and the
Llama-3-8B- and Llama-3.1-70B-shaped blocks at full size.  Outputs are
pre-filled with a poison pattern and followed by a guard region, so an
unwritten element or a write past the end fails."""
import numpy as np
import pytest

import oracle
from paper_2504_11651_amd import codec, synth

from conftest import gpu_available

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]

GUARD = 64
POISON = 0x5A5A


def decode_hlut(w, T, cap=32):
    import torch
    hs = codec.encode(w, layout=codec.make_layout(8, T, 11), max_code_len=cap)
    assert codec.validate(hs) == 0
    ds = codec.to_device(hs, "cuda")
    hl = codec.DeviceHlut(hs, "cuda")
    buf = torch.full((w.size + GUARD,), POISON, dtype=torch.int16, device="cuda")
    codec.decode_block_hlut(ds, hl, buf.view(torch.bfloat16))
    torch.cuda.synchronize()
    return hs, hl.k, buf


def check(w, hs, buf, with_oracle):
    import torch
    ref = torch.from_numpy(w.view(np.int16)).cuda()
    got = buf[:w.size]
    same = got == ref
    if not bool(same.all()):
        bad = torch.nonzero(~same).flatten()[:8].cpu().tolist()
        pytest.fail(f"{int((~same).sum())} of {w.size} differ, first at {bad}")
    assert bool((buf[w.size:] == POISON).all()), "write past the end"
    if with_oracle:
        dec = oracle.decode_serial(hs.exp, hs.sizes.total_bits, hs.sm, w.size,
                                   hs.codebook.lengths)
        assert np.array_equal(dec, w)


def fib_weights(terms, first, seed):
    fib = [1, 1]
    while len(fib) < terms:
        fib.append(fib[-1] + fib[-2])
    e = np.repeat(np.arange(first, first + terms, dtype=np.uint16), fib[:terms])
    rng = np.random.default_rng(seed)
    rng.shuffle(e)
    sm = rng.integers(0, 256, size=e.size, dtype=np.uint16)
    return ((sm & 0x80) << 8) | (e << 7) | (sm & 0x7F)


def patterns_below_240():
    p = synth.all_bf16_patterns()
    return p[((p >> 7) & 0xFF) < 240]


EDGE = {
    "one": lambda: synth.gaussian(1, 0.02, 1),
    "seven": lambda: synth.gaussian(7, 0.02, 2),
    "one_symbol": lambda: np.full(5000, 0x3F80, np.uint16),
    "two_symbols": lambda: np.array([0x3F80, 0xBF00, 0x3F80] * 999, np.uint16),
    "ragged": lambda: synth.gaussian(100_003, 0.02, 3),
    "patterns": patterns_below_240,
    "fib26_capped20": lambda: fib_weights(26, 90, 4),
    "wide_scale": lambda: synth.gaussian(300_000, 3.0, 5),
}


@pytest.mark.parametrize("T", [64, 256, 1024])
@pytest.mark.parametrize("case", sorted(EDGE))
def test_hlut_edge_cases(case, T):
    w = EDGE[case]()
    cap = 20 if case.startswith("fib") else 32
    hs, k, buf = decode_hlut(w, T, cap)
    if case.startswith("fib"):
        assert hs.codebook.max_code_len == 20
    check(w, hs, buf, with_oracle=True)


def test_hlut_empty_stream_launches_nothing():
    import torch
    hs = codec.encode(np.zeros(0, np.uint16))
    ds = codec.to_device(hs, "cuda")
    out = torch.empty(1, dtype=torch.bfloat16, device="cuda")
    hl_tables = torch.zeros(512, dtype=torch.uint8, device="cuda")

    class H:
        tables, k = hl_tables, 1
    codec.decode_block_hlut(ds, H, out)
    torch.cuda.synchronize()


@pytest.mark.parametrize("seed", range(20))
def test_hlut_random_streams(seed):
    rng = np.random.default_rng(4000 + seed)
    n = int(np.exp(rng.uniform(0, np.log(2_000_000))))
    T = int(rng.choice([64, 128, 256, 512, 1024]))
    scale = float(np.exp(rng.uniform(np.log(1e-4), np.log(10.0))))
    w = synth.gaussian(n, scale, 5000 + seed)
    if rng.random() < 0.3:
        w[rng.integers(0, n, size=max(1, n // 100))] = 0
    hs, k, buf = decode_hlut(w, T)
    check(w, hs, buf, with_oracle=n <= 300_000)


@pytest.mark.parametrize("name", ["llama3_8b_block", "llama31_70b_block"])
def test_hlut_full_blocks(name):
    w = synth.llama3_8b_block()[0] if name == "llama3_8b_block" else synth.llama31_70b_block()[0]
    hs, k, buf = decode_hlut(w, 256)
    assert 1 <= k <= 17
    check(w, hs, buf, with_oracle=False)


def test_hlut_refuses_reserved_exponents():
    hs = codec.encode(synth.special_values(4096))
    with pytest.raises(codec.DF11Error) as e:
        codec.build_hlut_tables(hs.codebook, 8)
    assert e.value.rc == -6
