"""GPU parity: the HIP decoder (through the C ABI) against the oracle, element
by element, on small and edge-case streams under several launch layouts."""
import numpy as np
import pytest

import oracle
from paper_2504_11651_amd import codec, synth

from conftest import gpu_available

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]

CASES = {
    "one": lambda: np.array([0xBF80], np.uint16),
    "two": lambda: np.array([0x3F80, 0x0001], np.uint16),
    "seventeen": lambda: synth.gaussian(17, 0.02, 17),
    "single_symbol": lambda: (np.arange(70_001, dtype=np.uint16) & 0x807F) | (100 << 7),
    "gauss_1000": lambda: synth.gaussian(1000, 0.02, 1),
    "gauss_65537": lambda: synth.gaussian(65_537, 0.02, 2),
    "gauss_1m": lambda: synth.gaussian(1_000_003, 0.02, 3),
    "gauss_wide": lambda: synth.gaussian(300_000, 5.0, 4),
    "special": lambda: synth.special_values(200_000),
    "patterns": synth.all_bf16_patterns,
    "fib24": lambda: synth.fibonacci_exponents(24),
    "heavy": lambda: synth.heavy_tailed_block(500_000, 2),
}
LAYOUTS = [(8, 64, 8), (8, 64, 11), (8, 64, 12), (8, 128, 8), (8, 128, 10), (8, 128, 11),
           (8, 128, 12), (8, 256, 12), (8, 512, 11), (8, 1024, 12)]


def oracle_reference(w: np.ndarray, cap: int = 32) -> np.ndarray:
    st = oracle.compress(w, cap, 8, 256)
    ref = oracle.decode_serial(st["exp"], st["total_bits"], st["sm"], w.size, st["lengths"])
    assert np.array_equal(ref, w)
    return ref


def gpu_decode(hs, poison: int, guard: int = 64, stream=None):
    import torch
    ds = codec.to_device(hs, "cuda")
    n = ds.n_elems
    buf = torch.full((n + guard,), poison, dtype=torch.int16, device="cuda")
    codec.decode_block(ds, buf[:n].view(torch.bfloat16), stream=stream)
    torch.cuda.synchronize()
    host = buf.cpu().numpy().view(np.uint16)
    assert (host[n:] == np.uint16(poison & 0xFFFF)).all(), "decoder wrote past the output"
    return host[:n]


@pytest.mark.parametrize("lay", LAYOUTS, ids=lambda l: "T%d_K%d" % l[1:])
@pytest.mark.parametrize("case", sorted(CASES))
def test_decode_matches_oracle(case, lay):
    w = CASES[case]()
    ref = oracle_reference(w)
    hs = codec.encode(w, layout=codec.make_layout(*lay))
    for poison in (0x5555, -0x5556):  # two patterns: every element must be written
        got = gpu_decode(hs, poison)
        bad = np.flatnonzero(got != ref)
        assert bad.size == 0, f"{bad.size} mismatches, first {bad[:8].tolist()}"


@pytest.mark.parametrize("cap,K", [(12, 8), (10, 8), (16, 9)])
def test_long_codes_through_escape_path(cap, K):
    """Capped Fibonacci histogram: most code lengths exceed the table width."""
    w = synth.fibonacci_exponents(28)
    ref = oracle_reference(w, cap)
    hs = codec.encode(w, layout=codec.make_layout(8, 256, K), max_code_len=cap)
    assert hs.codebook.max_code_len == cap
    got = gpu_decode(hs, 0x1234)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("T", [64, 128, 256, 1024])
def test_launch_shape(T):
    """The decoder's launch for a stream long enough to fill the GPU:
    - T = 64 or 128: one wavefront per block, W = block/64 waves per
      workgroup sharing the tables, LDS = tables + one output buffer per
      wave, a persistent grid of whole CUs' worth of workgroups, at least 3
      waves per SIMD;
    - T = 256: one workgroup of T threads per block, LDS = tables + 16 scan
      slots + one block buffer;
    - T = 1024: one workgroup of T/2 threads (two chunks per lane), LDS =
      tables + 16 scan slots + two block buffers (one where two do not fit:
      the one-symbol stream at T = 1024 in test_decode_matches_oracle).
    The decode in that shape is bit-exact."""
    import torch
    w = synth.gaussian(40_000_000, 0.02, 5)
    hs = codec.encode(w, layout=codec.make_layout(8, T, 11))
    ds = codec.to_device(hs, "cuda")
    grid, block, lds = codec.launch_shape(ds)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    nb = int(hs.sizes.num_blocks)
    tables = (8 * 2048 + 2 * 4 * 33 + 256 + 15) // 16 * 16
    buf = (int(hs.sizes.max_elems_per_block) + 128 + 15) // 16 * 16
    if T <= 128:
        W = block // 64
        assert block % 64 == 0 and W in (4, 8, 12, 16)
        assert lds == tables + W * buf
        assert grid <= (nb + W - 1) // W and grid % cus == 0
        assert grid * W >= 3 * 4 * cus  # at least 3 waves per SIMD
    elif T == 1024:
        assert block == T // 2 and lds == tables + 4 * 16 + 2 * buf
        assert grid <= nb
    else:
        assert block == T and lds == tables + 4 * 16 + buf
        assert grid <= nb
    out = torch.empty(w.size, dtype=torch.int16, device="cuda")
    codec.decode_block(ds, out.view(torch.bfloat16))
    torch.cuda.synchronize()
    assert torch.equal(out, torch.from_numpy(w.view(np.int16)).cuda())


def test_empty_stream_launches_nothing():
    import torch
    hs = codec.encode(np.zeros(0, np.uint16))
    ds = codec.to_device(hs, "cuda")
    out = torch.full((8,), 7, dtype=torch.int16, device="cuda")
    codec.decode_block(ds, out.view(torch.bfloat16))
    torch.cuda.synchronize()
    assert (out.cpu() == 7).all()


def test_decode_is_deterministic_and_stream_ordered():
    import torch
    w = synth.gaussian(2_000_000, 0.03, 9)
    hs = codec.encode(w)
    ds = codec.to_device(hs, "cuda")
    s = torch.cuda.Stream()
    outs = []
    for _ in range(3):
        o = torch.empty(w.size, dtype=torch.bfloat16, device="cuda")
        with torch.cuda.stream(s):
            codec.decode_block(ds, o, stream=s)
        outs.append(o)
    s.synchronize()
    for o in outs:
        assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16))
    assert np.array_equal(outs[0].view(torch.int16).cpu().numpy().view(np.uint16), w)


def test_decode_into_aligned_view_of_workspace():
    import torch
    w = synth.gaussian(123_457, 0.02, 10)
    hs = codec.encode(w)
    ds = codec.to_device(hs, "cuda")
    ws = torch.full((w.size + 1024,), -1, dtype=torch.int16, device="cuda")
    view = ws[512:512 + w.size]  # 1 KiB offset keeps 16-byte alignment
    codec.decode_block(ds, view.view(torch.bfloat16))
    torch.cuda.synchronize()
    host = ws.cpu().numpy().view(np.uint16)
    assert np.array_equal(host[512:512 + w.size], w)
    assert (host[:512] == 0xFFFF).all() and (host[512 + w.size:] == 0xFFFF).all()


def test_misaligned_output_is_rejected():
    import torch
    hs = codec.encode(synth.gaussian(1000, 0.02, 1))
    ds = codec.to_device(hs, "cuda")
    ws = torch.empty(2000, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(codec.DF11Error):
        codec.decode_block(ds, ws[1:1001])


def _random_case(seed: int):
    """Seeded random stream: log-uniform size and scale, a random share of
    special values and exact zeros, a random launch layout and code cap."""
    rng = np.random.default_rng(1000 + seed)
    n = int(np.exp(rng.uniform(0.0, np.log(2_000_000))))
    sigma = float(np.exp(rng.uniform(np.log(1e-4), np.log(10.0))))
    w = synth.gaussian(max(n, 1), sigma, 2000 + seed)
    k = int(rng.integers(0, 3))
    if k >= 1:  # some special values (Inf, NaN payloads, subnormals, huge)
        sv = synth.special_values(max(n // 50, 1), 3000 + seed)
        w[rng.integers(0, w.size, sv.size)] = sv
    if k == 2:  # and exact zeros
        w[rng.integers(0, w.size, max(w.size // 100, 1))] = 0
    lay = LAYOUTS[int(rng.integers(0, len(LAYOUTS)))]
    cap = int(rng.choice([24, 32]))
    return w, lay, cap


@pytest.mark.parametrize("seed", range(40))
def test_random_streams_round_trip(seed):
    w, lay, cap = _random_case(seed)
    hs = codec.encode(w, layout=codec.make_layout(*lay), max_code_len=cap)
    assert codec.validate(hs) == 0
    if w.size <= 200_000:  # the library's stream is the oracle's, byte for byte
        st = oracle.compress(w, cap, 8, lay[1])
        assert np.array_equal(st["exp"], hs.exp)
        assert np.array_equal(st["gaps_packed"], hs.gaps)
        assert np.array_equal(st["block_pos"], hs.block_pos)
    got = gpu_decode(hs, 0x2D2D)
    bad = np.flatnonzero(got != w)
    assert bad.size == 0, f"n={w.size} layout={lay} cap={cap}: {bad.size} mismatches, " \
                          f"first {bad[:8].tolist()}"
