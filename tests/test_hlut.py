"""Host-side pins of the paper's hierarchical lookup tables (Sec. 2.3.1;
appendix on compact lookup tables), built by df11_build_hlut_tables for the
ablation kernel:
  - the appendix's worked example, cut into 2-bit tables, gives exactly the
    three tables the paper prints (golden fixture with its citation);
  - decoding through the table hierarchy, as the paper describes it (LUT_1
    on the first byte, pointer entries 240..255 to LUT_(257-v) on the next
    byte, CodeLengths for the advance), gives the same symbol and length as
    the oracle's bit-by-bit tree walk, on every 16-bit prefix and on random
    32-bit windows of several code books;
  - code books the paper's format cannot express are refused."""
import functools
import json
import os

import numpy as np
import pytest

import oracle
from paper_2504_11651_amd import codec, synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def hierarchical_decode(tables, k, level_bits, window, nbits):
    """The paper's table walk over the first bits of ``window`` (an
    ``nbits``-bit integer, first bit most significant): (exponent, length)."""
    ent = 1 << level_bits
    i = 1
    e = int(tables[window >> (nbits - level_bits)])
    while e >= 240:
        i += 1
        t = 257 - e  # LUT_t, 1-based
        assert 2 <= t <= k, "pointer past the last table"
        chunk = (window >> (nbits - i * level_bits)) & (ent - 1)
        e = int(tables[(t - 1) * ent + chunk])
    return e, int(tables[k * ent + e])


def test_paper_worked_example_two_bit_tables():
    g = json.load(open(os.path.join(GOLDEN, "paper_lut_example.json")))
    names = g["symbols"]
    sym = {nm: 120 + i for i, nm in enumerate(names)}
    counts = np.zeros(256, np.uint64)
    for nm, c in zip(names, (8, 2, 2, 2, 1, 1)):
        counts[sym[nm]] = c
    cb = codec.codebook_from_counts(counts)
    tabs, k = codec.build_hlut_tables(cb, 2)
    assert k == 3
    # the paper's LUT0, LUT1, LUT2 are LUT_1, LUT_2, LUT_3 here; "->LUT1" is
    # the pointer to LUT_2 (value 255), "->LUT2" to LUT_3 (254)
    ptr = {"->LUT1": 255, "->LUT2": 254}
    for t, name in enumerate(("LUT0", "LUT1", "LUT2")):
        for two, target in g["two_level_tables"][name].items():
            want = ptr[target] if target.startswith("->") else sym[target]
            assert tabs[4 * t + int(two, 2)] == want, (name, two)
    for nm, l in g["code_lengths"].items():
        assert tabs[4 * k + sym[nm]] == l
    assert tabs.size == 4 * k + 256


def _fib_counts(terms, first):
    """Counts F1..F_terms on exponents first.. (their Huffman tree is a path)."""
    fib = [1, 1]
    while len(fib) < terms:
        fib.append(fib[-1] + fib[-2])
    c = np.zeros(256, np.uint64)
    c[first:first + terms] = fib[:terms]
    return c


@functools.lru_cache(maxsize=1)
def _books():
    return {
        "gauss": codec.build_codebook(synth.gaussian(500_000, 0.02, 11)),
        "llama3_8b_slice": codec.build_codebook(synth.llama3_8b_block()[0][:30_000_000]),
        "heavy": codec.build_codebook(synth.heavy_tailed_block(4_000_000)),
        "lm_head": codec.build_codebook(synth.lm_head(2048)),
        "fibonacci_30_capped_24": codec.codebook_from_counts(_fib_counts(30, 82), 24),
    }


@pytest.mark.parametrize("book", ["fibonacci_30_capped_24", "gauss", "heavy", "llama3_8b_slice",
                                  "lm_head"])
def test_hierarchical_decode_matches_oracle_tree_walk(book):
    cb = _books()[book]
    lengths = cb.lengths
    tabs, k = codec.build_hlut_tables(cb, 8)
    assert 1 <= k <= 17
    assert tabs.size == 256 * k + 256
    rng = np.random.default_rng(5)
    # every 16-bit prefix (random low bits), and random 32-bit windows
    wins = (np.arange(1 << 16, dtype=np.uint64) << np.uint64(16)) | \
        rng.integers(0, 1 << 16, size=1 << 16, dtype=np.uint64)
    wins = np.concatenate([wins, rng.integers(0, 1 << 32, size=20000, dtype=np.uint64)])
    for w in wins.tolist():
        want = oracle.decode_prefix(int(w), 32, lengths)
        if want is None:  # no code is a prefix (an incomplete one-symbol book)
            continue
        assert hierarchical_decode(tabs, k, 8, int(w), 32) == want, hex(w)


def test_refuses_reserved_exponents_and_too_many_tables():
    # Inf/NaN (exponent 255) and huge values use the pointer range
    cb = codec.build_codebook(synth.special_values(4096))
    with pytest.raises(codec.DF11Error) as e:
        codec.build_hlut_tables(cb, 8)
    assert e.value.rc == -6
    # Fibonacci counts at 1-bit levels need a table per internal node (39)
    cb = codec.codebook_from_counts(_fib_counts(40, 80), 32)
    with pytest.raises(codec.DF11Error) as e:
        codec.build_hlut_tables(cb, 1)
    assert e.value.rc == -6
