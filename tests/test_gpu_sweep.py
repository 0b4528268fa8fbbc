"""GPU parity of the matrix-size sweep's streams: LM-head-shaped slices (the
first R rows of a 128,256 x 4096 matrix, each slice its own stream), decoded
in the launch configuration the benchmark times.  Every decoded weight must
equal the input; the library's stream must be byte-identical to the
oracle's own; sampled blocks are decoded by the oracle and compared."""
import numpy as np
import pytest

from paper_2504_11651_amd import codec, synth

from conftest import gpu_available
from test_gpu_configs import check_against_oracle_stream, check_full, decode_on_gpu

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]


@pytest.mark.parametrize("rows", [1024, 8192, 128256])
def test_lm_head_slice_bit_exact(rows):
    w = synth.lm_head(rows)
    assert w.size == rows * synth.LM_HEAD_COLS
    hs = codec.encode(w)
    assert codec.validate(hs) == 0
    out = decode_on_gpu(hs)
    check_full(w, out)
    check_against_oracle_stream(w, hs, out, sample_blocks=6, seed=rows)
