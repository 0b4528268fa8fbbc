"""Host-side checks of the benchmark's contract (no GPU needed):
  - more than one GPU is refused with a message and exit status 2, before
    anything touches a device;
  - the committed decoder counter summaries match the current decoder
    source, so the bench line's measured HBM traffic is not stale."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


@pytest.mark.parametrize("workload", ["llama31_70b_block", "llama3_8b_block", "heavy_tailed_block",
                                      "matrix_4096"])
def test_decoder_profiles_match_current_source(workload):
    import bench
    from paper_2504_11651_amd import codec
    traffic = bench.profiled_traffic(workload, codec.make_layout())
    assert traffic is not None, f"profiles/ has no counter summary for {workload} with this decoder"
    assert traffic > 0
