"""Host-side checks of the benchmark's contract (no GPU needed):
  - more than one GPU is refused with a message and exit status 2, before
    anything touches a device;
  - the committed decoder counter summaries match the current decoder
    source and each workload's layout, so the bench line's measured HBM
    traffic is not stale;
  - the workload sizes the bench keeps (to pick a layout without generating
    weights) are the generators' sizes."""
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
    traffic = bench.profiled_traffic(workload, bench.layout_for(bench.WORKLOAD_WEIGHTS[workload]))
    assert traffic is not None, f"profiles/ has no counter summary for {workload} with this decoder"
    assert traffic > 0


def test_workload_weights_match_generators():
    import bench
    from paper_2504_11651_amd import synth
    assert bench.WORKLOAD_WEIGHTS["llama3_8b_block"] == sum(r * c for _, r, c in synth.LLAMA3_8B_BLOCK)
    assert bench.WORKLOAD_WEIGHTS["llama31_70b_block"] == sum(r * c for _, r, c in
                                                              synth.LLAMA31_70B_BLOCK)
    assert bench.WORKLOAD_WEIGHTS["matrix_4096"] == bench.workload("matrix_4096").size
    import inspect
    assert bench.WORKLOAD_WEIGHTS["heavy_tailed_block"] == \
        inspect.signature(synth.heavy_tailed_block).parameters["n"].default


def test_default_layout_by_size():
    """Large streams take 128-chunk blocks, shorter ones 64-chunk blocks."""
    from paper_2504_11651_amd import codec
    big = 192 << 20
    for n, T in ((0, 64), (1, 64), (big - 1, 64), (big, 128), (2 ** 32 - 1, 128)):
        lay = codec.default_layout(n)
        assert (lay.bytes_per_thread, lay.threads_per_block, lay.lut_bits) == (8, T, 11)


def test_decoder_hash_follows_code_not_comments():
    import bench
    a = 'int f(int x) { return x + 1; }  // one\n/* block\n comment */\nconst char *s = "//";\n'
    b = '// header\nint f(int x)  {\n  return x + 1;  /* inline */ }\nconst char *s = "//";\n'
    c = 'int f(int x) { return x + 2; }\nconst char *s = "//";\n'
    assert bench.code_only(a) == bench.code_only(b)
    assert bench.code_only(a) != bench.code_only(c)
    assert '"//"' in bench.code_only(a)  # string literals are code
