"""The host codec and the oracle under sanitizers (CPU only).

tests/sanitize/host_check.cpp cross-checks the library's host half
(df11_host.cpp, df11_tables.cpp: code book, encoder, metadata, tables,
validation) against the oracle on seeded inputs and layouts.  It is built
here twice with gcc/g++ (host code only, no GPU code): with
AddressSanitizer + UndefinedBehaviorSanitizer, and with ThreadSanitizer,
which watches the multi-threaded histogram and encoder on inputs large
enough to use several threads.  Any report or disagreement fails the test."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2504_11651_amd", "csrc")
DRIVER = os.path.join(ROOT, "tests", "sanitize", "host_check.cpp")
ORACLE = os.path.join(ROOT, "oracle", "df11_oracle.c")
INC = ["-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
       "-I", CSRC]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None,
                                reason="needs gcc/g++")


def _build(tmp, flags):
    objs = []
    for src in ("df11_host.cpp", "df11_tables.cpp"):
        o = os.path.join(tmp, src + ".o")
        subprocess.run(["g++", "-std=c++17", "-O1", "-g", *flags, *INC, "-c",
                        os.path.join(CSRC, src), "-o", o], check=True)
        objs.append(o)
    o = os.path.join(tmp, "oracle.o")
    subprocess.run(["gcc", "-std=c99", "-O1", "-g", *flags, "-c", ORACLE, "-o", o], check=True)
    exe = os.path.join(tmp, "host_check")
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", *flags, *INC, DRIVER, *objs, o,
                    "-lpthread", "-o", exe], check=True)
    return exe


def _run(exe, env_key, env_val):
    env = dict(os.environ, **{env_key: env_val})
    r = subprocess.run([exe, "large"], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "0 failures" in r.stdout


def test_host_codec_and_oracle_under_asan_ubsan(tmp_path):
    exe = _build(str(tmp_path), ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                                 "-fno-omit-frame-pointer"])
    _run(exe, "ASAN_OPTIONS", "detect_leaks=1:abort_on_error=0")


def test_threaded_encoder_under_tsan(tmp_path):
    exe = _build(str(tmp_path), ["-fsanitize=thread"])
    _run(exe, "TSAN_OPTIONS", "halt_on_error=1")
