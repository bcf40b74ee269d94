"""Host-side format code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): random checkpoints through the writer and a mutation fuzz of the
index decoder (tests/native/fuzz_format.cpp)."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2401_14351_amd", "csrc")
HOST_SOURCES = ["common.cpp", "format.cpp", "writer.cpp", "io.cpp"]


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_format_code_under_sanitizers(tmp_path):
    exe = tmp_path / "fuzz_format"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", f"-I{ROOT}/include", f"-I{CSRC}",
           os.path.join(ROOT, "tests", "native", "fuzz_format.cpp"),
           *[os.path.join(CSRC, s) for s in HOST_SOURCES], "-o", str(exe), "-lpthread"]
    subprocess.run(cmd, check=True)
    work = tmp_path / "ck"
    work.mkdir()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe), str(work), "40000"], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok "), r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr
