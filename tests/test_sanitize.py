"""Host-side code under sanitizers (CPU only): the format code under
AddressSanitizer and UndefinedBehaviorSanitizer (random checkpoints through
the writer and a mutation fuzz of the index decoder,
tests/native/fuzz_format.cpp), and the streamed load's pipeline under
ThreadSanitizer and AddressSanitizer with a CPU stand-in for the GPU
(tests/native/ring_cpu.cpp)."""

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


PIPELINE_SOURCES = ["common.cpp", "pipeline.cpp", "workers.cpp"]
# clang's ThreadSanitizer: the one in GCC 11 does not intercept
# pthread_cond_clockwait, which std::condition_variable::wait_for uses, and
# then reports false races on every mutex it waits with.
CLANG = os.environ.get("SLLM_TSAN_CXX", "/opt/rocm/llvm/bin/clang++")


def _build_ring(cxx, flags, exe):
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", *flags, f"-I{ROOT}/include", f"-I{CSRC}",
           os.path.join(ROOT, "tests", "native", "ring_cpu.cpp"), *[os.path.join(CSRC, s) for s in PIPELINE_SOURCES],
           "-o", str(exe), "-lpthread"]
    subprocess.run(cmd, check=True)


def _run_ring(exe, env_extra):
    env = dict(os.environ, **env_extra)
    r = subprocess.run([str(exe), "300"], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip().startswith("ok "), r.stdout
    return r


@pytest.mark.skipif(not os.path.exists(CLANG), reason="clang++ with ThreadSanitizer not available")
def test_stream_pipeline_under_tsan(tmp_path):
    """300 random ring geometries, four loads each, with injected read and
    move errors: every image byte-exact, no slot refilled while a batch still
    holds it, no data race."""
    exe = tmp_path / "ring_tsan"
    _build_ring(CLANG, ["-fsanitize=thread"], exe)
    r = _run_ring(exe, {"TSAN_OPTIONS": "halt_on_error=1"})
    assert "ThreadSanitizer" not in r.stderr, r.stderr


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_stream_pipeline_under_asan(tmp_path):
    exe = tmp_path / "ring_asan"
    _build_ring("g++", ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined"], exe)
    r = _run_ring(exe, {"ASAN_OPTIONS": "detect_leaks=1:abort_on_error=1", "UBSAN_OPTIONS": "print_stacktrace=1"})
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_chunk_reader_under_sanitizers(tmp_path):
    """Buffered chunk reads by pread and through the file mapping with
    streaming stores: bytes equal the file's at every destination alignment,
    and a read past a truncation is an I/O error rather than a fault."""
    exe = tmp_path / "io_cpu"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", f"-I{ROOT}/include", f"-I{CSRC}",
           os.path.join(ROOT, "tests", "native", "io_cpu.cpp"),
           *[os.path.join(CSRC, s) for s in ("common.cpp", "io.cpp")], "-o", str(exe), "-lpthread"]
    subprocess.run(cmd, check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe), str(tmp_path)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip() == "ok", r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_kept_threads_across_fork(tmp_path):
    """A child of fork() starts threads of its own instead of handing tasks
    to the parent's idle ones, which do not exist in the child."""
    exe = tmp_path / "workers_fork"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", f"-I{ROOT}/include", f"-I{CSRC}",
           os.path.join(ROOT, "tests", "native", "workers_fork.cpp"),
           *[os.path.join(CSRC, s) for s in ("common.cpp", "workers.cpp")], "-o", str(exe), "-lpthread"]
    subprocess.run(cmd, check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
