"""The C ABI from a plain C program (tests/native/c_load.c): no Python and
no torch in the process that loads.  It opens a converted checkpoint, loads
it into hipMalloc'd memory with both engines, cached and streamed, in the
file layout and at A2 = 256, and compares every byte with images the oracle
wrote."""

import os
import shutil
import subprocess

import pytest

import oracle
from paper_2401_14351_amd import binding, build, synth

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_c_program_loads_checkpoint(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    binding.lib()  # fail loudly if the library is missing
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    exe = tmp_path / "c_load"
    subprocess.run(["gcc", "-std=c11", "-O1", f"-I{rocm}/include", f"-I{ROOT}/include",
                    os.path.join(ROOT, "tests", "native", "c_load.c"), "-o", str(exe),
                    f"-L{build.PKG}", "-lsllm", f"-Wl,-rpath,{build.PKG}", f"-L{rocm}/lib", "-lamdhip64",
                    f"-Wl,-rpath,{rocm}/lib"], check=True)
    spec = synth.stress(n=300, max_bytes=1 << 16, seed=11)
    tensors = [(t.name, t.dtype, t.shape, d) for t, d in zip(spec.tensors, synth.materialize(spec))]
    A, C = 16, 64 << 10
    d = str(tmp_path / "ckpt")
    os.makedirs(d)
    binding.convert(iter(tensors), d, A, C)
    index = oracle.make_index(tensors, A, C)
    image = bytes(oracle.partition_bytes(tensors, A)[:index.total_bytes])
    (tmp_path / "want1").write_bytes(image)
    (tmp_path / "want2").write_bytes(bytes(oracle.repack(image, index, 256)))
    print("[c-abi] running", exe, "T", index.total_bytes, flush=True)
    r = subprocess.run([str(exe), d, str(tmp_path / "want1"), str(tmp_path / "want2"), str(C)],
                       capture_output=True, text=True, timeout=120)
    print(r.stdout, flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip().endswith("ok"), r.stdout
