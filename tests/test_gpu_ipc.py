"""Handoff from the loading process to another process (Sec. 4.1): the
consumer maps the buffer through its IPC handle, waits on the handoff event
on its own stream, and views every tensor at base + offset."""

import os
import subprocess
import sys

import pytest

from paper_2401_14351_amd import binding, synth

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def torch_cuda():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.lib()
    return torch


def test_ipc_handoff_opt125m(torch_cuda, tmp_path):
    torch = torch_cuda
    spec = synth.opt_125m()
    d = str(tmp_path / "opt")
    binding.convert(((t.name, t.dtype, t.shape, b) for _, t, b in synth.iter_tensors(spec)), d,
                    spec.alignment, spec.chunk_size)
    with binding.Pool(spec.chunk_size, 16) as pool:
        pool.cache(d)
        with binding.Checkpoint(d, pool=pool) as ck:
            # the shared buffer must be its own (small) allocation, not a block
            # carved from a large segment the caching allocator kept around
            torch.cuda.synchronize()
            torch.cuda.empty_cache()
            buf = torch.empty(ck.total_bytes, dtype=torch.uint8, device="cuda:0")
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                torch.cuda._sleep(50_000_000)  # the load is still queued when the consumer starts
            ck.load_into(buf, s)
            ex = binding.Export(buf, s)
            print("[gpu-ipc] starting the consumer; device-side event:", bool(ex.desc.flags & 1), flush=True)
            r = subprocess.run([sys.executable, os.path.join(HERE, "ipc_consumer.py"), d, ex.desc_bytes.hex(),
                                "opt-125m"], capture_output=True, text=True, timeout=240)
            print(r.stdout, r.stderr[-2000:], flush=True)
            assert r.returncode == 0 and "ipc ok 196 tensors" in r.stdout
            s.synchronize()
            ex.close()
        pool.evict(d)


def test_export_refuses_large_allocations(torch_cuda):
    torch = torch_cuda
    big = torch.empty(3 << 30, dtype=torch.uint8, device="cuda:0")
    with pytest.raises(binding.SllmError) as ei:
        binding.Export(big[:1024])
    assert ei.value.code == -1 and "larger" in ei.value.message
    del big
