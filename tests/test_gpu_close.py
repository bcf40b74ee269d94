"""sllm_close waits for the handle's device work, also for work that ran on
the caller's stream alone: a load from cached chunks by the kernel engine
(one launch on that stream) and a repack.  Without that wait the pool chunks
a load still reads could be evicted and refilled under it.  Each case
enqueues about 0.5 GB of work, closes the handle at once and checks that the
stream is then idle; the cached case then evicts the checkpoint, caches
another one into the same chunks and compares the first load's image with
the oracle's."""

import sys

import numpy as np
import pytest

import oracle
from paper_2401_14351_amd import binding, synth

pytestmark = pytest.mark.gpu

MiB = 1 << 20
C = 16 * MiB


def say(*a):
    print("[gpu-close]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.lib()
    return torch


def write(tmp_path, name, seed, A=4096):
    spec = synth.CheckpointSpec(name, seed, alignment=A, chunk_size=C,
                                tensors=[synth.TensorSpec(f"w{i}", "i8", (128 * MiB + 4096 * i + 7,), "bytes")
                                         for i in range(4)])
    tensors = [(t.name, t.dtype, t.shape, d) for t, d in zip(spec.tensors, synth.materialize(spec))]
    d = str(tmp_path / name)
    binding.convert(iter(tensors), d, A, C)
    return d, tensors


@pytest.mark.parametrize("A2", [0, 256])
def test_close_waits_for_a_cached_kernel_load(torch_cuda, tmp_path, A2):
    torch = torch_cuda
    d, tensors = write(tmp_path, "first", 41)
    d2, _ = write(tmp_path, "second", 42)
    index = oracle.make_index(tensors, 4096, C)
    image = bytes(oracle.partition_bytes(tensors, 4096)[:index.total_bytes])
    want = bytes(oracle.repack(image, index, A2)) if A2 else image
    n = -(-index.total_bytes // C)
    s = torch.cuda.Stream()
    with binding.Pool(C, n) as pool:
        pool.cache(d)
        buf = torch.empty(len(want), dtype=torch.uint8, device="cuda:0")
        ck = binding.Checkpoint(d, pool=pool, dev_alignment=A2)
        ck.load_into(buf, s)
        ck.close()
        idle = s.query()
        say("A2", A2, "stream idle after close:", idle)
        assert idle, "close returned while the load still ran on the caller's stream"
        pool.evict(d)
        pool.cache(d2)  # refills the chunks the load read
        torch.cuda.synchronize()
        got = buf.cpu().numpy().tobytes()
        if got != want:
            bad = np.nonzero(np.frombuffer(got, np.uint8) != np.frombuffer(want, np.uint8))[0]
            raise AssertionError(f"{bad.size} bytes differ, first at {bad[:4].tolist()}")
        pool.evict(d2)


def test_close_waits_for_a_repack(torch_cuda, tmp_path):
    torch = torch_cuda
    d, tensors = write(tmp_path, "third", 43, A=1)
    index = oracle.make_index(tensors, 1, C)
    image = bytes(oracle.partition_bytes(tensors, 1)[:index.total_bytes])
    want = bytes(oracle.repack(image, index, 4096))
    src = torch.frombuffer(bytearray(image), dtype=torch.uint8).to("cuda:0")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    out = torch.empty(len(want), dtype=torch.uint8, device="cuda:0")
    ck = binding.Checkpoint(d, dev_alignment=4096)
    for _ in range(8):  # about 8 GB of HBM traffic queued
        ck.repack(src, out, s)
    ck.close()
    idle = s.query()
    say("repack: stream idle after close:", idle)
    assert idle, "close returned while a repack still ran on the caller's stream"
    assert out.cpu().numpy().tobytes() == want
