"""Parity at full workload sizes, in the launch configuration bench.py times.

The expected layout comes from the oracle (offsets from the tensor sizes) and
the expected bytes from the input generator, tensor by tensor; nothing is
taken from the library's own files or index."""

import os
import sys

import numpy as np
import pytest

import oracle
from paper_2401_14351_amd import binding, synth

pytestmark = pytest.mark.gpu

SENTINEL = 0x5A


def say(*a):
    print("[gpu-full]", *a, flush=True)


@pytest.fixture(scope="module")
def torch_cuda():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.lib()
    return torch


def converted(spec):
    """The workload converted once per box (shared with bench.py)."""
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import bench

    d = os.path.join(os.environ.get("SLLM_BENCH_DIR", "/tmp/sllm_bench"), spec.name)
    bench.ensure_checkpoint(spec, d)
    return d


def check_tensors(torch, spec, buf, offsets, indices=None):
    """Every listed tensor's device bytes equal the generator's bytes."""
    idx = range(len(spec.tensors)) if indices is None else indices
    for i, t, want in synth.iter_tensors(spec, indices=idx):
        o = offsets[i]
        got = buf[o:o + t.nbytes].cpu().numpy()
        if not np.array_equal(got, want):
            bad = np.nonzero(got != want)[0]
            raise AssertionError(f"{t.name}: {bad.size} bytes differ, first at {bad[:4].tolist()}")


def check_zero_gaps(torch, buf, offsets, sizes, total):
    """Every byte outside the tensors' data (padding) is zero."""
    ends = [o + s for o, s in zip(offsets, sizes)]
    starts = list(offsets[1:]) + [total]
    for a, b in zip(ends, starts):
        if b > a and int(buf[a:b].to(torch.int32).abs().sum()) != 0:
            raise AssertionError(f"padding [{a}, {b}) is not zero")


def test_llama2_7b_cached_k1(torch_cuda):
    """13.48 GB, 291 tensors: cached 16 MiB chunks, one K1 launch (the bench step)."""
    torch = torch_cuda
    spec = synth.llama2("7b")
    d = converted(spec)
    offsets, T = oracle.plan_layout([t.nbytes for t in spec.tensors], spec.alignment)
    say("7b: T", T)
    with binding.Pool(spec.chunk_size, -(-T // spec.chunk_size)) as pool:
        pool.cache(d, io_threads=8)
        with binding.Checkpoint(d, pool=pool) as ck:
            assert ck.total_bytes == T
            assert [t.offset for t in ck.tensors()] == offsets
            buf = torch.full((T + 4096,), SENTINEL, dtype=torch.uint8, device="cuda:0")
            s = torch.cuda.current_stream()
            ck.load_into(buf, s)
            s.synchronize()
            assert ck.stats()["n_launches"] == 1
        pool.evict(d)
    assert bool((buf[T:] == SENTINEL).all())
    check_zero_gaps(torch, buf, offsets, [t.nbytes for t in spec.tensors], T)
    check_tensors(torch, spec, buf, offsets)
    say("7b: all tensors match")


def test_stress_8g_file_and_device_layout(torch_cuda):
    """The 8 GiB prefix of the stress workload (mixed dtypes, 4 KiB file
    alignment): cached K1 load, then the A2 = 256 layout through K1-scatter
    and through the HBM repack (K2)."""
    torch = torch_cuda
    spec = synth.config("stress-8g")
    d = converted(spec)
    sizes = [t.nbytes for t in spec.tensors]
    offsets, T = oracle.plan_layout(sizes, spec.alignment)
    d2, T2 = oracle.plan_layout(sizes, 256)
    say("stress-8g: n", len(sizes), "T", T, "T2", T2)
    with binding.Pool(spec.chunk_size, -(-T // spec.chunk_size)) as pool:
        pool.cache(d, io_threads=8)
        with binding.Checkpoint(d, pool=pool) as ck:
            buf = torch.empty(T, dtype=torch.uint8, device="cuda:0")
            ck.load_into(buf)
            torch.cuda.synchronize()
        check_zero_gaps(torch, buf, offsets, sizes, T)
        check_tensors(torch, spec, buf, offsets)
        with binding.Checkpoint(d, pool=pool, dev_alignment=256) as ck:
            assert ck.total_bytes == T2
            assert [t.offset for t in ck.tensors()] == d2
            direct = torch.full((T2 + 4096,), SENTINEL, dtype=torch.uint8, device="cuda:0")
            ck.load_into(direct)
            repacked = torch.full((T2 + 4096,), SENTINEL, dtype=torch.uint8, device="cuda:0")
            ck.repack(buf, repacked)
            torch.cuda.synchronize()
        pool.evict(d)
    for out in (direct, repacked):
        assert bool((out[T2:] == SENTINEL).all())
    assert torch.equal(direct, repacked)
    check_zero_gaps(torch, direct, d2, sizes, T2)
    check_tensors(torch, spec, direct, d2)
    say("stress-8g: file and device layouts match")
