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
    """The workload converted once per machine (shared with bench.py)."""
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
        # the HBM repack the bench times: A2 = 4 KiB, one K2 launch over the image
        sizes = [t.nbytes for t in spec.tensors]
        d2, T2 = oracle.plan_layout(sizes, 4096)
        with binding.Checkpoint(d, pool=pool, dev_alignment=4096) as ck:
            assert ck.total_bytes == T2 and [t.offset for t in ck.tensors()] == d2
            out = torch.full((T2 + 4096,), SENTINEL, dtype=torch.uint8, device="cuda:0")
            ck.repack(buf, out, s)
            s.synchronize()
        pool.evict(d)
    assert bool((buf[T:] == SENTINEL).all())
    check_zero_gaps(torch, buf, offsets, sizes, T)
    check_tensors(torch, spec, buf, offsets)
    say("7b: all tensors match")
    # every tensor of this model is a multiple of 4 KiB, so the 4 KiB layout
    # is the file layout: the repacked image equals the verified load
    assert d2 == offsets and T2 == T
    assert bool((out[T2:] == SENTINEL).all())
    assert torch.equal(out[:T2], buf[:T])
    say("7b: HBM repack matches")


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


def sample(n, k, seed):
    """k tensor indices drawn without replacement, plus the first and last."""
    rng = np.random.default_rng(seed)
    return sorted({0, n - 1, *rng.choice(n, size=min(k, n), replace=False).tolist()})


def check_sampled_gaps(torch, buf, offsets, sizes, total, indices):
    """The padding after each sampled tensor is zero."""
    for i in indices:
        a = offsets[i] + sizes[i]
        b = offsets[i + 1] if i + 1 < len(offsets) else total
        if b > a and int(buf[a:b].to(torch.int32).abs().sum()) != 0:
            raise AssertionError(f"padding [{a}, {b}) after tensor {i} is not zero")


def shm_dir(name):
    base = "/dev/shm/sllm_test"
    if not os.path.isdir("/dev/shm"):
        pytest.skip("no /dev/shm")
    return os.path.join(base, name)


def converted_at(spec, d):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import bench

    bench.ensure_checkpoint(spec, d)
    return d


@pytest.mark.parametrize("C_mib", [4, 16, 64])
def test_llama2_13b_chunk_sizes(torch_cuda, C_mib):
    """26.0 GB, 363 tensors, the chunk-size sweep: the partition cached in
    4 / 16 / 64 MiB pool chunks and moved by one K1 launch; every tensor
    against the generator at 16 MiB, sampled tensors at 4 and 64 MiB,
    nothing written past T."""
    torch = torch_cuda
    spec = synth.llama2("13b")
    d = converted(spec)
    sizes = [t.nbytes for t in spec.tensors]
    offsets, T = oracle.plan_layout(sizes, spec.alignment)
    C = C_mib << 20
    say("13b: C", C, "T", T)
    with binding.Pool(C, -(-T // C)) as pool:
        pool.cache(d, io_threads=8)
        with binding.Checkpoint(d, pool=pool) as ck:
            assert ck.total_bytes == T and [t.offset for t in ck.tensors()] == offsets
            buf = torch.full((T + 4096,), SENTINEL, dtype=torch.uint8, device="cuda:0")
            ck.load_into(buf)
            torch.cuda.synchronize()
            assert ck.stats()["from_cache"] == 1
        pool.evict(d)
    assert bool((buf[T:] == SENTINEL).all())
    if C_mib == 16:  # the workload's own chunk size: every tensor and every padding byte
        check_zero_gaps(torch, buf, offsets, sizes, T)
        check_tensors(torch, spec, buf, offsets)
        say("13b: all tensors match")
    else:
        idx = sample(len(sizes), 24, seed=C_mib)
        check_sampled_gaps(torch, buf, offsets, sizes, T, idx)
        check_tensors(torch, spec, buf, offsets, indices=idx)
        say("13b: sampled tensors match")
    del buf
    torch.cuda.empty_cache()


def test_llama2_13b_ring_4mib(torch_cuda):
    """The 13B partition streamed from the file through a 1 GiB ring of
    4 MiB slots (batched K1 launches); sampled tensors."""
    torch = torch_cuda
    spec = synth.llama2("13b")
    d = converted(spec)
    sizes = [t.nbytes for t in spec.tensors]
    offsets, T = oracle.plan_layout(sizes, spec.alignment)
    C = 4 << 20
    with binding.Pool(C, 256) as pool:
        with binding.Checkpoint(d, pool=pool, chunk_size=C, io_threads=8, ring_slots=256) as ck:
            buf = torch.full((T + 4096,), SENTINEL, dtype=torch.uint8, device="cuda:0")
            ck.load_into(buf)
            torch.cuda.synchronize()
            st = ck.stats()
            assert st["from_cache"] == 0 and st["n_launches"] < st["n_chunks"]
    assert bool((buf[T:] == SENTINEL).all())
    idx = sample(len(sizes), 24, seed=44)
    check_sampled_gaps(torch, buf, offsets, sizes, T, idx)
    check_tensors(torch, spec, buf, offsets, indices=idx)
    del buf
    torch.cuda.empty_cache()
    say("13b ring: sampled tensors match")


def test_llama2_70b_ring_from_shm(torch_cuda):
    """137.95 GB, 723 tensors (larger than the free space of a typical local
    disk, so the file sits in /dev/shm): streamed through a 16 x 64 MiB ring by 16 readers, as
    the bench runs it; sampled tensors."""
    torch = torch_cuda
    spec = synth.llama2("70b")
    d = shm_dir(spec.name)
    buf = None
    try:
        converted_at(spec, d)
        sizes = [t.nbytes for t in spec.tensors]
        offsets, T = oracle.plan_layout(sizes, spec.alignment)
        say("70b: T", T)
        with binding.Pool(spec.chunk_size, 16) as pool:
            with binding.Checkpoint(d, pool=pool, io_threads=16, ring_slots=16) as ck:
                assert ck.total_bytes == T
                buf = torch.full((T + 4096,), SENTINEL, dtype=torch.uint8, device="cuda:0")
                ck.load_into(buf)
                torch.cuda.synchronize()
        assert bool((buf[T:] == SENTINEL).all())
        idx = sample(len(sizes), 16, seed=70)
        check_sampled_gaps(torch, buf, offsets, sizes, T, idx)
        check_tensors(torch, spec, buf, offsets, indices=idx)
        say("70b: sampled tensors match")
    finally:
        import shutil

        shutil.rmtree(d, ignore_errors=True)
        buf = None  # drop the image before handing its memory back
        torch.cuda.empty_cache()


def test_stress_full_ring_from_shm(torch_cuda):
    """The full stress workload (20,000 tensors, all four dtypes, sizes
    log-uniform over [256 B, 64 MiB], 4 KiB alignment, 1 MiB chunks: about
    108 GB, in /dev/shm) streamed through a 1 GiB ring, then repacked in HBM
    into A2 = 256; sampled tensors and the padding after them, in both
    images."""
    torch = torch_cuda
    spec = synth.config("stress")
    d = shm_dir(spec.name)
    buf = out = None
    try:
        converted_at(spec, d)
        sizes = [t.nbytes for t in spec.tensors]
        offsets, T = oracle.plan_layout(sizes, spec.alignment)
        say("stress: n", len(sizes), "T", T)
        with binding.Pool(spec.chunk_size, 1024) as pool:
            with binding.Checkpoint(d, pool=pool, io_threads=8, ring_slots=1024) as ck:
                assert ck.total_bytes == T and [t.offset for t in ck.tensors()] == offsets
                buf = torch.full((T + 4096,), SENTINEL, dtype=torch.uint8, device="cuda:0")
                ck.load_into(buf)
                torch.cuda.synchronize()
        assert bool((buf[T:] == SENTINEL).all())
        idx = sample(len(sizes), 64, seed=5)
        check_sampled_gaps(torch, buf, offsets, sizes, T, idx)
        check_tensors(torch, spec, buf, offsets, indices=idx)
        say("stress: sampled tensors match")
        # the HBM repack of the whole image into A2 = 256 (about 13 million
        # tiles, several K2 launches); sampled tensors at their device offsets
        d2, T2 = oracle.plan_layout(sizes, 256)
        with binding.Checkpoint(d, dev_alignment=256) as ck:
            assert ck.total_bytes == T2 and [t.offset for t in ck.tensors()] == d2
            out = torch.full((T2 + 4096,), SENTINEL, dtype=torch.uint8, device="cuda:0")
            ck.repack(buf, out)
            torch.cuda.synchronize()
        buf = None
        torch.cuda.empty_cache()
        assert bool((out[T2:] == SENTINEL).all())
        check_sampled_gaps(torch, out, d2, sizes, T2, idx)
        check_tensors(torch, spec, out, d2, indices=idx)
        out = None
        say("stress: repacked sampled tensors match")
    finally:
        import shutil

        shutil.rmtree(d, ignore_errors=True)
        buf = out = None  # drop the images before handing their memory back
        torch.cuda.empty_cache()
