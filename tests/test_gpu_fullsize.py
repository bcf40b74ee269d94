"""Parity at full workload sizes, in the launch configuration bench.py times,
over every byte of every image.

The expected layout comes from the oracle (offsets from the tensor sizes)
and the expected bytes from the input generator: each tensor's digest is
taken from the generator's bytes while the checkpoint is converted, and
``verify.check_image`` compares the digest of every tensor's device bytes at
the oracle's offset with it, and every other byte of the image with zero.
Nothing is taken from the library's own files or index.  A sentinel after
each image checks that no byte past its end is written."""

import os
import shutil
import sys

import pytest

import oracle
from paper_2401_14351_amd import binding, synth, verify

pytestmark = pytest.mark.gpu

SENTINEL = 0x5A
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def say(*a):
    print("[gpu-full]", *a, flush=True)


@pytest.fixture(scope="module")
def torch_cuda():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.lib()
    return torch


def converted(spec, d=None):
    """The workload converted once per machine (shared with bench.py) and
    the digests of its tensors' generator bytes."""
    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    import bench

    d = d or bench.checkpoint_dir(spec)
    say(f"{spec.name}: converted checkpoint in {d}")
    return d, bench.ensure_checkpoint(spec, d)


def shm_dir(name):
    if not os.path.isdir("/dev/shm"):
        pytest.skip("no /dev/shm")
    return os.path.join("/dev/shm/sllm_test", name)


def fresh(torch, nbytes):
    """A device buffer with a sentinel tail past the image."""
    return torch.full((nbytes + 4096,), SENTINEL, dtype=torch.uint8, device="cuda:0")


def check(torch, buf, spec, offsets, total, digests, what):
    assert bool((buf[total:] == SENTINEL).all()), f"{what}: bytes past the image were written"
    got = verify.check_image(torch, buf, spec, offsets, total, digests)
    say(f"{what}: every byte matches ({got['tensors']} tensors, {got['bytes']} bytes, "
        f"{got['padding_bytes']} padding bytes)")


def release(torch):
    import gc

    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def test_llama2_7b_cached(torch_cuda):
    """13.48 GB, 291 tensors, cached 16 MiB chunks: one K1 launch (the bench
    step) and the copy engines' merged copies, in the file layout; K1-scatter
    and the copy engines + K2 into A2 = 4 KiB; the K2 repack of the loaded
    image.  Every 7B tensor is a multiple of 8 KiB, so the 4 KiB layout
    equals the file layout: those three are identity relocations (K2 copies
    in place of moving bytes)."""
    torch = torch_cuda
    spec = synth.llama2("7b")
    d, digests = converted(spec)
    sizes = [t.nbytes for t in spec.tensors]
    offsets, T = oracle.plan_layout(sizes, spec.alignment)
    d2, T2 = oracle.plan_layout(sizes, 4096)
    assert d2 == offsets and T2 == T  # the identity noted above
    say("7b: T", T)
    s = torch.cuda.current_stream()
    with binding.Pool(spec.chunk_size, -(-T // spec.chunk_size)) as pool:
        pool.cache(d, io_threads=8)
        buf = fresh(torch, T)
        with binding.Checkpoint(d, pool=pool) as ck:
            assert ck.total_bytes == T and [t.offset for t in ck.tensors()] == offsets
            ck.load_into(buf, s)
            s.synchronize()
            assert ck.stats()["n_launches"] == 1
        check(torch, buf, spec, offsets, T, digests, "7b K1")
        out = fresh(torch, T)
        with binding.Checkpoint(d, pool=pool, engine="sdma") as ck:
            ck.load_into(out, s)
            s.synchronize()
            st = ck.stats()
            assert st["from_cache"] == 1 and st["n_launches"] > 1
        check(torch, out, spec, offsets, T, digests, "7b SDMA (merged copies)")
        for engine in ("kernel", "sdma"):
            out.fill_(SENTINEL)
            with binding.Checkpoint(d, pool=pool, engine=engine, dev_alignment=4096) as ck:
                ck.load_into(out, s)
                s.synchronize()
            check(torch, out, spec, d2, T2, digests, f"7b A2=4096 by {engine} (identity layout)")
        out.fill_(SENTINEL)
        with binding.Checkpoint(d, pool=pool, dev_alignment=4096) as ck:
            ck.repack(buf, out, s)
            s.synchronize()
        check(torch, out, spec, d2, T2, digests, "7b K2 repack to A2=4096 (identity copy)")
        pool.evict(d)
    del buf, out
    release(torch)


def test_stress_8g_every_path(torch_cuda):
    """The 8 GiB prefix of the stress workload (1,520 tensors, mixed dtypes,
    4 KiB file alignment, padding after most tensors): cached K1 and copy
    engine loads in the file layout; into A2 = 256 by K1-scatter, by the copy
    engines + K2 (merged runs through HBM staging), and by the K2 repack of
    the file-layout image (a real relocation: T2 != T, unaligned shifts)."""
    torch = torch_cuda
    spec = synth.config("stress-8g")
    d, digests = converted(spec)
    sizes = [t.nbytes for t in spec.tensors]
    offsets, T = oracle.plan_layout(sizes, spec.alignment)
    d2, T2 = oracle.plan_layout(sizes, 256)
    assert T2 != T
    say("stress-8g: n", len(sizes), "T", T, "T2", T2)
    s = torch.cuda.current_stream()
    with binding.Pool(spec.chunk_size, -(-T // spec.chunk_size)) as pool:
        pool.cache(d, io_threads=8)
        buf = fresh(torch, T)
        out = fresh(torch, T2)
        for engine in ("kernel", "sdma"):
            buf.fill_(SENTINEL)
            with binding.Checkpoint(d, pool=pool, engine=engine) as ck:
                assert [t.offset for t in ck.tensors()] == offsets
                ck.load_into(buf, s)
                s.synchronize()
            check(torch, buf, spec, offsets, T, digests, f"stress-8g file layout by {engine}")
            out.fill_(SENTINEL)
            with binding.Checkpoint(d, pool=pool, engine=engine, dev_alignment=256) as ck:
                assert ck.total_bytes == T2 and [t.offset for t in ck.tensors()] == d2
                ck.load_into(out, s)
                s.synchronize()
            check(torch, out, spec, d2, T2, digests, f"stress-8g A2=256 by {engine}")
        out.fill_(SENTINEL)
        with binding.Checkpoint(d, pool=pool, dev_alignment=256) as ck:
            ck.repack(buf, out, s)
            s.synchronize()
        check(torch, out, spec, d2, T2, digests, "stress-8g K2 repack to A2=256")
        pool.evict(d)
    del buf, out
    release(torch)


def test_tensor_over_4gib(torch_cuda):
    """One tensor of 4,295,229,443 bytes packed densely between odd-sized
    ones: in-tensor offsets past 2^32 in every path.  At A2 = 256 its source
    shift is -10 bytes, so K1-scatter and K2 move it through the byte
    funnel.  Cached by both engines in the file layout and into A2 = 256,
    K2's repack of the file-layout image, and a streamed K1-scatter load."""
    torch = torch_cuda
    spec = synth.config("huge-tensor")
    assert max(t.nbytes for t in spec.tensors) > 1 << 32
    d, digests = converted(spec)
    sizes = [t.nbytes for t in spec.tensors]
    offsets, T = oracle.plan_layout(sizes, spec.alignment)
    d2, T2 = oracle.plan_layout(sizes, 256)
    assert (offsets[1] - d2[1]) % 16 != 0
    say("huge-tensor: T", T, "T2", T2)
    s = torch.cuda.current_stream()
    buf = fresh(torch, T)
    out = fresh(torch, T2)
    with binding.Pool(spec.chunk_size, -(-T // spec.chunk_size)) as pool:
        pool.cache(d, io_threads=8)
        for engine in ("kernel", "sdma"):
            buf.fill_(SENTINEL)
            with binding.Checkpoint(d, pool=pool, engine=engine) as ck:
                ck.load_into(buf, s)
                s.synchronize()
            check(torch, buf, spec, offsets, T, digests, f"huge-tensor file layout by {engine}")
            out.fill_(SENTINEL)
            with binding.Checkpoint(d, pool=pool, engine=engine, dev_alignment=256) as ck:
                assert [t.offset for t in ck.tensors()] == d2
                ck.load_into(out, s)
                s.synchronize()
            check(torch, out, spec, d2, T2, digests, f"huge-tensor A2=256 by {engine}")
        out.fill_(SENTINEL)
        with binding.Checkpoint(d, pool=pool, dev_alignment=256) as ck:
            ck.repack(buf, out, s)
            s.synchronize()
        check(torch, out, spec, d2, T2, digests, "huge-tensor K2 repack to A2=256")
        pool.evict(d)
    out.fill_(SENTINEL)
    with binding.Checkpoint(d, dev_alignment=256, io_threads=8, ring_slots=16) as ck:
        ck.load_into(out, s)
        s.synchronize()
    check(torch, out, spec, d2, T2, digests, "huge-tensor streamed K1-scatter to A2=256")
    del buf, out
    release(torch)


@pytest.mark.parametrize("C_mib", [4, 16, 64])
def test_llama2_13b_chunk_sizes(torch_cuda, C_mib):
    """26.0 GB, 363 tensors (a 2 KiB file tail), the chunk-size sweep: the
    partition cached in 4 / 16 / 64 MiB pool chunks and moved by one K1
    launch, and by the copy engines at the workload's 16 MiB."""
    torch = torch_cuda
    spec = synth.llama2("13b")
    d, digests = converted(spec)
    sizes = [t.nbytes for t in spec.tensors]
    offsets, T = oracle.plan_layout(sizes, spec.alignment)
    C = C_mib << 20
    say("13b: C", C, "T", T)
    engines = ("kernel", "sdma") if C_mib == 16 else ("kernel",)
    with binding.Pool(C, -(-T // C)) as pool:
        pool.cache(d, io_threads=8)
        buf = fresh(torch, T)
        for engine in engines:
            buf.fill_(SENTINEL)
            with binding.Checkpoint(d, pool=pool, engine=engine) as ck:
                assert ck.total_bytes == T and [t.offset for t in ck.tensors()] == offsets
                ck.load_into(buf)
                torch.cuda.synchronize()
                assert ck.stats()["from_cache"] == 1
            check(torch, buf, spec, offsets, T, digests, f"13b C={C_mib} MiB by {engine}")
        pool.evict(d)
    del buf
    release(torch)


def test_llama2_13b_ring_4mib(torch_cuda):
    """The 13B partition streamed from the file through a 1 GiB ring of
    4 MiB slots: batched K1 launches, then the copy engines' runs of
    consecutive slots."""
    torch = torch_cuda
    spec = synth.llama2("13b")
    d, digests = converted(spec)
    sizes = [t.nbytes for t in spec.tensors]
    offsets, T = oracle.plan_layout(sizes, spec.alignment)
    C = 4 << 20
    buf = fresh(torch, T)
    with binding.Pool(C, 256) as pool:
        for engine in ("kernel", "sdma"):
            buf.fill_(SENTINEL)
            with binding.Checkpoint(d, pool=pool, chunk_size=C, io_threads=8, ring_slots=256, engine=engine) as ck:
                ck.load_into(buf)
                torch.cuda.synchronize()
                st = ck.stats()
                # batched gathers; copies of runs of slots (runs may be single chunks)
                assert st["from_cache"] == 0 and st["n_launches"] <= st["n_chunks"]
                assert engine == "sdma" or st["n_launches"] < st["n_chunks"]
            check(torch, buf, spec, offsets, T, digests, f"13b ring of 4 MiB slots by {engine}")
    del buf
    release(torch)


def test_llama2_70b_ring_from_shm(torch_cuda):
    """137.95 GB, 723 tensors (larger than the free space of a typical local
    disk, so the file sits in /dev/shm): streamed through a 16 x 64 MiB ring
    by 16 readers, as the bench runs it, by K1 and by the copy engines."""
    torch = torch_cuda
    spec = synth.llama2("70b")
    d = shm_dir(spec.name)
    buf = None
    try:
        _, digests = converted(spec, d)
        sizes = [t.nbytes for t in spec.tensors]
        offsets, T = oracle.plan_layout(sizes, spec.alignment)
        say("70b: T", T)
        buf = fresh(torch, T)
        with binding.Pool(spec.chunk_size, 16) as pool:
            for engine in ("kernel", "sdma"):
                buf.fill_(SENTINEL)
                with binding.Checkpoint(d, pool=pool, io_threads=16, ring_slots=16, engine=engine) as ck:
                    assert ck.total_bytes == T
                    ck.load_into(buf)
                    torch.cuda.synchronize()
                check(torch, buf, spec, offsets, T, digests, f"70b ring by {engine}")
    finally:
        shutil.rmtree(d, ignore_errors=True)
        buf = None  # drop the image before handing its memory back
        release(torch)


def test_stress_full_ring_from_shm(torch_cuda):
    """The full stress workload (20,000 tensors, all four dtypes, sizes
    log-uniform over [256 B, 64 MiB], 4 KiB alignment, 1 MiB chunks: about
    108 GB, in /dev/shm) streamed through a 1 GiB ring by K1, repacked in HBM
    into A2 = 256 (about 13 million tiles, several K2 launches), and
    streamed again by the copy engines."""
    torch = torch_cuda
    spec = synth.config("stress")
    d = shm_dir(spec.name)
    buf = out = None
    try:
        _, digests = converted(spec, d)
        sizes = [t.nbytes for t in spec.tensors]
        offsets, T = oracle.plan_layout(sizes, spec.alignment)
        d2, T2 = oracle.plan_layout(sizes, 256)
        say("stress: n", len(sizes), "T", T, "T2", T2)
        buf = fresh(torch, T)
        with binding.Pool(spec.chunk_size, 1024) as pool:
            with binding.Checkpoint(d, pool=pool, io_threads=8, ring_slots=1024) as ck:
                assert ck.total_bytes == T and [t.offset for t in ck.tensors()] == offsets
                ck.load_into(buf)
                torch.cuda.synchronize()
            check(torch, buf, spec, offsets, T, digests, "stress ring by kernel")
            out = fresh(torch, T2)
            with binding.Checkpoint(d, dev_alignment=256) as ck:
                assert ck.total_bytes == T2 and [t.offset for t in ck.tensors()] == d2
                ck.repack(buf, out)
                torch.cuda.synchronize()
            check(torch, out, spec, d2, T2, digests, "stress K2 repack to A2=256")
            out = None
            release(torch)
            buf.fill_(SENTINEL)
            with binding.Checkpoint(d, pool=pool, io_threads=8, ring_slots=1024, engine="sdma") as ck:
                ck.load_into(buf)
                torch.cuda.synchronize()
            check(torch, buf, spec, offsets, T, digests, "stress ring by sdma")
    finally:
        shutil.rmtree(d, ignore_errors=True)
        buf = out = None  # drop the images before handing their memory back
        release(torch)
