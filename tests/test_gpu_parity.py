"""GPU parity: every byte a load writes (padding included) equals the CPU
oracle's image, for both engines, cached and streamed sources, the file
layout and device layouts (A2), and every chunk size on tiny checkpoints.

Expected bytes never come from the library: they are the oracle's partition
image (or its A2 repack) built from the generator's tensor bytes."""

import ctypes as C
import os
import sys

import numpy as np
import pytest

import oracle
from paper_2401_14351_amd import binding, synth

pytestmark = pytest.mark.gpu

SENTINEL = 0xA5


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.lib()  # fail loudly if the library is missing
    return torch


def tensors_of(spec):
    return [(t.name, t.dtype, t.shape, d) for t, d in zip(spec.tensors, synth.materialize(spec))]


def expected(tensors, A, A2=0):
    """The oracle's device image: the partition's first T bytes, or its A2 repack."""
    index = oracle.make_index(tensors, A, 1)
    H = oracle.partition_bytes(tensors, A)[:index.total_bytes]
    if A2:
        return bytes(oracle.repack(H, index, A2)), index
    return bytes(H), index


def run_load(torch, ck, expect_len, slack=64, stream=None):
    buf = torch.full((expect_len + slack,), SENTINEL, dtype=torch.uint8, device="cuda:0")
    s = stream or torch.cuda.current_stream()
    ck.load_into(buf, s)
    s.synchronize()
    host = buf.cpu().numpy()
    assert (host[expect_len:] == SENTINEL).all(), "bytes past the image were written"
    return host[:expect_len].tobytes()


def assert_same(got, want, what):
    if got != want:
        a = np.frombuffer(got, np.uint8)
        b = np.frombuffer(want, np.uint8)
        bad = np.nonzero(a != b)[0]
        raise AssertionError(f"{what}: {bad.size} bytes differ, first at {bad[:8].tolist()}")


# ---------------------------------------------------------------------------
# tiny checkpoints: every engine, source and layout
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("A", [1, 2, 16, 256, 4096])
@pytest.mark.parametrize("engine", ["kernel", "sdma"])
@pytest.mark.parametrize("A2", [0, 16, 256])
def test_tiny_streamed(torch_cuda, tmp_path, A, engine, A2):
    torch = torch_cuda
    for seed in range(4):
        spec = synth.tiny(seed, alignment=A, chunk_size=48)
        tensors = tensors_of(spec)
        binding.convert(iter(tensors), str(tmp_path / f"s{seed}"), A, spec.chunk_size)
        want, _ = expected(tensors, A, A2)
        say("tiny streamed", A, engine, A2, seed)
        with binding.Checkpoint(str(tmp_path / f"s{seed}"), engine=engine, dev_alignment=A2, ring_slots=3,
                                io_threads=2) as ck:
            assert ck.total_bytes == len(want)
            for rep in range(2):  # slots are reused across loads
                assert_same(run_load(torch, ck, len(want)), want, f"seed {seed} rep {rep}")


@pytest.mark.parametrize("A", [1, 16, 4096])
@pytest.mark.parametrize("engine", ["kernel", "sdma"])
@pytest.mark.parametrize("A2", [0, 32])
def test_tiny_cached(torch_cuda, tmp_path, A, engine, A2):
    torch = torch_cuda
    for seed, C_ in ((0, 64), (1, 4096), (2, 100), (5, 16)):
        spec = synth.tiny(seed, alignment=A)
        tensors = tensors_of(spec)
        d = str(tmp_path / f"c{seed}")
        binding.convert(iter(tensors), d, A, C_)
        want, index = expected(tensors, A, A2)
        n_chunks = -(-index.total_bytes // C_) + 2
        say("tiny cached", A, engine, A2, seed, C_)
        with binding.Pool(C_, n_chunks) as pool:
            pool.cache(d, io_threads=3)
            with binding.Checkpoint(d, pool=pool, engine=engine, dev_alignment=A2) as ck:
                assert ck.stats()["from_cache"] == 0
                assert_same(run_load(torch, ck, len(want)), want, f"seed {seed}")
                assert ck.stats()["from_cache"] == 1
            pool.evict(d)
            assert pool.info()["free_chunks"] == n_chunks


@pytest.mark.parametrize("engine", ["kernel", "sdma"])
@pytest.mark.parametrize("A,A2", [(16, 0), (1, 0), (4, 16)])
def test_every_chunk_size(torch_cuda, tmp_path, engine, A, A2):
    """Brute force over every chunk size that gives a distinct geometry."""
    torch = torch_cuda
    spec = synth.tiny(7, n=8, alignment=A, max_bytes=120)
    tensors = tensors_of(spec)
    d = str(tmp_path / "ck")
    binding.convert(iter(tensors), d, A, 64)
    want, index = expected(tensors, A, A2)
    T = index.total_bytes
    say("every chunk size", engine, A, A2, "T", T)
    for C_ in list(range(1, T + 2)) + [index.file_bytes, index.file_bytes + 1]:
        with binding.Checkpoint(d, engine=engine, chunk_size=C_, dev_alignment=A2, ring_slots=1 + C_ % 3,
                                io_threads=1 + C_ % 2) as ck:
            assert_same(run_load(torch, ck, len(want), slack=16), want, f"C={C_}")


def test_empty_checkpoint(torch_cuda, tmp_path):
    torch = torch_cuda
    binding.convert([], str(tmp_path), 256, 4096)
    with binding.Checkpoint(str(tmp_path)) as ck:
        assert ck.total_bytes == 0 and ck.tensors() == []
        run_load(torch, ck, 0)


# ---------------------------------------------------------------------------
# model-shaped workloads
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def opt125m(torch_cuda, tmp_path_factory):
    spec = synth.opt_125m()
    tensors = tensors_of(spec)
    d = str(tmp_path_factory.mktemp("opt"))
    binding.convert(iter(tensors), d, spec.alignment, spec.chunk_size)
    return spec, tensors, d


@pytest.mark.parametrize("engine", ["kernel", "sdma"])
@pytest.mark.parametrize("cached", [True, False])
def test_opt125m_file_layout(torch_cuda, opt125m, engine, cached):
    torch = torch_cuda
    spec, tensors, d = opt125m
    want, index = expected(tensors, spec.alignment)
    say("opt-125m", engine, "cached" if cached else "streamed")
    pool = binding.Pool(spec.chunk_size, 32) if cached else None
    try:
        if pool:
            pool.cache(d)
        with binding.Checkpoint(d, pool=pool, engine=engine, timing=True) as ck:
            got = run_load(torch, ck, len(want))
            assert_same(got, want, "opt-125m")
            st = ck.stats()
            assert st["bytes_loaded"] == index.total_bytes and st["from_cache"] == int(cached)
            assert st["device_ms"] > 0
            # views at base + offset hold each tensor's bytes
            buf = torch.empty(ck.total_bytes, dtype=torch.uint8, device="cuda:0")
            ck.load_into(buf)
            views = binding.views(buf, ck.tensors())
            torch.cuda.synchronize()
            for (name, dt, shape, data) in tensors[:40]:
                v = views[name]
                assert tuple(v.shape) == tuple(shape)
                assert v.contiguous().view(torch.uint8).cpu().numpy().tobytes() == data.tobytes()
    finally:
        if pool:
            pool.evict(d)
            pool.close()


@pytest.mark.parametrize("engine", ["kernel", "sdma"])
@pytest.mark.parametrize("shape", [{}, {"SLLM_K2_UNROLL": "4"}, {"SLLM_K2_NT": "0", "SLLM_K2_MAX_GRID": "997"},
                                   {"SLLM_K1_UNROLL": "4", "SLLM_K1_NT": "1", "SLLM_K1_BLOCKS": "96"},
                                   {"SLLM_K1_STREAM_BLOCKS": "3"}])
def test_opt125m_device_layout_and_repack(torch_cuda, opt125m, engine, shape, monkeypatch):
    """Every launch shape of the scatter and gather kernels gives the same bytes."""
    for k, v in shape.items():
        monkeypatch.setenv(k, v)
    torch = torch_cuda
    spec, tensors, d = opt125m
    A2 = 4096
    want2, _ = expected(tensors, spec.alignment, A2)
    want1, _ = expected(tensors, spec.alignment)
    say("opt-125m A2", engine, shape)
    with binding.Checkpoint(d, engine=engine, dev_alignment=A2) as ck:
        assert_same(run_load(torch, ck, len(want2)), want2, "A2 load")
        # the HBM-side repack (K2) of a file-layout image gives the same bytes
        src = torch.frombuffer(bytearray(want1), dtype=torch.uint8).to("cuda:0")
        dst = torch.full((len(want2) + 64,), SENTINEL, dtype=torch.uint8, device="cuda:0")
        ck.repack(src, dst)
        torch.cuda.synchronize()
        host = dst.cpu().numpy()
        assert (host[len(want2):] == SENTINEL).all()
        assert_same(host[:len(want2)].tobytes(), want2, "repack")


@pytest.mark.parametrize("A", [1, 4, 256, 4096])
def test_repack_tile_paths(torch_cuda, tmp_path, A):
    """The HBM repack moves 8 KiB destination tiles: tiles inside one
    tensor's data copy straight (aligned, or shifted when the file layout is
    not 16-byte aligned), the others (boundaries, padding, zero-size and tiny
    tensors) take the general path.  Tensors of up to ~200 KB at every file
    alignment, into A2 = 16 / 256 / 4096, through sllm_repack (the whole
    image), copy-engine loads from cached chunks (HBM staging windows of
    merged runs) and streamed ones (one chunk per window; C = 40000 is not a
    multiple of 16, so every window takes the general path)."""
    torch = torch_cuda
    for seed in range(3):
        spec = synth.tiny(100 + seed, n=48, alignment=A, max_bytes=200_000)
        tensors = tensors_of(spec)
        d = str(tmp_path / f"r{seed}")
        binding.convert(iter(tensors), d, A, 1 << 16)
        file_img, index = expected(tensors, A)
        src = torch.frombuffer(bytearray(file_img + bytes(64)), dtype=torch.uint8).to("cuda:0")
        for A2 in (16, 256, 4096):
            want, _ = expected(tensors, A, A2)
            say("repack tiles", A, A2, seed, len(want))
            with binding.Checkpoint(d, engine="sdma", dev_alignment=A2, chunk_size=1 << 16) as ck:
                dst = torch.full((len(want) + 64,), SENTINEL, dtype=torch.uint8, device="cuda:0")
                ck.repack(src, dst)
                torch.cuda.synchronize()
                host = dst.cpu().numpy()
                assert (host[len(want):] == SENTINEL).all()
                assert_same(host[:len(want)].tobytes(), want, f"repack A={A} A2={A2} seed {seed}")
                assert_same(run_load(torch, ck, len(want)), want, f"streamed sdma C=64K A2={A2}")
            with binding.Checkpoint(d, engine="sdma", dev_alignment=A2, chunk_size=40000) as ck:
                assert_same(run_load(torch, ck, len(want)), want, f"streamed sdma C=40000 A2={A2}")
            with binding.Pool(1 << 16, -(-index.total_bytes // (1 << 16)) + 1) as pool:
                pool.cache(d)
                with binding.Checkpoint(d, pool=pool, engine="sdma", dev_alignment=A2) as ck:
                    assert_same(run_load(torch, ck, len(want)), want, f"cached sdma A2={A2}")
                pool.evict(d)
    # 3,000 tensors of 1-32 bytes: at A2 = 16 a tile meets up to 512 slots,
    # more than the workgroup stages in LDS
    spec = synth.stress(n=3000, min_bytes=1, max_bytes=32, seed=9)
    tensors = tensors_of(spec)
    d = str(tmp_path / "small")
    binding.convert(iter(tensors), d, A, 1 << 16)
    file_img, _ = expected(tensors, A)
    want, _ = expected(tensors, A, 16)
    src = torch.frombuffer(bytearray(file_img + bytes(64)), dtype=torch.uint8).to("cuda:0")
    with binding.Checkpoint(d, engine="sdma", dev_alignment=16, chunk_size=1 << 16) as ck:
        dst = torch.full((len(want) + 64,), SENTINEL, dtype=torch.uint8, device="cuda:0")
        ck.repack(src, dst)
        torch.cuda.synchronize()
        host = dst.cpu().numpy()
        assert (host[len(want):] == SENTINEL).all()
        assert_same(host[:len(want)].tobytes(), want, f"repack of 3,000 small tensors, A={A}")
        assert_same(run_load(torch, ck, len(want)), want, f"streamed sdma, 3,000 small tensors, A={A}")


def test_stress_prefix_device_layout(torch_cuda, tmp_path):
    """Many small tensors of every dtype, 4 KiB file alignment, repacked to 256."""
    torch = torch_cuda
    spec = synth.stress(n=2000, max_bytes=1 << 18)
    tensors = tensors_of(spec)
    d = str(tmp_path)
    binding.convert(iter(tensors), d, spec.alignment, spec.chunk_size)
    for A2 in (0, 256, 16):
        want, _ = expected(tensors, spec.alignment, A2)
        for engine in ("kernel", "sdma"):
            say("stress prefix", A2, engine)
            with binding.Pool(spec.chunk_size, 1024) as pool:
                pool.cache(d)
                with binding.Checkpoint(d, pool=pool, engine=engine, dev_alignment=A2) as ck:
                    assert_same(run_load(torch, ck, len(want)), want, f"cached A2={A2} {engine}")
                pool.evict(d)
            with binding.Checkpoint(d, engine=engine, dev_alignment=A2, chunk_size=1 << 20) as ck:
                assert_same(run_load(torch, ck, len(want)), want, f"streamed A2={A2} {engine}")


# ---------------------------------------------------------------------------
# ordering and errors
# ---------------------------------------------------------------------------

def test_stream_ordering(torch_cuda, opt125m):
    """Work queued before the load runs first; work queued after sees all bytes."""
    torch = torch_cuda
    spec, tensors, d = opt125m
    want, _ = expected(tensors, spec.alignment)
    s = torch.cuda.Stream()
    with binding.Checkpoint(d, engine="sdma", n_streams=3) as ck:
        buf = torch.empty(len(want), dtype=torch.uint8, device="cuda:0")
        with torch.cuda.stream(s):
            torch.cuda._sleep(20_000_000)   # keep the stream busy so ordering matters
            buf.fill_(7)                    # queued before the load: must not clobber it
        ck.load_into(buf, s)
        with torch.cuda.stream(s):
            checksum = buf[: 1 << 20].to(torch.int64).sum()
        s.synchronize()
        want_np = np.frombuffer(want, np.uint8)
        assert int(checksum) == int(want_np[: 1 << 20].astype(np.int64).sum())
        assert_same(buf.cpu().numpy().tobytes(), want, "ordered load")


def test_load_errors(torch_cuda, opt125m):
    torch = torch_cuda
    spec, tensors, d = opt125m
    with binding.Checkpoint(d) as ck:
        small = torch.empty(ck.total_bytes - 1, dtype=torch.uint8, device="cuda:0")
        with pytest.raises(binding.SllmError) as ei:
            ck.load_into(small)
        assert ei.value.code == -6
        buf = torch.empty(ck.total_bytes + 16, dtype=torch.uint8, device="cuda:0")
        with pytest.raises(binding.SllmError) as ei:
            ck.load(buf.data_ptr() + 1, ck.total_bytes)
        assert ei.value.code == -1
        with pytest.raises(binding.SllmError) as ei:
            ck.find("no.such.tensor")
        assert ei.value.code == -8
        # host memory (pageable or pinned) is refused before any device work
        host = np.zeros(ck.total_bytes + 16, np.uint8)
        with pytest.raises(binding.SllmError) as ei:
            ck.load((host.ctypes.data + 15) & ~15, ck.total_bytes)
        assert ei.value.code == -1 and "not device memory" in ei.value.message
        pinned = torch.empty(ck.total_bytes, dtype=torch.uint8, pin_memory=True)
        with pytest.raises(binding.SllmError) as ei:
            ck.load_into(pinned)
        assert ei.value.code == -1 and "not device memory" in ei.value.message
        # the handle still works after the errors
        want, _ = expected(tensors, spec.alignment)
        assert_same(run_load(torch, ck, len(want)), want, "after errors")


def test_pool_rules(torch_cuda, opt125m):
    spec, tensors, d = opt125m
    with binding.Pool(spec.chunk_size, 4) as tiny_pool:
        with pytest.raises(binding.SllmError) as ei:
            tiny_pool.cache(d)             # 15 chunks needed
        assert ei.value.code == -4
        assert tiny_pool.info()["free_chunks"] == 4
    pool = binding.Pool(spec.chunk_size, 20)
    pool.cache(d)
    with pytest.raises(binding.SllmError) as ei:
        pool.cache(d)
    assert ei.value.code == -7
    ck = binding.Checkpoint(d, pool=pool)
    with pytest.raises(binding.SllmError) as ei:
        pool.evict(d)
    assert ei.value.code == -7
    with pytest.raises(binding.SllmError) as ei:
        pool.close()
    assert ei.value.code == -7
    ck.close()
    pool.evict(d)
    with pytest.raises(binding.SllmError) as ei:
        pool.evict(d)
    assert ei.value.code == -8
    pool.close()


def test_io_error_mid_load(torch_cuda, tmp_path):
    """A read failure stops the load with SLLM_E_IO; the handle stays usable."""
    torch = torch_cuda
    spec = synth.opt_125m()
    tensors = tensors_of(spec)
    d = tmp_path / "ck"
    binding.convert(iter(tensors), str(d), spec.alignment, spec.chunk_size)
    want, _ = expected(tensors, spec.alignment)
    with binding.Checkpoint(str(d), chunk_size=1 << 20) as ck:
        path = d / "sllm.part0"
        full = open(path, "rb").read()
        with open(path, "r+b") as f:
            f.truncate(len(full) // 2)      # later chunks now hit end of file
        buf = torch.empty(len(want), dtype=torch.uint8, device="cuda:0")
        with pytest.raises(binding.SllmError) as ei:
            ck.load_into(buf)
        assert ei.value.code == -2
        with open(path, "wb") as f:
            f.write(full)
        assert_same(run_load(torch, ck, len(want)), want, "after restoring the file")


@pytest.mark.parametrize("engine", ["kernel", "sdma"])
def test_direct_io(torch_cuda, opt125m, engine):
    """O_DIRECT reads (straight into pinned chunks, or through the bounce
    buffer where the kernel refuses that) give the same bytes."""
    torch = torch_cuda
    spec, tensors, d = opt125m
    want, index = expected(tensors, spec.alignment)
    say("direct io", engine)
    with binding.Checkpoint(d, engine=engine, direct_io=True, chunk_size=1 << 20, io_threads=4) as ck:
        assert_same(run_load(torch, ck, len(want)), want, "direct streamed")
        st = ck.stats()
        if st["direct_io"]:
            assert st["bytes_read"] == index.file_bytes  # direct reads run to the 4 KiB-padded end
            assert st["bytes_bounced"] in (0, st["bytes_read"])
    with binding.Pool(1 << 20, 300) as pool:
        pool.cache(d, direct_io=True)
        with binding.Checkpoint(d, pool=pool, engine=engine) as ck:
            assert_same(run_load(torch, ck, len(want)), want, "direct cached")
        pool.evict(d)


def test_single_hip_runtime(torch_cuda):
    """The library and torch share one HIP runtime (streams and pointers agree)."""
    assert len(binding._hip_runtimes()) == 1


@pytest.mark.parametrize("shape", [{"SLLM_K1_UNROLL": "2"}, {"SLLM_K1_UNROLL": "4", "SLLM_K1_NT": "1"},
                                   {"SLLM_K1_BLOCKS": "1024"}, {"SLLM_K1_BLOCKS": "7", "SLLM_K1_UNROLL": "4"},
                                   {"SLLM_K1_STREAM_BLOCKS": "1"}, {"SLLM_K1_STREAM_BLOCKS": "1024"},
                                   {"SLLM_SPLIT_CHUNKS": "0"}, {"SLLM_SPLIT_CHUNKS": "1000000"},
                                   {"SLLM_READ_STREAM": "0"}, {"SLLM_READ_MAPPED": "1", "SLLM_SPLIT_CHUNKS": "1000000"}])
def test_gather_shapes(torch_cuda, opt125m, shape, monkeypatch):
    """Every launch shape of the chunk gather, and every way the streamed
    load reads its chunks (whole or in pieces, directly, through the
    streaming buffer or the mapping), gives the same bytes."""
    for k, v in shape.items():
        monkeypatch.setenv(k, v)
    torch = torch_cuda
    spec, tensors, d = opt125m
    want, _ = expected(tensors, spec.alignment)
    with binding.Pool(spec.chunk_size, 16) as pool:
        pool.cache(d)
        with binding.Checkpoint(d, pool=pool) as ck:
            assert_same(run_load(torch, ck, len(want)), want, f"cached {shape}")
        pool.evict(d)
    with binding.Checkpoint(d, chunk_size=3 << 20) as ck:
        assert_same(run_load(torch, ck, len(want)), want, f"streamed {shape}")


@pytest.mark.parametrize("engine", ["kernel", "sdma"])
def test_pipeline_timeline(torch_cuda, opt125m, tmp_path, monkeypatch, engine):
    """SLLM_TRACE_FILE: each streamed load appends its timeline; every chunk
    is read, moved and done once, in that order, and a slot is read again
    only after the chunk it held is done.  The loads stay byte-exact."""
    import csv

    torch = torch_cuda
    spec, tensors, d = opt125m
    want, _ = expected(tensors, spec.alignment)
    path = tmp_path / "trace.csv"
    monkeypatch.setenv("SLLM_TRACE_FILE", str(path))
    C = 1 << 20
    with binding.Checkpoint(d, engine=engine, chunk_size=C, ring_slots=8, io_threads=4) as ck:
        for rep in range(2):
            assert_same(run_load(torch, ck, len(want)), want, f"traced load {rep}")
    n = -(-len(want) // C)
    rows = list(csv.DictReader(open(path)))
    loads = sorted({r["load"] for r in rows})
    assert len(loads) == 2
    for ld in loads:
        t = {}
        for r in rows:
            if r["load"] == ld:
                key = (int(r["chunk"]), r["event"])
                assert key not in t, f"{key} recorded twice"
                t[key] = (float(r["t_s"]), int(r["slot"]))
        assert len(t) == 4 * n
        uses = {}
        for k in range(n):
            times = [t[(k, e)][0] for e in ("read_begin", "read_end", "moved", "done")]
            assert times == sorted(times), (k, times)
            uses.setdefault(t[(k, "read_begin")][1], []).append((times[0], times[3]))
        for slot, u in uses.items():
            u.sort()
            assert all(b[0] >= a[1] for a, b in zip(u, u[1:])), f"slot {slot} refilled before its chunk was done"


@pytest.mark.parametrize("engine", ["kernel", "sdma"])
@pytest.mark.parametrize("C", [64 << 10, (64 << 10) + 48, 1 << 20])
def test_streamed_batches(torch_cuda, opt125m, engine, C):
    """Many small chunks through a deep ring: the issue loop moves every
    ready chunk of a pass in one batched gather (up to 64 slots, at most a
    quarter of the ring)."""
    torch = torch_cuda
    spec, tensors, d = opt125m
    want, _ = expected(tensors, spec.alignment)
    with binding.Checkpoint(d, engine=engine, chunk_size=C, ring_slots=48, io_threads=8) as ck:
        for rep in range(2):
            assert_same(run_load(torch, ck, len(want)), want, f"C={C} rep {rep}")
        st = ck.stats()
        n = -(-len(want) // C)
        assert st["n_chunks"] == n
        if engine == "kernel" and C % 16 == 0:
            assert st["n_launches"] <= n
        say("batches", engine, C, "chunks", n, "launches", st["n_launches"])


def test_concurrent_handles(torch_cuda, opt125m):
    """Handles are independent: two threads load through separate handles
    (one pool cache, separate streams) and a third streams from the file."""
    import threading

    torch = torch_cuda
    spec, tensors, d = opt125m
    want, _ = expected(tensors, spec.alignment)
    errors, results = [], {}
    with binding.Pool(spec.chunk_size, 16 + 8) as pool:
        pool.cache(d)

        def work(tag, **kw):
            try:
                s = torch.cuda.Stream()
                with binding.Checkpoint(d, **kw) as ck:
                    for rep in range(3):
                        buf = torch.empty(len(want), dtype=torch.uint8, device="cuda:0")
                        ck.load_into(buf, s)
                        s.synchronize()
                        results[(tag, rep)] = buf.cpu().numpy().tobytes()
            except Exception as e:  # noqa: BLE001
                errors.append(e)

        ts = [threading.Thread(target=work, args=("k1",), kwargs=dict(pool=pool)),
              threading.Thread(target=work, args=("sdma",), kwargs=dict(pool=pool, engine="sdma")),
              threading.Thread(target=work, args=("ring",), kwargs=dict(chunk_size=4 << 20))]
        for t in ts:
            t.start()
        for t in ts:
            t.join()
        pool.evict(d)
    assert not errors, errors
    assert len(results) == 9
    for k, v in results.items():
        assert_same(v, want, str(k))


def test_fragmented_pool(torch_cuda, opt125m, tmp_path):
    """After evictions a cached partition's chunks are scattered over the
    pool (not adjacent in host memory): every engine and layout still loads
    it exactly."""
    torch = torch_cuda
    spec, tensors, d = opt125m
    want, _ = expected(tensors, spec.alignment)
    want2, _ = expected(tensors, spec.alignment, 256)
    C = 4 << 20  # the OPT-125M partition takes 60 chunks
    smalls = []
    for i in range(24):  # one-chunk checkpoints
        sp = synth.tiny(100 + i, alignment=256)
        sd = str(tmp_path / f"s{i}")
        binding.convert(iter(tensors_of(sp)), sd, 256, C)
        smalls.append(sd)
    with binding.Pool(C, 24 + 60) as pool:
        for sd in smalls:
            pool.cache(sd)          # chunks 0..23
        for sd in smalls[::2]:
            pool.evict(sd)          # holes at 0, 2, ..., 22
        pool.cache(d)               # 12 holes, then chunks 24..71
        for engine in ("kernel", "sdma"):
            for a2, ref in ((0, want), (256, want2)):
                with binding.Checkpoint(d, pool=pool, engine=engine, dev_alignment=a2) as ck:
                    assert_same(run_load(torch, ck, len(ref)), ref, f"fragmented {engine} A2={a2}")
        pool.evict(d)
        for sd in smalls[1::2]:
            pool.evict(sd)
        assert pool.info()["free_chunks"] == 24 + 60


@pytest.mark.parametrize("A2", [16, 256, 4096])
def test_offsets_scan_20000_tensors(torch_cuda, tmp_path, A2):
    """20,000 tensors (the stress workload's count, here with small sizes):
    the device offsets scan runs over 20 blocks of 1,024 entries with a
    carry; sllm_open checks it against the host plan, and the loaded device
    layout matches the oracle's."""
    torch = torch_cuda
    spec = synth.stress(n=20000, min_bytes=1, max_bytes=600, seed=77)
    tensors = tensors_of(spec)
    d = str(tmp_path)
    binding.convert(iter(tensors), d, spec.alignment, 1 << 20)
    want, index = expected(tensors, spec.alignment, A2)
    d2, T2 = oracle.device_layout(index, A2)
    with binding.Checkpoint(d, dev_alignment=A2, chunk_size=1 << 20) as ck:
        assert [t.offset for t in ck.tensors()] == d2 and ck.total_bytes == T2
        assert_same(run_load(torch, ck, len(want)), want, f"A2={A2}")


@pytest.mark.parametrize("threaded", [True, False])
@pytest.mark.parametrize("cached", [True, False])
def test_load_with_views(torch_cuda, opt125m, cached, threaded, monkeypatch):
    """Views built while the load runs on a helper thread (or after it, for
    few tensors) hold every tensor's bytes once the stream is synchronized,
    and a load error reaches the caller."""
    torch = torch_cuda
    monkeypatch.setattr(binding, "_THREADED_VIEWS_MIN", 0 if threaded else 1 << 30)
    spec, tensors, d = opt125m
    pool = binding.Pool(spec.chunk_size, 32) if cached else None
    try:
        if pool:
            pool.cache(d)
        with binding.Checkpoint(d, pool=pool) as ck:
            buf = torch.full((ck.total_bytes,), SENTINEL, dtype=torch.uint8, device="cuda:0")
            s = torch.cuda.Stream()
            marks = []
            views = ck.load_with_views(buf, s, after_load=lambda: marks.append(1))
            s.synchronize()
            assert marks == [1] and len(views) == len(tensors)
            for (name, dt, shape, data) in tensors:
                v = views[name]
                assert tuple(v.shape) == tuple(shape)
                assert v.contiguous().view(torch.uint8).cpu().numpy().tobytes() == data.tobytes(), name
            small = torch.empty(ck.total_bytes - 1, dtype=torch.uint8, device="cuda:0")
            with pytest.raises(binding.SllmError) as e:
                ck.load_with_views(small, s)
            assert e.value.code == -6
    finally:
        if pool:
            pool.evict(d)
            pool.close()


@pytest.mark.parametrize("engine", ["kernel", "sdma"])
@pytest.mark.parametrize("direct", [False, True])
def test_open_cache_keeps_first_load(torch_cuda, opt125m, engine, direct):
    """SLLM_OPEN_CACHE: the first load streams the file into one pool chunk
    per partition chunk and leaves them as the pool's cached copy; the next
    load of the handle and a new handle's load come from that cache, every
    load byte-identical; eviction waits for the handle to close."""
    torch = torch_cuda
    spec, tensors, d = opt125m
    want, index = expected(tensors, spec.alignment)
    n = -(-index.total_bytes // spec.chunk_size)
    with binding.Pool(spec.chunk_size, n + 3) as pool:
        with binding.Checkpoint(d, pool=pool, engine=engine, cache=True, direct_io=direct, io_threads=4) as ck:
            info = pool.info()
            assert info["free_chunks"] == 3 and info["cached_checkpoints"] == 0
            assert_same(run_load(torch, ck, len(want)), want, "first load")
            st = ck.stats()
            assert st["from_cache"] == 0 and st["bytes_read"] >= index.total_bytes
            info = pool.info()
            assert info["cached_checkpoints"] == 1 and info["free_chunks"] == 3
            with pytest.raises(binding.SllmError) as ei:
                pool.evict(d)
            assert ei.value.code == -7
            assert_same(run_load(torch, ck, len(want)), want, "second load")
            assert ck.stats()["from_cache"] == 1
            with binding.Checkpoint(d, pool=pool, engine=engine, cache=True) as ck2:
                assert_same(run_load(torch, ck2, len(want)), want, "another handle")
                assert ck2.stats()["from_cache"] == 1
        pool.evict(d)
        assert pool.info()["free_chunks"] == n + 3


def test_open_cache_rules(torch_cuda, opt125m, tmp_path):
    """SLLM_OPEN_CACHE needs a pool with room and the pool's chunk size; a
    failed first load caches nothing and gives every chunk back at close."""
    torch = torch_cuda
    spec, tensors, d = opt125m
    want, index = expected(tensors, spec.alignment)
    n = -(-index.total_bytes // spec.chunk_size)
    with pytest.raises(binding.SllmError) as ei:
        binding.Checkpoint(d, cache=True)
    assert ei.value.code == -1
    with binding.Pool(spec.chunk_size, n - 1) as small:
        with pytest.raises(binding.SllmError) as ei:
            binding.Checkpoint(d, pool=small, cache=True)
        assert ei.value.code == -4
        assert small.info()["free_chunks"] == n - 1
    with binding.Pool(spec.chunk_size, n) as pool:
        with pytest.raises(binding.SllmError) as ei:
            binding.Checkpoint(d, pool=pool, cache=True, chunk_size=spec.chunk_size // 2)
        assert ei.value.code == -1
        # a read failure in the first load: nothing is cached
        d2 = tmp_path / "ck"
        binding.convert(iter(tensors), str(d2), spec.alignment, spec.chunk_size)
        path = d2 / "sllm.part0"
        full = open(path, "rb").read()
        with binding.Checkpoint(str(d2), pool=pool, cache=True) as ck:
            with open(path, "r+b") as f:
                f.truncate(len(full) // 2)
            buf = torch.empty(len(want), dtype=torch.uint8, device="cuda:0")
            with pytest.raises(binding.SllmError) as ei:
                ck.load_into(buf)
            assert ei.value.code == -2
            assert pool.info()["cached_checkpoints"] == 0
            with open(path, "wb") as f:
                f.write(full)
            assert_same(run_load(torch, ck, len(want)), want, "after restoring the file")
            assert pool.info()["cached_checkpoints"] == 1
        pool.evict(str(d2))
        assert pool.info()["free_chunks"] == n


@pytest.mark.parametrize("engine", ["kernel", "sdma"])
def test_mapped_reader(torch_cuda, opt125m, engine, monkeypatch, tmp_path):
    """The opt-in mapped reader (SLLM_READ_MAPPED=1: page tables populated
    per step, streaming-store copies): streamed loads at a page-multiple and
    an odd chunk size, the DRAM-tier fill, and a truncated file failing with
    SLLM_E_IO and leaving the handle usable."""
    monkeypatch.setenv("SLLM_READ_MAPPED", "1")
    torch = torch_cuda
    spec, tensors, d = opt125m
    want, _ = expected(tensors, spec.alignment)
    for C in (1 << 20, 40000):
        with binding.Checkpoint(d, engine=engine, chunk_size=C, ring_slots=6, io_threads=3) as ck:
            assert_same(run_load(torch, ck, len(want)), want, f"mapped streamed C={C}")
    with binding.Pool(1 << 20, -(-len(want) // (1 << 20))) as pool:
        pool.cache(d, io_threads=4)
        with binding.Checkpoint(d, pool=pool, engine=engine) as ck:
            assert_same(run_load(torch, ck, len(want)), want, "mapped fill, cached load")
        pool.evict(d)
    c = tmp_path / "trunc"
    binding.convert(iter(tensors), str(c), spec.alignment, spec.chunk_size)
    with binding.Checkpoint(str(c), engine=engine, chunk_size=1 << 20) as ck:
        path = c / "sllm.part0"
        full = open(path, "rb").read()
        with open(path, "r+b") as f:
            f.truncate(len(full) // 2)
        buf = torch.empty(len(want), dtype=torch.uint8, device="cuda:0")
        with pytest.raises(binding.SllmError) as ei:
            ck.load_into(buf)
        assert ei.value.code == -2
        with open(path, "wb") as f:
            f.write(full)
        assert_same(run_load(torch, ck, len(want)), want, "mapped, after restoring the file")


@pytest.mark.parametrize("engine", ["kernel", "sdma"])
@pytest.mark.parametrize("A2", [0, 256])
@pytest.mark.parametrize("cached", [False, True])
def test_load_into_a_region_of_an_arena(torch_cuda, tmp_path, engine, A2, cached):
    """The destination is a region inside a larger device allocation (a
    serving arena): the load writes exactly that region, every byte equal to
    the oracle's, nothing before or after it; views built over the region
    hold each tensor's bytes; a region that is not 16-byte aligned, or one
    byte short, is refused before any device work."""
    torch = torch_cuda
    spec = synth.tiny(21, n=20, alignment=256, max_bytes=50_000)
    tensors = tensors_of(spec)
    d = str(tmp_path / "arena")
    binding.convert(iter(tensors), d, 256, 4096)
    want, index = expected(tensors, 256, A2)
    pool = binding.Pool(4096, -(-index.total_bytes // 4096)) if cached else None
    try:
        if pool:
            pool.cache(d)
        with binding.Checkpoint(d, pool=pool, engine=engine, dev_alignment=A2, ring_slots=4) as ck:
            s = torch.cuda.Stream()
            for start in (16, 48, 4096 + 16):
                say("arena region", engine, A2, cached, start)
                arena = torch.full((start + len(want) + 64,), SENTINEL, dtype=torch.uint8, device="cuda:0")
                region = arena[start:start + len(want)]
                s.wait_stream(torch.cuda.current_stream())
                ck.load_into(region, s)
                s.synchronize()
                host = arena.cpu().numpy()
                assert (host[:start] == SENTINEL).all(), f"bytes before the region written (start {start})"
                assert (host[start + len(want):] == SENTINEL).all(), f"bytes after the region written (start {start})"
                assert_same(host[start:start + len(want)].tobytes(), want, f"region at {start}")
                region.fill_(SENTINEL)
                views = ck.load_with_views(region, s)
                s.synchronize()
                for (name, dt, shape, data) in tensors:
                    v = views[name]
                    assert tuple(v.shape) == tuple(shape), name
                    got = v.reshape(-1).contiguous().view(torch.uint8).cpu().numpy().tobytes()  # 0-d: one element
                    assert got == data.tobytes(), name
            arena = torch.full((len(want) + 64,), SENTINEL, dtype=torch.uint8, device="cuda:0")
            with pytest.raises(binding.SllmError) as e:  # 8-byte aligned only
                ck.load(arena.data_ptr() + 8, len(want), s)
            assert e.value.code == -1
            with pytest.raises(binding.SllmError) as e:  # a region one byte short
                ck.load(arena.data_ptr() + 16, len(want) - 1, s)
            assert e.value.code == -6
            torch.cuda.synchronize()
            assert (arena.cpu().numpy() == SENTINEL).all(), "a refused load wrote bytes"
    finally:
        if pool:
            pool.evict(d)
            pool.close()
