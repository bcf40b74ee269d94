"""The allocation-free repack (sllm_repack_noalloc) against sllm_repack and
the oracle, through the C ABI: two calls in a row, the second on a smaller
checkpoint, so nothing the first call left in the library's scratch area can
leak into the second; the destination windowed into many plan windows; the
handle's own alignment; and the errors it reports before any device work."""

import ctypes as C
import sys

import numpy as np
import pytest

import oracle
from paper_2401_14351_amd import binding, synth

pytestmark = pytest.mark.gpu

SENTINEL = 0xC3


def say(*a):
    print("[gpu-noalloc]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.lib()  # fail loudly if the library is missing
    return torch


def converted(spec, d):
    tensors = [(t.name, t.dtype, t.shape, x) for t, x in zip(spec.tensors, synth.materialize(spec))]
    binding.convert(iter(tensors), d, spec.alignment, spec.chunk_size)
    index = oracle.make_index(tensors, spec.alignment, 1)
    image = bytes(oracle.partition_bytes(tensors, spec.alignment)[:index.total_bytes])
    return tensors, index, image


def device_bytes(torch, data: bytes, slack: int = 64):
    return torch.frombuffer(bytearray(data + bytes(slack)), dtype=torch.uint8).to("cuda:0")


def sentinel_buf(torch, n: int, slack: int = 64):
    return torch.full((n + slack,), SENTINEL, dtype=torch.uint8, device="cuda:0")


def rc_of(h, a2, src, src_bytes, dst, dst_bytes):
    return binding.lib().sllm_repack_noalloc(h, a2, src, src_bytes, dst, dst_bytes, None)


def image_of(torch, buf, n):
    torch.cuda.synchronize()
    host = buf.cpu().numpy()
    assert (host[n:] == SENTINEL).all(), "bytes past the image were written"
    return host[:n].tobytes()


def repack_both(torch, d, index, image, a2):
    """sllm_repack (a handle opened with A2) and sllm_repack_noalloc (an
    index-only handle, A2 passed in) of the same source, on one stream."""
    want = bytes(oracle.repack(image, index, a2))
    src = device_bytes(torch, image)
    ref = sentinel_buf(torch, len(want))
    out = sentinel_buf(torch, len(want))
    with binding.Checkpoint(d, dev_alignment=a2) as ck:
        assert ck.total_bytes == len(want)
        ck.repack(src, ref)
    with binding.Checkpoint(d, index_only=True) as ix:
        h = ix._h
        rc = rc_of(h, a2, src.data_ptr(), src.numel(), out.data_ptr(), out.numel())
        assert rc == binding.SLLM_OK, binding.lib().sllm_last_error().decode()
        got = image_of(torch, out, len(want))
    assert image_of(torch, ref, len(want)) == want, "sllm_repack differs from the oracle"
    if got != want:
        a, b = np.frombuffer(got, np.uint8), np.frombuffer(want, np.uint8)
        bad = np.nonzero(a != b)[0]
        raise AssertionError(f"no-alloc repack A2={a2}: {bad.size} bytes differ, first at {bad[:8].tolist()}")
    return len(want)


def test_two_calls_then_smaller(torch_cuda, tmp_path):
    torch = torch_cuda
    big = synth.stress(n=600, max_bytes=1 << 20)  # 4 KiB file alignment: padding after most tensors
    d1 = str(tmp_path / "big")
    _, ix1, img1 = converted(big, d1)
    say("first call: stress n=600 T", ix1.total_bytes)
    n1 = repack_both(torch, d1, ix1, img1, 256)
    small = synth.tiny(7, n=48, alignment=1, max_bytes=200_000)  # dense file layout: unaligned shifts
    d2 = str(tmp_path / "small")
    _, ix2, img2 = converted(small, d2)
    say("second call: tiny n=48 A=1 T", ix2.total_bytes)
    n2 = repack_both(torch, d2, ix2, img2, 16)
    assert n2 < n1 and len(small.tensors) < len(big.tensors)


def test_many_windows(torch_cuda, tmp_path, monkeypatch):
    """Three plan blocks (48 KiB of destination) a window: the repack runs
    as many plan + K2 passes through the same scratch plan area."""
    torch = torch_cuda
    spec = synth.stress(n=200, max_bytes=256 << 10, seed=77)
    d = str(tmp_path / "w")
    _, ix, img = converted(spec, d)
    monkeypatch.setenv("SLLM_NOALLOC_PLAN_BLOCKS", "3")
    for a2 in (4096, 256, 16):
        say("windows of 3 plan blocks, A2", a2)
        repack_both(torch, d, ix, img, a2)


def test_handle_alignment(torch_cuda, tmp_path):
    """dev_alignment = 0 takes the handle's own A2."""
    torch = torch_cuda
    spec = synth.tiny(11, n=40, alignment=16, max_bytes=50_000)
    d = str(tmp_path / "h")
    _, ix, img = converted(spec, d)
    want = bytes(oracle.repack(img, ix, 4096))
    src = device_bytes(torch, img)
    out = sentinel_buf(torch, len(want))
    with binding.Checkpoint(d, dev_alignment=4096) as ck:
        ck.repack_noalloc(src, out)
    assert image_of(torch, out, len(want)) == want


def test_errors(torch_cuda, tmp_path):
    torch = torch_cuda
    spec = synth.tiny(3, n=12, alignment=16)
    d = str(tmp_path / "e")
    _, ix, img = converted(spec, d)
    want = bytes(oracle.repack(img, ix, 256))
    src = device_bytes(torch, img)
    dst = sentinel_buf(torch, len(want))
    with binding.Checkpoint(d, index_only=True) as ck:
        h = ck._h
        cases = [(0, len(img), len(want), -1, "no alignment"), (8, len(img), len(want), -1, "A2 < 16"),
                 (48, len(img), len(want), -1, "A2 not a power of two"),
                 (256, len(img) - 1, len(want), -6, "source too small"),
                 (256, len(img), len(want) - 1, -6, "destination too small")]
        for a2, sb, db, code, what in cases:
            rc = rc_of(h, a2, src.data_ptr(), sb, dst.data_ptr(), db)
            assert rc == code, (what, rc, binding.lib().sllm_last_error().decode())
        # a host buffer is refused, not written
        host = (C.c_uint8 * (len(want) + 64))()
        rc = rc_of(h, 256, src.data_ptr(), len(img), C.addressof(host), len(want))
        assert rc == -1, binding.lib().sllm_last_error().decode()
    assert rc_of(None, 256, src.data_ptr(), len(img), dst.data_ptr(), len(want)) == -1
    assert image_of(torch, dst, len(want)) == bytes([SENTINEL]) * len(want)


def test_too_many_tensors(torch_cuda, tmp_path):
    """One tensor more than the scratch area holds: RANGE, before any device work."""
    n = 65537
    d = str(tmp_path / "many")
    tensors = [(f"z{i}", "i8", (0,), np.zeros(0, np.uint8)) for i in range(n)]
    binding.convert(iter(tensors), d, 16, 1 << 20)
    torch = torch_cuda
    src = torch.zeros(64, dtype=torch.uint8, device="cuda:0")
    dst = torch.zeros(64, dtype=torch.uint8, device="cuda:0")
    with binding.Checkpoint(d, index_only=True) as ck:
        rc = rc_of(ck._h, 256, src.data_ptr(), 64, dst.data_ptr(), 64)
        assert rc == -6, binding.lib().sllm_last_error().decode()
        assert b"65537" in binding.lib().sllm_last_error()


def test_captured_in_a_graph(torch_cuda, tmp_path):
    """The allocation-free repack recorded into a HIP graph (its first call,
    which looks up the scratch area, runs eagerly before the capture) and
    replayed three times over three different source images, with eager
    copies and synchronizations between the replays: every replay equals the
    oracle's repack of the image it read."""
    torch = torch_cuda
    spec = synth.stress(n=120, max_bytes=256 << 10, seed=31)
    d = str(tmp_path / "g")
    _, ix, img = converted(spec, d)
    a2 = 256
    T = ix.total_bytes
    want0 = bytes(oracle.repack(img, ix, a2))
    src = device_bytes(torch, img)
    out = sentinel_buf(torch, len(want0))
    rng = np.random.default_rng(5)
    with binding.Checkpoint(d, index_only=True) as ck:
        h = ck._h
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):  # the eager first call: scratch lookup, same bytes
            assert rc_of(h, a2, src.data_ptr(), src.numel(), out.data_ptr(), out.numel()) == 0
        torch.cuda.current_stream().wait_stream(side)
        assert image_of(torch, out, len(want0)) == want0
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            s = torch.cuda.current_stream()
            rc = binding.lib().sllm_repack_noalloc(h, a2, src.data_ptr(), src.numel(), out.data_ptr(), out.numel(),
                                                   C.c_void_p(s.cuda_stream))
        assert rc == 0, binding.lib().sllm_last_error().decode()
        for k in range(3):
            # a new source image: random bytes in the tensors' slots, the
            # file layout's zero padding kept (the repack reads only data bytes)
            raw = bytearray(img)
            for e in ix.entries:
                raw[e.offset:e.offset + e.nbytes] = rng.integers(0, 256, e.nbytes, dtype=np.uint8).tobytes()
            new = bytes(raw)
            src[:T].copy_(torch.frombuffer(bytearray(new), dtype=torch.uint8))
            out[:len(want0)].fill_(SENTINEL)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert image_of(torch, out, len(want0)) == bytes(oracle.repack(new, ix, a2)), f"replay {k}"


def test_allocates_no_device_memory(torch_cuda, tmp_path):
    """After the first call on the device (which loads the library's code
    object and with it the scratch area), further calls leave the device's
    free memory exactly as it was: nothing is allocated, not even inside
    the runtime."""
    torch = torch_cuda
    spec = synth.stress(n=300, max_bytes=1 << 20, seed=41)
    d = str(tmp_path / "m")
    _, ix, img = converted(spec, d)
    want = bytes(oracle.repack(img, ix, 256))
    src = device_bytes(torch, img)
    out = sentinel_buf(torch, len(want))
    with binding.Checkpoint(d, index_only=True) as ck:
        h = ck._h
        assert rc_of(h, 256, src.data_ptr(), src.numel(), out.data_ptr(), out.numel()) == 0
        torch.cuda.synchronize()
        free0, _ = torch.cuda.mem_get_info()
        for _ in range(3):
            assert rc_of(h, 256, src.data_ptr(), src.numel(), out.data_ptr(), out.numel()) == 0
        torch.cuda.synchronize()
        free1, _ = torch.cuda.mem_get_info()
    assert free1 == free0, f"device free memory moved by {free0 - free1} bytes"
    assert image_of(torch, out, len(want)) == want
