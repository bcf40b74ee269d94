"""The binding's host logic on the CPU: views at base + offset over an image
the oracle built (a torch CPU tensor stands in for the device buffer), in the
file layout and in device layouts, with the offsets an index-only open
reports."""

import os

import numpy as np
import pytest
import torch

import oracle
from paper_2401_14351_amd import binding, synth

TORCH_DTYPE = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16, "i8": torch.int8}


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("libsllm.so not built")
    return binding.lib()


@pytest.mark.parametrize("A,A2", [(16, 0), (1, 0), (4096, 256), (1, 16)])
def test_views_over_oracle_image(L, tmp_path, A, A2):
    spec = synth.tiny(31, n=40, alignment=A, max_bytes=5000)
    tensors = [(t.name, t.dtype, t.shape, d) for t, d in zip(spec.tensors, synth.materialize(spec))]
    binding.convert(iter(tensors), str(tmp_path), A, 4096)
    index = oracle.make_index(tensors, A, 4096)
    image = oracle.partition_bytes(tensors, A)[:index.total_bytes]
    if A2:
        image = oracle.repack(image, index, A2)
    buf = torch.frombuffer(bytearray(bytes(image) + bytes(64)), dtype=torch.uint8)
    with binding.Checkpoint(str(tmp_path), index_only=True, dev_alignment=A2) as ck:
        entries = ck.tensors()
        assert ck.total_bytes == len(image)
    views = binding.views(buf, entries)
    assert list(views) == [name for name, *_ in tensors]
    typed = 0
    for (name, dt, shape, data), e in zip(tensors, entries):
        v = views[name]
        if e.nbytes:  # a view at base + offset, no copy (torch gives empty tensors no address)
            assert v.data_ptr() == buf.data_ptr() + e.offset
        raw = v.contiguous().reshape(-1).view(torch.uint8).numpy().tobytes()
        assert raw == np.asarray(data).tobytes(), name
        isz = torch.tensor([], dtype=TORCH_DTYPE[dt]).element_size()
        if e.offset % isz == 0:
            typed += 1
            assert v.dtype == TORCH_DTYPE[dt] and tuple(v.shape) == tuple(shape), name
        else:  # dense file layout: a tensor off its element alignment stays raw bytes
            assert v.dtype == torch.uint8 and v.numel() == e.nbytes, name
    assert typed > 0


def test_contiguous_strides():
    assert binding._contiguous_strides(()) == ()
    assert binding._contiguous_strides((3, 5)) == (5, 1)
    assert binding._contiguous_strides((2, 0, 4)) == (4, 4, 1)
    assert binding._contiguous_strides((7,)) == (1,)


@pytest.mark.parametrize("start", [16, 4096 + 48, 3])
def test_views_of_a_sliced_buffer(L, tmp_path, start):
    """The buffer is a slice that starts inside a larger allocation (a region
    of a preallocated arena): every view still sits at buf + offset and holds
    the tensor's bytes, not bytes from before the slice."""
    spec = synth.tiny(33, n=30, alignment=16, max_bytes=3000)
    tensors = [(t.name, t.dtype, t.shape, d) for t, d in zip(spec.tensors, synth.materialize(spec))]
    binding.convert(iter(tensors), str(tmp_path), 16, 4096)
    index = oracle.make_index(tensors, 16, 4096)
    image = bytes(oracle.partition_bytes(tensors, 16)[:index.total_bytes])
    arena = torch.full((start + len(image) + 64,), 0xEE, dtype=torch.uint8)
    arena[start:start + len(image)] = torch.frombuffer(bytearray(image), dtype=torch.uint8)
    buf = arena[start:start + len(image)]
    with binding.Checkpoint(str(tmp_path), index_only=True) as ck:
        entries = ck.tensors()
    views = binding.views(buf, entries)
    for (name, dt, shape, data), e in zip(tensors, entries):
        v = views[name]
        if e.nbytes:
            assert v.data_ptr() == buf.data_ptr() + e.offset, name
        raw = v.contiguous().reshape(-1).view(torch.uint8).numpy().tobytes()
        assert raw == np.asarray(data).tobytes(), name
        isz = torch.tensor([], dtype=TORCH_DTYPE[dt]).element_size()
        if start % isz == 0 and e.offset % isz == 0:
            assert v.dtype == TORCH_DTYPE[dt] and tuple(v.shape) == tuple(shape), name
        else:  # the slice starts off the element alignment: raw bytes
            assert v.dtype == torch.uint8 and v.numel() == e.nbytes, name


def test_buffers_must_be_flat_bytes(L, tmp_path):
    spec = synth.tiny(34, n=4, alignment=16)
    tensors = [(t.name, t.dtype, t.shape, d) for t, d in zip(spec.tensors, synth.materialize(spec))]
    binding.convert(iter(tensors), str(tmp_path), 16, 4096)
    with binding.Checkpoint(str(tmp_path), index_only=True) as ck:
        entries = ck.tensors()
        for bad in (torch.zeros(64, dtype=torch.float32), torch.zeros(8, 8, dtype=torch.uint8),
                    torch.zeros(128, dtype=torch.uint8)[::2]):
            with pytest.raises(ValueError):
                binding.views(bad, entries)
            with pytest.raises(ValueError):
                ck.load_into(bad)
