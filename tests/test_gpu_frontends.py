"""The small-checkpoint workload and the converter front-end on the GPU,
every byte against the oracle's layout and the generator's bytes:

* the rank-32 LoRA adapter of a 70B model (1,120 tensors, 0.83 GB; the
  paper's adapter-loading case, Sec. 7.2), cached and streamed, by both
  engines, in the file layout and at A2 = 256;
* checkpoints written as safetensors shards (by the test's own raw writer,
  so no safetensors package is needed) and converted by
  ``sllm_convert_safetensors``, then loaded.

Also the pool's arena boundaries: with arenas of a few chunks the copy
engines' merged copies must stop at every arena end."""

import json
import os
import struct

import numpy as np
import pytest

import oracle
from paper_2401_14351_amd import binding, synth, verify

pytestmark = pytest.mark.gpu

SENTINEL = 0xC3
ST_DTYPE = {"f32": "F32", "f16": "F16", "bf16": "BF16", "i8": "I8"}


def say(*a):
    print("[gpu-front]", *a, flush=True)


@pytest.fixture(scope="module")
def torch_cuda():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.lib()
    return torch


def load_and_check(torch, ck, spec, offsets, total, digests, what, stream=None):
    buf = torch.full((total + 4096,), SENTINEL, dtype=torch.uint8, device="cuda:0")
    s = stream or torch.cuda.current_stream()
    ck.load_into(buf, s)
    s.synchronize()
    assert bool((buf[total:] == SENTINEL).all()), f"{what}: bytes past the image were written"
    verify.check_image(torch, buf, spec, offsets, total, digests, window=64 << 20)
    say(what, "every byte matches")
    return ck.stats()


@pytest.fixture(scope="module")
def lora(tmp_path_factory):
    spec = synth.config("lora-70b-r32")
    d = str(tmp_path_factory.mktemp("lora"))
    digests = []

    def tensors():
        for _, t, data, dg in verify.generate(spec):
            digests.append(dg)
            yield t.name, t.dtype, t.shape, data

    binding.convert(tensors(), d, spec.alignment, spec.chunk_size)
    return spec, d, digests


@pytest.mark.parametrize("engine", ["kernel", "sdma"])
@pytest.mark.parametrize("A2", [0, 256])
def test_lora_adapter(torch_cuda, lora, engine, A2):
    torch = torch_cuda
    spec, d, digests = lora
    sizes = [t.nbytes for t in spec.tensors]
    offsets, T = oracle.plan_layout(sizes, A2 or spec.alignment)
    assert len(sizes) == 1120
    C = spec.chunk_size
    with binding.Pool(C, -(-T // C) + 8) as pool:
        pool.cache(d, io_threads=8)
        with binding.Checkpoint(d, pool=pool, engine=engine, dev_alignment=A2) as ck:
            assert [t.offset for t in ck.tensors()] == offsets
            st = load_and_check(torch, ck, spec, offsets, T, digests, f"lora cached {engine} A2={A2}")
            assert st["from_cache"] == 1
        pool.evict(d)
        with binding.Checkpoint(d, pool=pool, engine=engine, dev_alignment=A2, io_threads=4, ring_slots=8) as ck:
            st = load_and_check(torch, ck, spec, offsets, T, digests, f"lora streamed {engine} A2={A2}")
            assert st["from_cache"] == 0


def write_safetensors(path, spec, indices, data):
    """One shard: a JSON header (tensors in the given order, data offsets
    increasing) followed by the tensors' raw bytes."""
    header, parts, off = {}, [], 0
    for i in indices:
        t = spec.tensors[i]
        header[t.name] = {"dtype": ST_DTYPE[t.dtype], "shape": list(t.shape), "data_offsets": [off, off + t.nbytes]}
        parts.append(data[i].tobytes())
        off += t.nbytes
    h = json.dumps(header).encode()
    h += b" " * (-len(h) % 8)
    with open(path, "wb") as f:
        f.write(struct.pack("<Q", len(h)) + h)
        for p in parts:
            f.write(p)


@pytest.mark.parametrize("workload,shards", [("opt-125m", 3), ("lora-70b-r32", 2), ("tiny", 2)])
def test_safetensors_shards(torch_cuda, tmp_path, workload, shards):
    torch = torch_cuda
    spec = synth.tiny(5, n=40, alignment=16, max_bytes=5000) if workload == "tiny" else synth.config(workload)
    data = synth.materialize(spec)
    digests = [verify.combine([verify._hash(b[o:o + synth.block_size(t)])
                               for o in range(0, t.nbytes, synth.block_size(t))])
               for t, b in zip(spec.tensors, data)]
    n = len(spec.tensors)
    cuts = [n * k // shards for k in range(shards + 1)]
    paths = []
    for k in range(shards):
        p = str(tmp_path / f"model-{k:05d}-of-{shards:05d}.safetensors")
        write_safetensors(p, spec, range(cuts[k], cuts[k + 1]), data)
        paths.append(p)
    del data
    d = str(tmp_path / "converted")
    binding.convert_safetensors(paths, d, spec.alignment, spec.chunk_size)
    sizes = [t.nbytes for t in spec.tensors]
    offsets, T = oracle.plan_layout(sizes, spec.alignment)
    with binding.Checkpoint(d, index_only=True) as ck:  # the shards' order is the spec's order
        assert [t.name for t in ck.tensors()] == [t.name for t in spec.tensors]
    with binding.Pool(spec.chunk_size, -(-T // spec.chunk_size) + 1) as pool:
        pool.cache(d)
        for engine in ("kernel", "sdma"):
            with binding.Checkpoint(d, pool=pool, engine=engine) as ck:
                load_and_check(torch, ck, spec, offsets, T, digests, f"safetensors {workload} by {engine}")
        pool.evict(d)


@pytest.mark.parametrize("source", ["cached", "streamed"])
def test_copies_stop_at_arena_ends(torch_cuda, tmp_path, monkeypatch, source):
    """Pools of 1 MiB arenas holding three 320 KiB chunks each: copy-engine
    loads merge runs of chunks only inside one arena, in the file layout and
    through HBM staging at A2 = 256, and every byte still lands."""
    torch = torch_cuda
    spec = synth.stress(n=400, max_bytes=1 << 20, seed=21)
    C = 320 << 10
    d = str(tmp_path / "ck")
    digests = []

    def tensors():
        for _, t, data, dg in verify.generate(spec):
            digests.append(dg)
            yield t.name, t.dtype, t.shape, data

    binding.convert(tensors(), d, spec.alignment, C)
    sizes = [t.nbytes for t in spec.tensors]
    monkeypatch.setenv("SLLM_POOL_ARENA_MB", "1")
    offsets, T = oracle.plan_layout(sizes, spec.alignment)
    n_chunks = -(-T // C)
    with binding.Pool(C, n_chunks if source == "cached" else 24) as pool:
        if source == "cached":
            pool.cache(d)
        for A2 in (0, 256):
            offs, total = oracle.plan_layout(sizes, A2) if A2 else (offsets, T)
            kw = {} if source == "cached" else dict(ring_slots=24, io_threads=3)
            with binding.Checkpoint(d, pool=pool, engine="sdma", dev_alignment=A2, **kw) as ck:
                st = load_and_check(torch, ck, spec, offs, total, digests, f"arenas {source} A2={A2}")
                if source == "cached" and not A2:  # 3 chunks an arena: at least n/3 copies
                    assert st["n_launches"] >= -(-n_chunks // 3)
        if source == "cached":
            pool.evict(d)
