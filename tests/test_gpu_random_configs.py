"""Seeded random sweep of load configurations on small checkpoints: file
alignment, device alignment, engine, cached or streamed (buffered or direct
reads, kept slots), chunk size, ring size and reader count drawn at random,
every byte of every load (and, with a device alignment, of the HBM repack
of the file-layout image) compared with the oracle's image and a sentinel
past it.  A second generator draws the library's tuning knobs for each
configuration (kernel grids and tile shapes, batch target, split reads,
read mode, copy size, pinned arena size, sometimes a chunk large enough to
be read in pieces), so that the knobs are exercised in combination; the
first generator's sequence of configurations does not depend on them.
Each configuration is printed before it runs."""

import os
import sys

import numpy as np
import pytest

import oracle
from paper_2401_14351_amd import binding, synth

pytestmark = pytest.mark.gpu

SENTINEL = 0x3C
# a longer or different sweep: SLLM_RAND_CONFIGS=5000 SLLM_RAND_SEED=7
N_CONFIGS = int(os.environ.get("SLLM_RAND_CONFIGS", "1500"))
SEED = int(os.environ.get("SLLM_RAND_SEED", "20240114"))


def say(*a):
    print("[gpu-rand]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.lib()
    return torch


def draw(rng):
    A = int(rng.choice([1, 2, 4, 16, 256, 4096]))
    A2 = int(rng.choice([0, 0, 16, 32, 256, 4096]))
    engine = str(rng.choice(["kernel", "sdma"]))
    source = str(rng.choice(["cached", "streamed", "streamed", "direct", "keep"]))
    if source == "direct":
        C = 4096 * int(rng.integers(1, 65))
    else:
        C = int(rng.choice([16, 48, 4096, 65536, 1 << 20, 16 * int(rng.integers(1, 5000)),
                            int(rng.integers(1, 100000))]))
    kind = str(rng.choice(["tiny", "stress"]))
    seed = int(rng.integers(0, 1 << 30))
    if kind == "tiny":
        spec = synth.tiny(seed, n=int(rng.integers(1, 40)), alignment=A, max_bytes=int(rng.integers(1, 200_000)))
    else:
        spec = synth.stress(n=int(rng.integers(1, 200)), seed=seed, min_bytes=1,
                            max_bytes=int(rng.integers(2, 1 << 20)))
    return dict(A=A, A2=A2, engine=engine, source=source, C=C, kind=kind, seed=seed, spec=spec,
                ring=int(rng.integers(1, 9)), io=int(rng.integers(1, 5)))


# each knob: values drawn with equal weight, None leaves the default
KNOBS = {
    "SLLM_K1_BLOCKS": [None, None, "1", "3", "2048"],
    "SLLM_K1_STREAM_BLOCKS": [None, None, "1", "5", "1024"],
    "SLLM_K1_UNROLL": [None, None, "1", "2"],
    "SLLM_K1_NT": [None, "1"],
    "SLLM_K2_NT": [None, "0"],
    "SLLM_K2_UNROLL": [None, "4"],
    "SLLM_K2_MAX_GRID": [None, None, "7", "997"],
    "SLLM_BATCH_TARGET_MB": [None, "0", "1"],
    "SLLM_SPLIT_CHUNKS": [None, "0", "1", "1000"],
    "SLLM_READ_STREAM": [None, "0"],
    "SLLM_READ_MAPPED": [None, None, "1"],
    "SLLM_SDMA_MAX_COPY_MB": [None, "1"],
    "SLLM_POOL_ARENA_MB": [None, None, "1", "3"],
}


def draw_knobs(rng):
    env = {}
    for name, values in KNOBS.items():
        v = values[int(rng.integers(0, len(values)))]
        if v is not None:
            env[name] = v
    # sometimes chunks of 2-5 MiB, which the first readers take in pieces
    big_chunk = 4096 * int(rng.integers(512, 1281)) if rng.integers(0, 4) == 0 else 0
    return env, big_chunk


def test_random_configurations(torch_cuda, tmp_path, monkeypatch):
    torch = torch_cuda
    rng = np.random.default_rng(SEED)
    knob_rng = np.random.default_rng(SEED + 1)
    for i in range(N_CONFIGS):
        cfg = draw(rng)
        env, big_chunk = draw_knobs(knob_rng)
        spec = cfg.pop("spec")
        say(i, cfg, env, "big chunk" if big_chunk else "")
        for name in KNOBS:
            monkeypatch.delenv(name, raising=False)
        for name, v in env.items():
            monkeypatch.setenv(name, v)
        tensors = [(t.name, t.dtype, t.shape, d) for t, d in zip(spec.tensors, synth.materialize(spec, threads=4))]
        A, A2 = cfg["A"], cfg["A2"]
        # at most 2048 chunks (every pool chunk takes at least 4 KiB of pinned memory)
        _, T = oracle.plan_layout([t.nbytes for t in spec.tensors], A)
        C = max(big_chunk or cfg["C"], -(-T // 2048))
        if cfg["source"] == "direct":
            C = -(-C // 4096) * 4096
        cfg["C"] = C
        say(i, "T", T, "C", C)
        d = str(tmp_path / f"c{i}")
        os.makedirs(d)
        binding.convert(iter(tensors), d, A, C)
        index = oracle.make_index(tensors, A, C)
        image = bytes(oracle.partition_bytes(tensors, A)[:index.total_bytes])
        want = bytes(oracle.repack(image, index, A2)) if A2 else image
        n_chunks = max(1, -(-index.total_bytes // C))
        pool = None
        kw = dict(engine=cfg["engine"], dev_alignment=A2)
        if cfg["source"] == "cached":
            pool = binding.Pool(C, n_chunks)
            pool.cache(d, io_threads=cfg["io"])
            kw.update(pool=pool)
        elif cfg["source"] == "keep":
            pool = binding.Pool(C, n_chunks)
            kw.update(pool=pool, cache=True, io_threads=cfg["io"])
        else:
            kw.update(chunk_size=C, ring_slots=cfg["ring"], io_threads=cfg["io"], direct_io=cfg["source"] == "direct")
        try:
            with binding.Checkpoint(d, **kw) as ck:
                assert ck.total_bytes == len(want)
                for rep in range(2):
                    buf = torch.full((len(want) + 64,), SENTINEL, dtype=torch.uint8, device="cuda:0")
                    ck.load_into(buf)
                    torch.cuda.synchronize()
                    host = buf.cpu().numpy()
                    assert (host[len(want):] == SENTINEL).all(), f"config {i}: bytes past the image written"
                    got = host[:len(want)].tobytes()
                    if got != want:
                        a = np.frombuffer(got, np.uint8)
                        b = np.frombuffer(want, np.uint8)
                        bad = np.nonzero(a != b)[0]
                        raise AssertionError(f"config {i} {cfg} load {rep}: {bad.size} bytes differ, "
                                             f"first at {bad[:8].tolist()}")
                if A2:  # the HBM repack of the file-layout image gives the same bytes
                    src = torch.frombuffer(bytearray(image + bytes(16)), dtype=torch.uint8).to("cuda:0")
                    out = torch.full((len(want) + 64,), SENTINEL, dtype=torch.uint8, device="cuda:0")
                    ck.repack(src, out)
                    torch.cuda.synchronize()
                    host = out.cpu().numpy()
                    assert (host[len(want):] == SENTINEL).all(), f"config {i}: repack wrote past the image"
                    assert host[:len(want)].tobytes() == want, f"config {i} {cfg}: repack differs"
        finally:
            if pool is not None:
                if cfg["source"] in ("cached", "keep") and pool.info()["cached_checkpoints"]:
                    pool.evict(d)
                pool.close()
