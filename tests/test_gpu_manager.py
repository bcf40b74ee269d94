"""A model manager's use of one shared pinned pool, from several threads at
once (Sec. 4.2: the pool is the DRAM tier that the loading of many models
shares; chunks are allocated and freed under the application's control).

Eight threads each run a seeded random sequence of operations over four small
checkpoints that share one chunk size: open a handle (either engine, file
layout or a 256-byte device layout, streaming through pool chunks or
caching what it reads) and load it once or twice on a stream of its own,
cache a checkpoint in the pool, or evict one.  Every load is compared byte
for byte with the oracle's image.  The pool's refusals that such a mix
makes legitimate are accepted: no free chunks (NOMEM), already cached or in
use (BUSY), not cached (NOTFOUND); any other error fails the test.  At the
end every chunk is back in the pool."""

import sys
import threading

import numpy as np
import pytest

import oracle
from paper_2401_14351_amd import binding, synth

pytestmark = pytest.mark.gpu

C = 64 << 10
ALLOWED = {-4, -7, -8}  # NOMEM, BUSY, NOTFOUND


def say(*a):
    print("[gpu-manager]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.lib()
    return torch


def checkpoints(tmp_path):
    specs = [synth.tiny(11, n=30, alignment=256, max_bytes=60_000),
             synth.tiny(12, n=7, alignment=1, max_bytes=200_000),
             synth.stress(n=150, seed=13, min_bytes=1, max_bytes=8_000),
             synth.tiny(14, n=3, alignment=4096, max_bytes=5_000)]
    out = []
    for i, spec in enumerate(specs):
        A = spec.alignment
        tensors = [(t.name, t.dtype, t.shape, d) for t, d in zip(spec.tensors, synth.materialize(spec, threads=4))]
        d = str(tmp_path / f"m{i}")
        binding.convert(iter(tensors), d, A, C)
        index = oracle.make_index(tensors, A, C)
        image = bytes(oracle.partition_bytes(tensors, A)[:index.total_bytes])
        out.append((d, {0: image, 256: bytes(oracle.repack(image, index, 256))}))
        say("checkpoint", i, "T", index.total_bytes, "chunks", -(-index.total_bytes // C))
    return out


def test_threads_share_one_pool(torch_cuda, tmp_path):
    torch = torch_cuda
    ckpts = checkpoints(tmp_path)
    counts = {"loads": 0, "cached": 0, "evicted": 0, "refused": 0}
    errors = []
    lock = threading.Lock()

    def note(key):
        with lock:
            counts[key] += 1

    def attempt(fn):
        try:
            fn()
            return True
        except binding.SllmError as e:
            if e.code not in ALLOWED:
                raise
            note("refused")
            return False

    with binding.Pool(C, 40) as pool:
        def worker(tid):
            rng = np.random.default_rng(1000 + tid)
            stream = torch.cuda.Stream()
            try:
                for step in range(150):
                    d, want = ckpts[int(rng.integers(0, len(ckpts)))]
                    op = int(rng.integers(0, 6))
                    if op == 4:
                        if attempt(lambda: pool.cache(d, io_threads=int(rng.integers(1, 4)))):
                            note("cached")
                        continue
                    if op == 5:
                        if attempt(lambda: pool.evict(d)):
                            note("evicted")
                        continue
                    A2 = int(rng.choice([0, 256]))
                    kw = dict(pool=pool, engine=str(rng.choice(["kernel", "sdma"])), dev_alignment=A2,
                              io_threads=int(rng.integers(1, 4)), ring_slots=int(rng.integers(1, 5)),
                              cache=bool(rng.integers(0, 2)))
                    ck = None
                    try:
                        ck = binding.Checkpoint(d, **kw)
                    except binding.SllmError as e:
                        if e.code not in ALLOWED:
                            raise
                        note("refused")
                        continue
                    with ck:
                        for _ in range(int(rng.integers(1, 3))):
                            buf = torch.empty(len(want[A2]), dtype=torch.uint8, device="cuda:0")
                            if not attempt(lambda: ck.load_into(buf, stream)):
                                break
                            stream.synchronize()
                            got = buf.cpu().numpy().tobytes()
                            assert got == want[A2], f"thread {tid} step {step} {d} {kw}: image differs"
                            note("loads")
            except Exception as e:  # noqa: BLE001
                errors.append((tid, repr(e)))
                say("thread", tid, "failed:", repr(e))

        threads = [threading.Thread(target=worker, args=(t,)) for t in range(8)]
        for t in threads:
            t.start()
        for t in threads:
            t.join()
        say(counts)
        assert not errors, errors
        for d, _ in ckpts:
            attempt(lambda: pool.evict(d))
        info = pool.info()
        assert info["cached_checkpoints"] == 0
        assert info["free_chunks"] == info["n_chunks"]
    assert counts["loads"] > 300 and counts["cached"] > 0 and counts["evicted"] > 0
