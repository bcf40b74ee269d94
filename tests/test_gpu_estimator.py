"""The loading-time estimator (Sec. 6) fed from a load's own counters:
sllm_estimator_complete_load takes the time from the handle's stats (open
time plus the load's device time with timing on, else its host time) and
refines the bandwidth of the slowest tier the load crossed."""

import pytest

from paper_2401_14351_amd import binding, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.lib()
    return torch


def fed_seconds(st):
    return st["open_s"] + max(st["load_s"], st["device_ms"] * 1e-3 if st["device_ms"] >= 0 else 0.0)


def test_complete_load_from_stats(torch_cuda, tmp_path):
    torch = torch_cuda
    spec = synth.stress(n=200, max_bytes=1 << 20, seed=91)
    tensors = [(t.name, t.dtype, t.shape, x) for t, x in zip(spec.tensors, synth.materialize(spec))]
    d = str(tmp_path / "c")
    binding.convert(iter(tensors), d, spec.alignment, spec.chunk_size)
    est = binding.Estimator(50e9, 5e9, weight=1.0)  # weight 1: the estimate is the latest sample
    try:
        with binding.Pool(spec.chunk_size, 256) as pool:
            pool.cache(d)
            buf = None
            # cached, timed: open + device time
            with binding.Checkpoint(d, pool=pool, timing=True) as ck:
                T = ck.total_bytes
                buf = torch.empty(T, dtype=torch.uint8, device="cuda:0")
                task, _ = est.enqueue(T, binding.TIER_DRAM)
                ck.load_into(buf)
                torch.cuda.synchronize()
                st = ck.stats()
                assert st["device_ms"] > 0 and st["bytes_loaded"] == T
                est.complete_load(task, ck)
            assert est.bandwidth(binding.TIER_DRAM) == pytest.approx(T / fed_seconds(st), rel=1e-9)
            # cached, untimed: open + host time of the call
            with binding.Checkpoint(d, pool=pool) as ck:
                task, _ = est.enqueue(T, binding.TIER_DRAM)
                ck.load_into(buf)
                torch.cuda.synchronize()
                st = ck.stats()
                assert st["device_ms"] < 0
                est.complete_load(task, ck)
            assert est.bandwidth(binding.TIER_DRAM) == pytest.approx(T / (st["open_s"] + st["load_s"]), rel=1e-9)
            pool.evict(d)
        # streamed from the file: the storage tier (the slower one) is refined
        before = est.bandwidth(binding.TIER_DRAM)
        with binding.Checkpoint(d, timing=True, ring_slots=8, io_threads=2) as ck:
            task, _ = est.enqueue(T, binding.TIER_DRAM | binding.TIER_STORAGE)
            ck.load_into(buf)
            torch.cuda.synchronize()
            st = ck.stats()
            est.complete_load(task, ck)
        assert est.bandwidth(binding.TIER_STORAGE) == pytest.approx(T / fed_seconds(st), rel=1e-9)
        assert est.bandwidth(binding.TIER_DRAM) == before
        # an unknown task is refused, and a completed one cannot complete again
        with binding.Checkpoint(d, timing=True, ring_slots=8) as ck:
            ck.load_into(buf)
            torch.cuda.synchronize()
            with pytest.raises(binding.SllmError) as e:
                est.complete_load(task, ck)
            assert e.value.code == -8
    finally:
        est.close()
