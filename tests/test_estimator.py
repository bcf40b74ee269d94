"""The loading-time estimate of Sec. 6 (q + n / b, slowest tier, refined
from measured loads): hand-worked cases, host-only."""

import pytest

from paper_2401_14351_amd import binding

GB = 1e9


@pytest.fixture()
def est():
    if not __import__("os").path.exists(binding.LIB_PATH):
        pytest.skip("libsllm.so not built")
    e = binding.Estimator(50 * GB, 5 * GB, weight=0.5)
    yield e
    e.close()


def test_single_tier_and_slowest_tier(est):
    assert est.query(10 * GB, binding.TIER_DRAM) == pytest.approx(0.2)
    assert est.query(10 * GB, binding.TIER_STORAGE) == pytest.approx(2.0)
    # a pipelined file -> DRAM -> HBM load runs at the slower (storage) rate
    assert est.query(10 * GB, binding.TIER_DRAM | binding.TIER_STORAGE) == pytest.approx(2.0)


def test_queue_accumulates_and_refines(est):
    t1, eta1 = est.enqueue(10 * GB, binding.TIER_DRAM)          # 0 + 10/50
    t2, eta2 = est.enqueue(5 * GB, binding.TIER_DRAM | binding.TIER_STORAGE)   # 0.2 + 5/5
    assert eta1 == pytest.approx(0.2) and eta2 == pytest.approx(1.2)
    assert est.query(9 * GB, binding.TIER_DRAM) == pytest.approx(1.2 + 0.18)
    est.complete(t1, 0.25)                                        # measured 40 GB/s
    assert est.bandwidth(binding.TIER_DRAM) == pytest.approx(45 * GB)   # 0.5 * 50 + 0.5 * 40
    assert est.query(9 * GB, binding.TIER_DRAM) == pytest.approx(1.0 + 0.2)
    est.complete(t2, 2.0)                                         # 2.5 GB/s attributed to storage
    assert est.bandwidth(binding.TIER_STORAGE) == pytest.approx(3.75 * GB)
    assert est.bandwidth(binding.TIER_DRAM) == pytest.approx(45 * GB)
    assert est.query(0, binding.TIER_DRAM) == pytest.approx(0.0)


def test_errors(est):
    with pytest.raises(binding.SllmError) as ei:
        est.complete(99, 1.0)
    assert ei.value.code == -8
    t, _ = est.enqueue(1, binding.TIER_DRAM)
    with pytest.raises(binding.SllmError):
        est.complete(t, 0.0)
    with pytest.raises(binding.SllmError):
        est.query(1, 0)
    with pytest.raises(binding.SllmError):
        est.query(1, 4)
    with pytest.raises(binding.SllmError):
        binding.Estimator(0, 1)
    with pytest.raises(binding.SllmError):
        binding.Estimator(1, 1, weight=0)


def test_complete_load_needs_a_load(est, tmp_path):
    """A handle that has loaded nothing (an index-only open) gives no
    measurement: INVAL, and the task stays queued."""
    import numpy as np

    d = str(tmp_path / "c")
    binding.convert(iter([("w", "f32", (4,), np.arange(4, dtype=np.float32))]), d, 256, 1 << 20)
    task, _ = est.enqueue(10 * GB, binding.TIER_DRAM)
    with binding.Checkpoint(d, index_only=True) as ck:
        with pytest.raises(binding.SllmError) as e:
            est.complete_load(task, ck)
        assert e.value.code == -1
    assert est.query(0, binding.TIER_DRAM) == pytest.approx(0.2)
    est.complete(task, 0.2)
