"""Host-side arithmetic of bench.py that needs no GPU: the PCI Express
capability decoding behind the link ceiling, the ceiling itself, and the
share of the repack kernel's tiles on each path (checked against a per-tile
brute force over small layouts), and where a converted workload is kept."""

import os
import random
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _config_space(cap_at=0x48, mps_code=1, mps_sup_code=2, mrrs_code=2, rcb128=True, port_type=0):
    """256 bytes of config space: a power-management capability at 0x40
    pointing to a PCI Express capability at cap_at."""
    cfg = bytearray(256)
    cfg[6:8] = (0x10).to_bytes(2, "little")       # status: capability list present
    cfg[0x34] = 0x40
    cfg[0x40], cfg[0x41] = 0x01, cap_at           # PM capability, next
    cfg[cap_at], cfg[cap_at + 1] = 0x10, 0x00     # PCI Express capability, end of list
    cfg[cap_at + 2:cap_at + 4] = (port_type << 4 | 2).to_bytes(2, "little")
    cfg[cap_at + 4:cap_at + 8] = mps_sup_code.to_bytes(4, "little")
    cfg[cap_at + 8:cap_at + 10] = (mps_code << 5 | mrrs_code << 12).to_bytes(2, "little")
    cfg[cap_at + 0x10:cap_at + 0x12] = (0x8 if rcb128 else 0).to_bytes(2, "little")
    return bytes(cfg)


def test_pcie_capability_decoding():
    got = bench.pcie_capability(_config_space())
    assert got == {"mps": 256, "mps_supported": 512, "mrrs": 512, "rcb": 128, "port_type": 0}
    got = bench.pcie_capability(_config_space(cap_at=0x70, mps_code=0, mps_sup_code=0, mrrs_code=5,
                                              rcb128=False, port_type=4))
    assert got == {"mps": 128, "mps_supported": 128, "mrrs": 4096, "rcb": 64, "port_type": 4}


def test_pcie_capability_unreadable_or_absent():
    full = _config_space()
    assert bench.pcie_capability(full[:64]) == {}            # what an unprivileged reader sees
    no_list = bytearray(full)
    no_list[6] = 0
    assert bench.pcie_capability(bytes(no_list)) == {}
    loop = bytearray(256)                                      # a capability list that points at itself
    loop[6], loop[0x34], loop[0x40], loop[0x41] = 0x10, 0x40, 0x01, 0x40
    assert bench.pcie_capability(bytes(loop)) == {}


def test_tlp_ceiling():
    encoded = 32.0 * 16 * 128 / 130 / 8                        # PCIe 5.0 x16 after 128b/130b
    assert encoded == pytest.approx(63.0154, rel=1e-5)
    assert bench.tlp_ceiling(encoded, 256) == pytest.approx(encoded * 256 / 276)
    assert bench.tlp_ceiling(encoded, 256) == pytest.approx(58.449, rel=1e-4)
    assert bench.tlp_ceiling(encoded, 128) < bench.tlp_ceiling(encoded, 256) < bench.tlp_ceiling(encoded, 512)


def _tile_paths_brute(file_off, dev_off, sizes, T2):
    """Each 8 KiB destination tile classified by looking at its 16 KiB plan
    block byte range directly."""
    straight = shifted = 0
    tiles = -(-T2 // bench.K2_TILE)
    for t in range(tiles):
        y = t * bench.K2_TILE
        b0 = (y // bench.K2_PLAN) * bench.K2_PLAN
        b1 = b0 + bench.K2_PLAN
        for o, d, s in zip(file_off, dev_off, sizes):
            if d <= b0 and b1 <= d + s:
                if (o - d) % 16 == 0:
                    straight += 1
                else:
                    shifted += 1
                break
    return tiles, straight, shifted


@pytest.mark.parametrize("A,A2", [(4096, 256), (1, 256), (16, 4096), (256, 16)])
def test_k2_tile_paths_against_brute_force(A, A2):
    rng = random.Random(A * 7 + A2)
    for _ in range(5):
        sizes = [rng.choice([0, 1, 100, 4096, 16384, 40000, 65536, 200000, 16384 * 5 + 7]) for _ in range(30)]
        file_off, _ = oracle.plan_layout(sizes, A)
        dev_off, T2 = oracle.plan_layout(sizes, A2)
        got = bench.k2_tile_paths(file_off, dev_off, sizes, T2)
        tiles, straight, shifted = _tile_paths_brute(file_off, dev_off, sizes, T2)
        assert (got["tiles"], got["straight"], got["shifted"]) == (tiles, straight, shifted)
        assert got["general"] == tiles - straight - shifted


def test_checkpoint_dir_choice(tmp_path, monkeypatch):
    """Where the bench and the full-size tests keep a converted workload:
    $SLLM_BENCH_DIR when set; else a directory that already holds a
    converted copy with the right key; else the first base whose file
    system has room (payload + a full alignment per tensor + 4 KiB + 1 GiB);
    else the first base, where the write reports the shortage."""
    from paper_2401_14351_amd import synth

    spec = synth.config("opt-125m")
    need = spec.payload_bytes + len(spec.tensors) * spec.alignment + 4096 + (1 << 30)
    a, b = str(tmp_path / "disk"), str(tmp_path / "shm")
    monkeypatch.setattr(bench, "BENCH_BASES", (a, b))
    monkeypatch.delenv("SLLM_BENCH_DIR", raising=False)
    free = {a: need, b: need}
    monkeypatch.setattr(bench, "_free_bytes", lambda p: free[p])
    assert bench.checkpoint_dir(spec) == os.path.join(a, spec.name)
    free[a] = need - 1
    assert bench.checkpoint_dir(spec) == os.path.join(b, spec.name)
    free[b] = 0
    assert bench.checkpoint_dir(spec) == os.path.join(a, spec.name)
    # a converted copy is used wherever it is, whatever the free space
    os.makedirs(os.path.join(b, spec.name))
    with open(os.path.join(b, spec.name, "bench.key"), "w") as f:
        f.write(bench.spec_key(spec))
    assert bench.checkpoint_dir(spec) == os.path.join(b, spec.name)
    monkeypatch.setenv("SLLM_BENCH_DIR", str(tmp_path / "env"))
    assert bench.checkpoint_dir(spec) == str(tmp_path / "env" / spec.name)
