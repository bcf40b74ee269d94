"""Checkpoint-load benchmark: host DRAM -> HBM GB/s and time-to-ready for the
Llama-2-7B-shaped bf16 checkpoint (13.48 GB, 291 tensors, 256 B alignment,
16 MiB chunks) on one MI355X.

One step is the whole warm-DRAM path of a load: sllm_open (index read and
validation, attach to the partition cached in the pinned chunk pool),
sllm_load (the chunk-gather kernel moves every chunk from mapped pinned host
memory into the preallocated HBM buffer on the caller's stream), the tensor
views at base + offset, and the stream synchronization that makes them ready.
Setup (synthetic checkpoint, conversion, pinned pool, DRAM-tier fill, the HBM
buffer) is outside the timed region, as in a model manager that has
preallocated its pool and buffers.

Prints one JSON line.  Extra fields: the peaks measured in the same run
(pinned->HBM copy engine, HBM copy), the kernel's own GB/s from HIP events on
its stream, and the CPU oracle reader timed on one host core.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import shutil
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2401_14351_amd import binding, synth, verify  # noqa: E402

METRIC = "checkpoint load GB/s host DRAM→HBM + time-to-ready (s), 7B-shaped bf16"
PCIE_GEN5_X16_GBPS = 64.0   # MI355X host link: PCIe 5.0 x16, 32 GT/s x 16 lanes per direction
HBM_PEAK_GBPS = 8000.0      # MI355X HBM3E
DATA = {"llama": "synthetic (seeded N(0,0.02) bf16 weights, RMSNorm weights 1.0)",
        "opt-125m": "synthetic (seeded N(0,0.02) fp16 weights)",
        "stress": "synthetic (seeded uniform random bytes, f32/f16/bf16/i8 tensors)",
        "lora": "synthetic (seeded N(0,0.02) bf16 LoRA A/B matrices)",
        "huge-tensor": "synthetic (seeded uniform random bytes; one int8 tensor over 4 GiB)"}
REGIME = {"dram": "warm host DRAM (pinned pool)",
          "ring": "file through pinned ring slots (buffered reads)",
          "direct": "file through pinned ring slots (O_DIRECT reads)"}


def kernel_source_hash(*sources: str) -> str:
    """SHA-256 over the kernel's source files (csrc/), in the order given."""
    h = hashlib.sha256()
    for name in sources:
        h.update(open(os.path.join(ROOT, "paper_2401_14351_amd", "csrc", name), "rb").read())
    return h.hexdigest()


def profiled_counters(summary: str, *sources: str):
    """Counter figures recorded in profiles/<summary> ('counters: {json}' line),
    or None when that file is missing or the kernel's sources (the .hip file
    and the header that shapes its arguments) have changed since the counters
    were taken (their SHA-256 no longer matches)."""
    path = os.path.join(ROOT, "profiles", summary)
    if not os.path.exists(path):
        return None
    rec = None
    for line in open(path):
        if line.startswith("counters: "):
            rec = json.loads(line[len("counters: "):])
    if rec is None:
        return None
    return rec if kernel_source_hash(*sources) == rec.get("source_sha256") else None


K1_SOURCES = ("kernels.hip", "kernels.hpp")
K2_SOURCES = ("layout.hip", "device_layout.hpp")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def spec_key(spec) -> str:
    h = hashlib.sha256()
    h.update(f"{spec.name}/{spec.seed}/{spec.alignment}/{spec.chunk_size}/{synth.BLOCK}".encode())
    for t in spec.tensors:
        h.update(f"{t.name}:{t.dtype}:{t.shape}:{t.init};".encode())
    return h.hexdigest()[:16]


BENCH_BASES = ("/tmp/sllm_bench", "/dev/shm/sllm_bench")


def _free_bytes(path: str) -> int:
    """Free bytes of the file system that holds `path` (or its nearest
    existing parent)."""
    while path and not os.path.exists(path):
        path = os.path.dirname(path)
    try:
        return shutil.disk_usage(path or "/").free
    except OSError:
        return 0


def checkpoint_dir(spec) -> str:
    """Where the converted workload lives: under $SLLM_BENCH_DIR if set;
    else where a converted copy already is; else the first of /tmp and
    /dev/shm whose file system has room for it (an upper bound: payload plus
    a full alignment per tensor plus the 4 KiB tail, and 1 GiB to spare), so
    that a small local disk does not stop the larger workloads."""
    env = os.environ.get("SLLM_BENCH_DIR")
    if env:
        return os.path.join(env, spec.name)
    key = spec_key(spec)
    for base in BENCH_BASES:
        marker = os.path.join(base, spec.name, "bench.key")
        if os.path.exists(marker):
            with open(marker) as f:
                if f.read() == key:
                    return os.path.join(base, spec.name)
    need = spec.payload_bytes + len(spec.tensors) * spec.alignment + 4096 + (1 << 30)
    for base in BENCH_BASES:
        d = os.path.join(base, spec.name)
        # a partial copy of this workload there will be overwritten: count it as free
        have = _free_bytes(base) + (_dir_bytes(d) if os.path.isdir(d) else 0)
        if have >= need:
            return d
    return os.path.join(BENCH_BASES[0], spec.name)  # the write reports what is missing


def _dir_bytes(d: str) -> int:
    total = 0
    for f in os.listdir(d):
        try:
            total += os.path.getsize(os.path.join(d, f))
        except OSError:
            pass
    return total


def ensure_checkpoint(spec, d: str):
    """Generate and convert the synthetic checkpoint unless it already
    exists; return the digests of its tensors' generator bytes (computed
    while converting, or regenerated if a converted copy has none)."""
    marker = os.path.join(d, "bench.key")
    key = spec_key(spec)
    have_key = None
    if os.path.exists(marker):
        with open(marker) as f:
            have_key = f.read()
    if have_key == key:
        digests = verify.load_digests(d, key, len(spec.tensors))
        if digests is None:
            t0 = time.time()
            digests = verify.generated_digests(spec)
            verify.save_digests(d, key, digests)
            log(f"digests of {spec.name} regenerated in {time.time() - t0:.1f} s")
        return digests
    os.makedirs(d, exist_ok=True)
    if os.path.exists(marker):
        os.remove(marker)
    t0 = time.time()
    digests = []

    def tensors():
        for _, t, data, dg in verify.generate(spec):
            digests.append(dg)
            yield t.name, t.dtype, t.shape, data

    binding.convert(tensors(), d, spec.alignment, spec.chunk_size, fsync=True)
    verify.save_digests(d, key, digests)
    with open(marker, "w") as f:
        f.write(key)
    log(f"converted {spec.name} into {d} in {time.time() - t0:.1f} s")
    return digests


def measure_peaks(torch, nbytes: int = 1 << 30, reps: int = 5, streams=(1, 2, 4)):
    """The pinned->HBM copy-engine peak: best of `reps` copies of `nbytes`
    split evenly over 1, 2 and 4 streams (one hipMemcpyAsync per stream,
    timed from a fork on the current stream to the join of them all), and
    the best HBM->HBM copy.  Returns (best H2D GB/s, {streams: GB/s}, HBM GB/s)."""
    host = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    dev = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    dev2 = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    s = torch.cuda.current_stream()
    side = [torch.cuda.Stream() for _ in range(max(streams))]
    joins = [torch.cuda.Event() for _ in side]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    by_streams = {}
    for k in streams:
        part = -(-nbytes // k)
        best = 0.0
        for _ in range(reps):
            e0.record(s)
            for j in range(k):
                a, b = j * part, min(nbytes, (j + 1) * part)
                side[j].wait_event(e0)
                with torch.cuda.stream(side[j]):
                    dev[a:b].copy_(host[a:b], non_blocking=True)
                joins[j].record(side[j])
                s.wait_event(joins[j])
            e1.record(s)
            e1.synchronize()
            best = max(best, nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e9)
        by_streams[k] = round(best, 3)
    d2d = 0.0
    for _ in range(reps):
        e0.record(s)
        dev2.copy_(dev)
        e1.record(s)
        e1.synchronize()
        d2d = max(d2d, 2 * nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del host, dev, dev2
    return max(by_streams.values()), by_streams, d2d


def host_info():
    """Cores this process may use, CPU model and NUMA node count of the host."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        nodes = [n for n in os.listdir("/sys/devices/system/node") if n.startswith("node") and n[4:].isdigit()]
    except OSError:
        nodes = []
    return {"nproc": len(os.sched_getaffinity(0)), "cpu_count": os.cpu_count(), "cpu_model": model,
            "numa_nodes": len(nodes) or None, "gpu_links": gpu_links()}


def gpu_links():
    """PCIe link (speed, width) of each AMD GPU, from sysfs: the host link
    that bounds every DRAM -> HBM transfer."""
    out = []
    base = "/sys/class/drm"
    try:
        cards = sorted(c for c in os.listdir(base) if c.startswith("card") and c[4:].isdigit())
    except OSError:
        return out
    for c in cards:
        dev = os.path.join(base, c, "device")

        def read(name):
            try:
                return open(os.path.join(dev, name)).read().strip()
            except OSError:
                return None

        if read("vendor") != "0x1002":
            continue
        out.append({"pci": os.path.basename(os.path.realpath(dev)), "speed": read("current_link_speed"),
                    "width": read("current_link_width"), "max_speed": read("max_link_speed"),
                    "max_width": read("max_link_width")})
    return out


def pcie_capability(cfg: bytes) -> dict:
    """Max Payload Size (set and supported), Max Read Request Size, Read
    Completion Boundary and port type from a PCI function's config space
    bytes: the PCI Express capability (ID 0x10) found by walking the
    capability list.  Empty when the bytes do not reach it."""
    u16 = lambda o: int.from_bytes(cfg[o:o + 2], "little")
    u32 = lambda o: int.from_bytes(cfg[o:o + 4], "little")
    if len(cfg) < 64 or not u16(6) & 0x10:  # no capability list
        return {}
    ptr, seen = cfg[0x34] & 0xFC, 0
    while ptr and ptr + 0x14 <= len(cfg) and seen < 48:
        if cfg[ptr] == 0x10:
            devcap, devctl, lnkctl = u32(ptr + 4), u16(ptr + 8), u16(ptr + 0x10)
            return {"mps": 128 << ((devctl >> 5) & 7), "mps_supported": 128 << (devcap & 7),
                    "mrrs": 128 << ((devctl >> 12) & 7), "rcb": 128 if lnkctl & 0x8 else 64,
                    "port_type": (u16(ptr + 2) >> 4) & 0xF}
        ptr, seen = cfg[ptr + 1] & 0xFC, seen + 1
    return {}


def pcie_function(bdf: str):
    """pcie_capability of one PCI function from sysfs; `readable` is the
    number of config bytes this process may read (64 without privileges,
    too few to reach the capability)."""
    try:
        cfg = open(f"/sys/bus/pci/devices/{bdf}/config", "rb").read()
    except OSError as e:
        return {"bdf": bdf, "readable": 0, "error": str(e)}
    return {"bdf": bdf, "readable": len(cfg), **pcie_capability(cfg)}


def pcie_path(bdf: str):
    """pcie_function for the GPU and every bridge above it, GPU first."""
    try:
        parts = os.path.realpath(f"/sys/bus/pci/devices/{bdf}").split("/")
    except OSError:
        return []
    path = [c for c in parts if len(c) == 12 and c[4] == ":" and c[7] == ":" and c[10] == "."]
    return [pcie_function(b) for b in reversed(path)]


def tlp_ceiling(gen5_lanes_gbps: float, payload: int, overhead: int = 20) -> float:
    """Data rate of a link carrying only completions of `payload` bytes: each
    adds `overhead` bytes (4-byte framing token with the sequence number,
    12-byte completion header, 4-byte LCRC) on the 128b/130b-encoded lanes.
    Flow-control and acknowledgement packets and SKP ordered sets are not
    counted, so the real ceiling sits a little lower."""
    return gen5_lanes_gbps * payload / (payload + overhead)


def pcie_ceiling():
    """The host link's data ceiling for transfers into the GPU, derived from
    what sysfs reports: lanes x rate after line encoding (128b/130b from
    8 GT/s on), less the per-completion overhead at the smallest Max Payload
    Size on the path from the root port to the GPU.  Where this process may
    not read that far into config space, 256-byte payloads are assumed (and
    the record says so)."""
    links = gpu_links()
    if not links:
        return None
    g = links[0]
    try:
        rate = float(str(g["speed"]).split()[0])
        width = int(g["width"])
    except (TypeError, ValueError):
        return {"link": g}
    encoded = rate * width * (128 / 130 if rate >= 8 else 0.8) / 8
    path = pcie_path(g["pci"])
    mps = [f["mps"] for f in path if "mps" in f]
    payload = min(mps) if mps else 256
    return {"link": f"{g['speed']} x{g['width']}", "encoded_GBps": round(encoded, 3), "path": path,
            "payload": payload, "payload_source": "Max Payload Size on the path (config space)" if mps else
            "assumed: config space past 64 bytes is not readable without privileges",
            "tlp_ceiling_GBps": round(tlp_ceiling(encoded, payload), 3)}


def cpu_baseline(d: str, budget_s: float):
    """The oracle reader on one host core over a bounded prefix of the same file."""
    import oracle

    index = oracle.read_index(d)
    C = index.chunk_size
    n_all = -(-index.total_bytes // C)
    prev = os.sched_getaffinity(0)
    core = min(prev)
    os.sched_setaffinity(0, {core})
    try:
        # grow the sample until one read of it takes about budget_s / 2
        k = min(8, n_all)
        while True:
            t0 = time.perf_counter()
            oracle.read(d, C, max_chunks=k)
            dt = time.perf_counter() - t0
            if dt >= budget_s / 2 or k == n_all:
                break
            k = min(n_all, max(k + 1, int(k * min(8.0, budget_s / 2 / max(dt, 1e-3)))))
        # a whole file that reads faster than that: time several passes over it
        passes = 1
        if k == n_all and dt < budget_s / 2:
            passes = 0
            t0 = time.perf_counter()
            while passes < 2 or time.perf_counter() - t0 < budget_s * 0.7:
                oracle.read(d, C, max_chunks=k)
                passes += 1
            dt = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, prev)
    nbytes = min(k * C, index.total_bytes) * passes
    what = f"first {k} of {n_all} chunks" if passes == 1 else f"{passes} passes over all {n_all} chunks"
    return {"value": round(nbytes / dt / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"oracle chunked reader (file -> host buffer, page cache warm), {what} "
                      f"({nbytes / 1e9:.2f} GB) in {dt:.1f} s on one core",
            "host": host_info()}


def storage_peak(path: str, block: int = 4 << 20, depth: int = 32, budget_s: float = 4.0):
    """Direct sequential reads of `block` bytes with `depth` requests in flight
    (the storage peak the paper measures with FIO: 4 MiB, direct, depth 32),
    over the checkpoint's own data file.  None if the file system refuses
    O_DIRECT."""
    import itertools
    import mmap
    import threading

    try:
        fd = os.open(path, os.O_RDONLY | os.O_DIRECT)
    except OSError:
        return None
    try:
        nblocks = os.fstat(fd).st_size // block
        if nblocks == 0:
            return None
        counter = itertools.count()
        total = [0] * depth
        deadline = time.perf_counter() + budget_s

        def worker(i):
            buf = mmap.mmap(-1, block)
            while time.perf_counter() < deadline:
                k = next(counter) % nblocks
                total[i] += os.preadv(fd, [buf], k * block)

        t0 = time.perf_counter()
        threads = [threading.Thread(target=worker, args=(i,)) for i in range(depth)]
        for t in threads:
            t.start()
        for t in threads:
            t.join()
        dt = time.perf_counter() - t0
        return {"GBps": round(sum(total) / dt / 1e9, 3), "block": block, "depth": depth,
                "bytes": sum(total), "device": block_device(path)}
    finally:
        os.close(fd)


def timeline_summary(path: str, T: int):
    """The streamed pipeline's timeline (written by the library under
    SLLM_TRACE_FILE) reduced to a few figures per load, then averaged: the
    share of the load's span during which some reader is reading, during
    which the GPU holds chunks (moved and not yet seen done), during which
    both happen, the mean reads and GPU-held chunks in flight, the time to
    the first move and the drain after the last read."""
    import csv
    from collections import defaultdict

    def union(iv):
        tot, cs, ce = 0.0, None, None
        for s, e in sorted(iv):
            if cs is None:
                cs, ce = s, e
            elif s <= ce:
                ce = max(ce, e)
            else:
                tot += ce - cs
                cs, ce = s, e
        return tot + (ce - cs if cs is not None else 0.0)

    def both(a, b):
        ev = sorted([(s, 0, 1) for s, _ in a] + [(e, 0, -1) for _, e in a] +
                    [(s, 1, 1) for s, _ in b] + [(e, 1, -1) for _, e in b])
        count, last, tot = [0, 0], None, 0.0
        for t, w, d in ev:
            if last is not None and count[0] > 0 and count[1] > 0:
                tot += t - last
            count[w] += d
            last = t
        return tot

    loads = defaultdict(lambda: defaultdict(dict))
    for r in csv.DictReader(open(path)):
        loads[r["load"]][int(r["chunk"])][r["event"]] = float(r["t_s"])
    per = []
    for chunks in loads.values():
        reads = [(c["read_begin"], c["read_end"]) for c in chunks.values()]
        gpu = [(c["moved"], c["done"]) for c in chunks.values()]
        t0, t1 = min(s for s, _ in reads), max(e for _, e in gpu)
        span = t1 - t0
        per.append({"span_ms": span * 1e3, "GBps": T / span / 1e9,
                    "reading_pct": 100 * union(reads) / span, "gpu_holding_pct": 100 * union(gpu) / span,
                    "both_pct": 100 * both(reads, gpu) / span,
                    "reads_in_flight": sum(e - s for s, e in reads) / span,
                    "chunks_on_gpu": sum(e - s for s, e in gpu) / span,
                    "first_move_ms": (min(s for s, _ in gpu) - t0) * 1e3,
                    "drain_ms": (t1 - max(e for _, e in reads)) * 1e3})
    return {"loads": len(per), "chunks": len(next(iter(loads.values()))) if loads else 0,
            **{k: round(statistics.mean(p[k] for p in per), 2) for k in per[0]}} if per else None


def estimator_online(d, open_kw, buf, stream, T, tiers, dram_bps, storage_bps, loads: int = 10):
    """The loading-time estimator in use (Sec. 6): before each load its time
    is estimated (q + n / b, sllm_estimator_enqueue); the load runs on a
    handle opened with timing; then sllm_estimator_complete_load refines b
    from that handle's own counters (open time plus the load's device time).
    Reports how far each estimate was from the load's time-to-ready measured
    around open, load and synchronize."""
    est = binding.Estimator(dram_bps, storage_bps, weight=0.5)
    err, fed = [], []
    for _ in range(loads):
        task, eta = est.enqueue(T, tiers)
        t0 = time.perf_counter()
        with binding.Checkpoint(d, timing=True, **open_kw) as ck:
            ck.load_into(buf, stream)
            stream.synchronize()
            ready = time.perf_counter() - t0
            est.complete_load(task, ck)
            st = ck.stats()
        err.append(abs(eta - ready))
        fed.append(st["open_s"] + max(st["load_s"], st["device_ms"] * 1e-3))
    tail = err[len(err) // 2:]
    out = {"loads": loads, "fed_from": "sllm_get_stats of each load's handle (open_s + device time)",
           "mean_abs_err_ms": round(statistics.mean(tail) * 1e3, 3), "max_abs_err_ms": round(max(tail) * 1e3, 3),
           "first_err_ms": round(err[0] * 1e3, 3), "mean_fed_s": round(statistics.mean(fed), 5),
           "dram_GBps": round(est.bandwidth(binding.TIER_DRAM) / 1e9, 3),
           "storage_GBps": round(est.bandwidth(binding.TIER_STORAGE) / 1e9, 3)}
    est.close()
    return out


def ablation(torch, spec, d: str, digests, io_threads: int = 8):
    """The paper's loading ladder (Sec. 7.2, performance breakdown) rebuilt on
    this machine: each rung loads the same partition file into one HBM
    buffer and adds one technique to the rung before it.  Rungs 1-5 are
    plain host code (torch copies), rung 6 is this library's streamed
    pipeline.  Before each rung the buffer is filled with a sentinel; after
    it every byte is checked against the generator's bytes."""
    import errno
    import mmap
    import threading

    import numpy as np

    path = os.path.join(d, "sllm.part0")
    with binding.Checkpoint(d, index_only=True) as ck:
        tensors, T = ck.tensors(), ck.total_bytes
    offsets = [t.offset for t in tensors]
    C = spec.chunk_size
    dev = torch.empty(T, dtype=torch.uint8, device="cuda:0")
    bounced = [False]

    def cold():
        fd = os.open(path, os.O_RDONLY)
        os.posix_fadvise(fd, 0, 0, os.POSIX_FADV_DONTNEED)
        os.close(fd)

    def read_by_tensor():
        # one read per tensor into a fresh pageable buffer, one copy per tensor
        fd = os.open(path, os.O_RDONLY)
        for t in tensors:
            b = os.pread(fd, t.nbytes, t.offset)
            if t.nbytes:
                dev[t.offset:t.offset + t.nbytes].copy_(torch.frombuffer(bytearray(b), dtype=torch.uint8))
        os.close(fd)

    def chunked(direct: bool, threads: int, pinned: bool):
        # C-byte chunk reads (a shared counter hands out chunk numbers), each
        # copied to the GPU by the thread that read it: from a pageable
        # buffer (the runtime stages it), or from the thread's pinned buffer
        # (DMA straight from it).  Direct reads into pinned memory that the
        # kernel refuses (EFAULT) land in a page-aligned bounce buffer first.
        fd = os.open(path, os.O_RDONLY | (os.O_DIRECT if direct else 0))
        size = os.fstat(fd).st_size
        n = -(-T // C)
        counter = iter(range(n))
        lock = threading.Lock()
        errors = []

        def worker():
            try:
                bounce = mmap.mmap(-1, C)  # page-aligned, pageable
                host = torch.frombuffer(bounce, dtype=torch.uint8)
                pin = torch.empty(C, dtype=torch.uint8, pin_memory=True) if pinned else None
                pin_view = memoryview(pin.numpy()) if pinned else None
                while True:
                    with lock:
                        k = next(counter, None)
                    if k is None:
                        return
                    want = min(C, size - k * C)
                    m = min(C, T - k * C)
                    if pinned:
                        try:
                            got = os.preadv(fd, [pin_view[:want]], k * C)
                        except OSError as e:
                            if e.errno != errno.EFAULT:
                                raise
                            bounced[0] = True
                            got = os.preadv(fd, [memoryview(bounce)[:want]], k * C)
                            pin[:m].copy_(host[:m])
                        src = pin
                    else:
                        got = os.preadv(fd, [memoryview(bounce)[:want]], k * C)
                        src = host
                    if got < m:
                        raise OSError(f"short read of chunk {k}: {got} of {m} bytes")
                    dev[k * C:k * C + m].copy_(src[:m])
            except BaseException as e:  # reported by the caller
                errors.append(e)

        ts = [threading.Thread(target=worker) for _ in range(threads)]
        for t in ts:
            t.start()
        for t in ts:
            t.join()
        os.close(fd)
        if errors:
            raise errors[0]

    def pipeline():
        with binding.Pool(C, 4 * io_threads) as pool:
            with binding.Checkpoint(d, pool=pool, direct_io=True, io_threads=io_threads,
                                    ring_slots=4 * io_threads) as ck:
                ck.load_into(dev)
                torch.cuda.synchronize()

    rungs = [("ReadByTensor", True, read_by_tensor),
             ("+bulk (16 MiB chunk reads)", True, lambda: chunked(False, 1, False)),
             ("+direct I/O", False, lambda: chunked(True, 1, False)),
             (f"+{io_threads} I/O threads", False, lambda: chunked(True, io_threads, False)),
             ("+pinned memory (copies from pinned chunks)", False, lambda: chunked(True, io_threads, True)),
             ("+pipeline (streamed ring)", False, pipeline)]
    out, prev = [], None
    for name, needs_cold, fn in rungs:
        dev.fill_(0x5A)
        if needs_cold:
            cold()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        fn()
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        gbps = T / dt / 1e9
        got = verify.check_image(torch, dev, spec, offsets, T, digests)
        out.append({"rung": name, "s": round(dt, 3), "GBps": round(gbps, 3),
                    "step_gain": None if prev is None else round(gbps / prev, 2),
                    "verified": f"every byte ({got['tensors']} tensors, {got['bytes']} bytes)"})
        prev = gbps
        log("ablation", out[-1])
    del dev
    return out, {"direct_reads_into_pinned_memory": "refused (EFAULT): bounced" if bounced[0] else "accepted"}


def thread_sweep(d: str, C: int, threads=(1, 2, 4, 8, 16)):
    """The storage -> pinned DRAM stage alone (filling the chunk pool from the
    partition file, no device work) with 1 to 16 I/O threads: direct reads
    from a dropped cache, then buffered reads from a warm page cache.  The
    paper finds a few cores enough to saturate its storage (Sec. 7.2)."""
    path = os.path.join(d, "sllm.part0")
    with binding.Checkpoint(d, index_only=True) as ck:
        T = ck.total_bytes
    out = {"direct": [], "buffered": []}
    with binding.Pool(C, -(-T // C)) as pool:
        for mode in ("direct", "buffered"):
            fd = os.open(path, os.O_RDONLY)
            if mode == "direct":
                os.posix_fadvise(fd, 0, 0, os.POSIX_FADV_DONTNEED)
            else:
                while os.read(fd, 64 << 20):  # warm the page cache
                    pass
            os.close(fd)
            for k in threads:
                t0 = time.perf_counter()
                pool.cache(d, io_threads=k, direct_io=mode == "direct")
                dt = time.perf_counter() - t0
                pool.evict(d)
                out[mode].append({"io_threads": k, "s": round(dt, 3), "GBps": round(T / dt / 1e9, 3)})
                log("thread sweep", mode, out[mode][-1])
    return out


def block_device(path: str) -> str:
    """Name and kind of the block device holding `path` (from sysfs)."""
    try:
        st = os.stat(path)
        dev = f"{os.major(st.st_dev)}:{os.minor(st.st_dev)}"
        name = os.path.basename(os.path.realpath(f"/sys/dev/block/{dev}"))
        rot = open(f"/sys/class/block/{name}/queue/rotational").read().strip() if os.path.exists(
            f"/sys/class/block/{name}/queue/rotational") else "?"
        kind = "NVMe" if name.startswith("nvme") else "virtio" if name.startswith("vd") else "other"
        return f"{name} ({kind}, rotational={rot})"
    except OSError:
        return "unknown"


K2_TILE = 8192    # bytes of the device image per K2 workgroup
K2_PLAN = 16384   # bytes of the device image per entry of K2's plan


def k2_tile_paths(file_off, dev_off, sizes, T2):
    """How K2's tiles split between its paths for a whole-image repack: a tile
    whose plan block lies inside one tensor's data copies straight (source
    and destination agree mod 16) or through the byte funnel (they do not);
    every other tile (tensor edges, padding, small tensors) takes the staged
    general path."""
    import numpy as np

    o = np.asarray(file_off, dtype=np.int64)
    dv = np.asarray(dev_off, dtype=np.int64)
    s = np.asarray(sizes, dtype=np.int64)
    blocks = np.maximum(0, (dv + s) // K2_PLAN - (-(-dv // K2_PLAN)))
    tiles = blocks * (K2_PLAN // K2_TILE)
    aligned = (o - dv) % 16 == 0
    total = -(-T2 // K2_TILE)
    straight, shifted = int(tiles[aligned].sum()), int(tiles[~aligned].sum())
    return {"tiles": total, "straight": straight, "shifted": shifted, "general": total - straight - shifted,
            "straight_frac": round(straight / total, 4) if total else None,
            "shifted_frac": round(shifted / total, 4) if total else None,
            "general_frac": round((total - straight - shifted) / total, 4) if total else None}


def measure_k2(torch, workload: str, dev_alignment: int, stream, reps: int = 6, verify_image: bool = True):
    """K2 on a repack that moves bytes: the workload's file-layout image,
    loaded into HBM through a pinned ring, repacked into alignment
    `dev_alignment` by sllm_repack `reps` times (the first untimed), each
    timed with HIP events on the stream K2 runs on; then every byte of the
    result is checked against the generator's bytes."""
    spec = synth.config(workload)
    d = checkpoint_dir(spec)
    digests = ensure_checkpoint(spec, d)
    with binding.Checkpoint(d, index_only=True) as ck:
        T, file_off = ck.total_bytes, [t.offset for t in ck.tensors()]
    with binding.Checkpoint(d, index_only=True, dev_alignment=dev_alignment) as ck:
        T2, dev_off = ck.total_bytes, [t.offset for t in ck.tensors()]
    sizes = [t.nbytes for t in spec.tensors]
    src = torch.empty(T, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty(T2, dtype=torch.uint8, device="cuda:0")
    slots = max(16, (1 << 30) // spec.chunk_size)
    with binding.Pool(spec.chunk_size, slots) as ring:
        with binding.Checkpoint(d, pool=ring, io_threads=8, ring_slots=slots) as ck:
            ck.load_into(src, stream)
            stream.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ms = []
    with binding.Checkpoint(d, dev_alignment=dev_alignment, ring_slots=2, io_threads=1) as ck:
        for i in range(reps):
            e0.record(stream)
            ck.repack(src, dst, stream)
            e1.record(stream)
            e1.synchronize()
            if i:
                ms.append(e0.elapsed_time(e1))
    gbps = (T + T2) / (statistics.mean(ms) * 1e-3) / 1e9
    summary = f"k2_tiles_repack_{workload}.md"
    k2c = profiled_counters(summary, *K2_SOURCES)
    out = {"workload": spec.name, "tensors": len(sizes), "alignment": spec.alignment, "dev_alignment": dev_alignment,
           "bytes_read": T, "bytes_written": T2, "padding_written": T2 - sum(sizes),
           "kernel_ms": round(statistics.mean(ms), 3), "kernel_ms_min": round(min(ms), 3),
           "achieved_GBps": round(gbps, 1), "bound": "hbm", "peak": HBM_PEAK_GBPS,
           "frac_hbm_peak": round(gbps / HBM_PEAK_GBPS, 4),
           "traffic": (k2c["fetch_bytes_per_launch"] + k2c["write_bytes_per_launch"]) if k2c else None,
           "traffic_profile": f"profiles/{summary}" if k2c else None,
           "tile_paths": k2_tile_paths(file_off, dev_off, sizes, T2)}
    if verify_image:
        t0 = time.perf_counter()
        got = verify.check_image(torch, dst, spec, dev_off, T2, digests)
        out["parity"] = {"checked": "every byte of the repacked image", **got, "s": round(time.perf_counter() - t0, 2)}
    del src, dst
    torch.cuda.empty_cache()
    return out


def measure_extras(torch, spec, d, pool, buf, stream, engine):
    """Other engines and tiers on the same checkpoint (outside the graded
    step).  Each extra runs on its own: one that fails (a full disk, say)
    records its error and leaves the others and the graded line intact."""
    out = {}
    T = buf.numel()

    def attempt(name, fn):
        try:
            out[name] = fn()
            log(f"{name}:", out[name])
        except Exception as e:  # noqa: BLE001
            out[name] = {"error": f"{type(e).__name__}: {e}"}
            log(f"{name} failed: {e}")

    # the copy-engine path from the same cached chunks
    other = "sdma" if engine == "kernel" else "kernel"

    def other_engine():
        times = []
        for i in range(6):
            t0 = time.perf_counter()
            with binding.Checkpoint(d, pool=pool, engine=other) as ck:
                ck.load_into(buf, stream)
                stream.synchronize()
            if i:
                times.append(time.perf_counter() - t0)
        return {"time_to_ready_s": round(statistics.median(times), 5),
                "GBps": round(T / statistics.median(times) / 1e9, 3)}

    attempt(f"engine_{other}", other_engine)
    # K2 on repacks that move bytes: the 8 GiB stress prefix (4 KiB file
    # alignment, padding after most tensors) into A2 = 256, and the same
    # tensors packed densely (A = 1), whose shifts need the byte funnel
    attempt("repack_k2", lambda: measure_k2(torch, "stress-8g", 256, stream))
    attempt("repack_k2_dense", lambda: measure_k2(torch, "stress-8g-dense", 256, stream))

    # the 7B image into A2 = 4 KiB: every 7B tensor is a multiple of 8 KiB,
    # so that layout equals the file layout and K2 only copies (an upper
    # bound, every tile straight)
    def identity_copy():
        with binding.Checkpoint(d, pool=pool, dev_alignment=4096) as ck:
            T2 = ck.total_bytes
            dst = torch.empty(T2, dtype=torch.uint8, device="cuda:0")
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            ms = []
            for i in range(6):
                e0.record(stream)
                ck.repack(buf, dst, stream)
                e1.record(stream)
                e1.synchronize()
                if i:
                    ms.append(e0.elapsed_time(e1))
            del dst
        k2 = (T + T2) / (statistics.mean(ms) * 1e-3) / 1e9
        k2c = profiled_counters("k2_tiles_repack_llama-2-7b.md", *K2_SOURCES)
        return {"workload": spec.name, "dev_alignment": 4096, "bytes_read": T, "bytes_written": T2,
                "note": "identity layout (every tensor a multiple of 8 KiB): a copy, not a relocation",
                "kernel_ms": round(statistics.mean(ms), 3), "achieved_GBps": round(k2, 1), "bound": "hbm",
                "peak": HBM_PEAK_GBPS, "frac_hbm_peak": round(k2 / HBM_PEAK_GBPS, 4),
                "traffic": (k2c["fetch_bytes_per_launch"] + k2c["write_bytes_per_launch"]) if k2c else None}

    attempt("repack_k2_identity_copy", identity_copy)

    # streamed from the file with direct I/O through a 1 GiB ring, 16 readers
    # (cold: O_DIRECT bypasses the page cache), next to the storage device's
    # own peak measured the way the paper normalizes storage bandwidth
    def direct_ring():
        slots = max(16, (1 << 30) // spec.chunk_size)
        with binding.Pool(spec.chunk_size, slots) as ring_pool:
            with binding.Checkpoint(d, pool=ring_pool, engine=engine, direct_io=True, io_threads=16,
                                    ring_slots=slots) as ck:
                t0 = time.perf_counter()
                ck.load_into(buf, stream)
                stream.synchronize()
                dt = time.perf_counter() - t0
                st = ck.stats()
        peak = storage_peak(os.path.join(d, "sllm.part0"))
        return {"GBps": round(T / dt / 1e9, 3), "s": round(dt, 3), "direct_io": int(st["direct_io"]),
                "io_threads": 16, "ring_slots": slots, "read_wait_s": round(st["read_wait_s"], 3),
                "device": block_device(d), "storage_peak_GBps": peak["GBps"] if peak else None}

    attempt("file_direct_ring", direct_ring)

    # the tiers in one pass: a first load straight from the file (O_DIRECT)
    # that leaves the partition cached in the pool (SLLM_OPEN_CACHE), then a
    # load of the same handle from that cache
    def direct_then_cached():
        pool.evict(d)
        try:
            t0 = time.perf_counter()
            with binding.Checkpoint(d, pool=pool, engine=engine, cache=True, direct_io=True, io_threads=16) as ck:
                ck.load_into(buf, stream)
                stream.synchronize()
                t1 = time.perf_counter()
                first = ck.stats()
                ck.load_into(buf, stream)
                stream.synchronize()
                t2 = time.perf_counter()
                second = ck.stats()
        finally:
            if not pool.info()["cached_checkpoints"]:  # leave the partition cached, as found
                pool.cache(d)
        return {"first_GBps": round(T / (t1 - t0) / 1e9, 3), "first_s": round(t1 - t0, 3),
                "first_from_cache": int(first["from_cache"]), "second_GBps": round(T / (t2 - t1) / 1e9, 3),
                "second_from_cache": int(second["from_cache"]), "cached_after": pool.info()["cached_checkpoints"]}

    attempt("file_direct_then_cached", direct_then_cached)

    # the one-time conversion (Sec. 4.1; reported, not graded): the first
    # tensors of the workload, about 1 GiB held in memory, written by the
    # batch converter and by the streaming writer, each with fsync, on the
    # checkpoint's file system if it has room for both copies
    def convert():
        import tempfile

        k, nbytes = 0, 0
        while k < len(spec.tensors) and nbytes < (1 << 30):
            nbytes += spec.tensors[k].nbytes
            k += 1
        need = 2 * (nbytes + k * spec.alignment + 4096) + (1 << 30)
        bases = [os.path.dirname(os.path.abspath(d))] + list(BENCH_BASES)
        base = next((b for b in bases if _free_bytes(b) >= need), None)
        if base is None:
            return {"skipped": f"no file system with {need} bytes free for the two copies"}
        os.makedirs(base, exist_ok=True)
        sub = [(t.name, t.dtype, t.shape, data) for _, t, data in synth.iter_tensors(spec, indices=range(k))]
        tmp = tempfile.mkdtemp(dir=base)
        try:
            t0 = time.perf_counter()
            binding.convert_array(sub, os.path.join(tmp, "batch"), spec.alignment, spec.chunk_size, fsync=True)
            t_batch = time.perf_counter() - t0
            t0 = time.perf_counter()
            binding.convert(iter(sub), os.path.join(tmp, "stream"), spec.alignment, spec.chunk_size, fsync=True)
            t_stream = time.perf_counter() - t0
        finally:
            shutil.rmtree(tmp, ignore_errors=True)
        return {"tensors": k, "bytes": nbytes, "batch_GBps": round(nbytes / t_batch / 1e9, 3),
                "streaming_GBps": round(nbytes / t_stream / 1e9, 3), "fsync": True, "device": block_device(base)}

    attempt("convert", convert)
    return out


def calibration_copy(torch):
    """One 1 GiB HBM -> HBM copy: the kernel whose counter readings scale
    FETCH_SIZE and WRITE_SIZE to bytes."""
    a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda:0")
    b = torch.empty(1 << 30, dtype=torch.uint8, device="cuda:0")
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    log("calibration copy: 1 GiB HBM -> HBM")


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama-2-7b",
                    choices=list(synth.WORKLOADS) + ["stress-8g", "stress-8g-dense", "lora-70b-r32", "huge-tensor"])
    ap.add_argument("--engine", default="kernel", choices=["kernel", "sdma"])
    ap.add_argument("--regime", default="dram", choices=["dram", "ring", "direct"],
                    help="dram: partition cached in the pinned pool (graded); ring: streamed from the file "
                         "through pinned slots (buffered reads); direct: the same with O_DIRECT reads")
    ap.add_argument("--chunk-size", type=int, default=0, help="chunk size in bytes (default: the workload's)")
    ap.add_argument("--dev-alignment", type=int, default=0,
                    help="load into a device layout with this alignment (K1-scatter, or copy engine + K2)")
    ap.add_argument("--io-threads", type=int, default=8)
    ap.add_argument("--ring-slots", type=int, default=0,
                    help="pinned ring slots for streamed regimes (default: 1 GiB of slots, at least 16)")
    ap.add_argument("--dir", default=None, help="where the converted checkpoint lives")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle reading")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-peaks", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the copy-engine, repack and cold direct-read measurements")
    ap.add_argument("--no-verify", action="store_true", help="skip the sampled parity check")
    ap.add_argument("--ablation", action="store_true",
                    help="run the paper's loading ladder (per-tensor reads ... pipeline) on the file instead")
    ap.add_argument("--thread-sweep", action="store_true",
                    help="time the file -> pinned pool stage alone with 1-16 I/O threads instead")
    ap.add_argument("--trace", default=None,
                    help="streamed regimes: write the timed loads' pipeline timeline (CSV) to this file and "
                         "summarize it (tracing waits for each load's last batches)")
    ap.add_argument("--repack-only", action="store_true",
                    help="time and check only the HBM repack (K2) of --workload into --dev-alignment (default 256)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="end with one 1 GiB HBM->HBM copy (the counter calibration kernel)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU: this loader has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    if args.repack_only:
        import torch

        torch.cuda.init()
        stream = torch.cuda.Stream()
        k2 = measure_k2(torch, args.workload, args.dev_alignment or 256, stream, reps=args.steps + 1)
        print(json.dumps({"repack_k2": k2}), flush=True)
        if args.calib_copy:
            calibration_copy(torch)
        return

    spec = synth.config(args.workload)
    d = args.dir or checkpoint_dir(spec)
    digests = ensure_checkpoint(spec, d)
    cpu = None if args.no_cpu_baseline else cpu_baseline(d, args.cpu_budget)  # before any GPU work
    if cpu:
        log("cpu baseline:", cpu["sample"], cpu["value"], "GB/s")

    import torch

    torch.cuda.init()
    if args.ablation:
        ladder, notes = ablation(torch, spec, d, digests, args.io_threads)
        base = ladder[0]["GBps"]
        sweep = thread_sweep(d, args.chunk_size or spec.chunk_size)
        print(json.dumps({"ablation": ladder, "workload": spec.name,
                          "io_threads": args.io_threads, "device": block_device(d),
                          "storage_peak": storage_peak(os.path.join(d, "sllm.part0")),
                          "total_gain": round(ladder[-1]["GBps"] / base, 2), **notes,
                          "thread_sweep": sweep, "host": host_info()}), flush=True)
        return
    if args.thread_sweep:
        sweep = thread_sweep(d, args.chunk_size or spec.chunk_size)
        print(json.dumps({"thread_sweep": sweep, "workload": spec.name, "device": block_device(d),
                          "storage_peak": storage_peak(os.path.join(d, "sllm.part0")), "host": host_info()}),
              flush=True)
        return
    stream = torch.cuda.Stream()
    h2d_peak, h2d_by_streams, hbm_peak = (None, None, None) if args.no_peaks else measure_peaks(torch)
    log(f"measured peaks: pinned->HBM copy {h2d_peak} GB/s (by streams {h2d_by_streams}), HBM copy {hbm_peak} GB/s")

    C = args.chunk_size or spec.chunk_size
    if not args.ring_slots:
        args.ring_slots = max(16, (1 << 30) // C)
    with binding.Checkpoint(d, index_only=True, dev_alignment=args.dev_alignment) as probe:
        T = probe.total_bytes
    with binding.Checkpoint(d, index_only=True) as probe:
        T_file = probe.total_bytes
    n_chunks = -(-T_file // C)
    cached = args.regime == "dram"
    t0 = time.time()
    pool = binding.Pool(C, n_chunks if cached else args.ring_slots)
    pool_alloc_s = time.time() - t0
    log(f"pinned pool: {n_chunks if cached else args.ring_slots} x {C / 2**20:g} MiB in {pool_alloc_s:.1f} s")
    fill_s = None
    if cached:
        t0 = time.time()
        pool.cache(d, io_threads=args.io_threads)
        fill_s = time.time() - t0
        log(f"DRAM tier filled in {fill_s:.1f} s")
    open_kw = dict(pool=pool, engine=args.engine, dev_alignment=args.dev_alignment)
    if not cached:
        open_kw.update(chunk_size=C, io_threads=args.io_threads, ring_slots=args.ring_slots,
                       direct_io=args.regime == "direct")
    t0 = time.perf_counter()
    buf = torch.empty(T, dtype=torch.uint8, device="cuda:0")
    torch.cuda.synchronize()
    hbm_alloc_s = time.perf_counter() - t0
    last_stats = {}

    ev0 = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ev1 = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ready, loads, open_s = [], [], []

    def step(i=None):
        t_open = time.perf_counter()
        ck = binding.Checkpoint(d, **open_kw)
        t_load = time.perf_counter()
        if i is not None:
            ev0[i].record(stream)
        # the views are built while the load runs (sllm_load on a helper thread)
        views = ck.load_with_views(buf, stream, after_load=None if i is None else lambda: ev1[i].record(stream))
        stream.synchronize()
        t_end = time.perf_counter()
        last_stats.update(ck.stats())
        open_s.append(last_stats["open_s"])
        ck.close()
        return t_end - t_open, t_end - t_load, views

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    tracing = bool(args.trace) and not cached
    if tracing:
        if os.path.exists(args.trace):
            os.remove(args.trace)
        os.environ["SLLM_TRACE_FILE"] = os.path.abspath(args.trace)
    t_start = time.perf_counter()
    for i in range(args.steps):
        r, l, views = step(i)
        ready.append(r)
        loads.append(l)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    if tracing:
        os.environ.pop("SLLM_TRACE_FILE", None)

    # after timing, every byte of the last step's image: each tensor's bytes
    # at the offset the library's index gives equal the generator's, every
    # other byte of [0, T) is zero
    del views
    parity = None
    if not args.no_verify:
        with binding.Checkpoint(d, index_only=True, dev_alignment=args.dev_alignment) as probe:
            offsets = [t.offset for t in probe.tensors()]
        t0 = time.perf_counter()
        try:
            got = verify.check_image(torch, buf, spec, offsets, T, digests)
        except verify.Mismatch as e:
            raise SystemExit(f"bench: the loaded image differs from the generator's bytes: {e}")
        parity = {"checked": "every byte of the last timed step's image", **got,
                  "s": round(time.perf_counter() - t0, 2)}
        log("parity:", parity)
    extras = ({} if (args.no_extras or not cached or args.dev_alignment) else
              measure_extras(torch, spec, d, pool, buf, stream, args.engine))
    # one-time set-up outside time-to-ready, as a model manager that keeps its
    # pinned pool and HBM buffer pays it once
    extras["setup"] = {"pinned_pool_alloc_s": round(pool_alloc_s, 3), "hbm_buffer_alloc_s": round(hbm_alloc_s, 4)}
    if fill_s is not None:
        extras["dram_tier_fill"] = {"GBps": round(T / fill_s / 1e9, 3), "s": round(fill_s, 3),
                                    "io_threads": args.io_threads, "source": "converted file, page cache warm"}
    storage = None
    if not cached and args.regime == "direct":
        storage = storage_peak(os.path.join(d, "sllm.part0"))
        extras["storage_peak"] = storage
    tiers = binding.TIER_DRAM | (0 if cached else binding.TIER_STORAGE)
    try:
        extras["estimator"] = estimator_online(d, open_kw, buf, stream, T, tiers, (h2d_peak or 50.0) * 1e9,
                                               (storage["GBps"] if storage else 5.0) * 1e9,
                                               loads=10 if cached else 3)
    except Exception as e:  # noqa: BLE001  (an extra: the graded line still prints)
        extras["estimator"] = {"error": f"{type(e).__name__}: {e}"}
        log(f"estimator failed: {e}")
    if tracing:
        extras["timeline"] = timeline_summary(args.trace, T)
    if not cached:
        extras["ring"] = {"io_threads": args.io_threads, "ring_slots": args.ring_slots,
                          "direct_io": int(last_stats.get("direct_io", 0)),
                          "bytes_read": int(last_stats.get("bytes_read", 0)),
                          "bytes_bounced": int(last_stats.get("bytes_bounced", 0)),
                          "chunks": int(last_stats.get("n_chunks", 0)),
                          "launches": int(last_stats.get("n_launches", 0)),
                          "read_wait_s": round(last_stats.get("read_wait_s", 0.0), 4),
                          "reader_busy_s": round(last_stats.get("reader_busy_s", 0.0), 3),
                          "reader_starved_s": round(last_stats.get("reader_starved_s", 0.0), 3),
                          "device": block_device(d)}

    link = pcie_ceiling()
    kernel_ms = [a.elapsed_time(b) for a, b in zip(ev0, ev1)]
    k_avg_s = statistics.mean(kernel_ms) * 1e-3
    achieved = T / k_avg_s / 1e9
    value = T * args.steps / elapsed / 1e9
    k1_counters = (profiled_counters("k1_gather_llama-2-7b.md", *K1_SOURCES)
                   if cached and args.engine == "kernel" and spec.name == "llama-2-7b" and C == 16 << 20
                   and not args.dev_alignment else None)
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": next((v for k, v in DATA.items() if spec.name.startswith(k)), DATA["llama"]),
        "config": {"workload": spec.name, "bytes": T, "tensors": len(spec.tensors), "chunk_size": C,
                   "alignment": spec.alignment, "dev_alignment": args.dev_alignment, "engine": args.engine,
                   "regime": REGIME[args.regime]},
        "time_to_ready_s": round(statistics.median(ready), 5),
        "time_to_ready_min_s": round(min(ready), 5),
        "load_GBps": round(T / statistics.median(loads) / 1e9, 3),
        "load_GBps_best": round(T / min(loads) / 1e9, 3),
        "open_ms": round(statistics.median(open_s[-args.steps:]) * 1e3, 3),
        "roofline": {"bound": "pcie", "achieved": round(achieved, 3), "peak": PCIE_GEN5_X16_GBPS, "unit": "GB/s",
                     "frac": round(achieved / PCIE_GEN5_X16_GBPS, 4),
                     "traffic": k1_counters["fetch_bytes_per_launch"] if k1_counters else None,
                     "traffic_write": k1_counters["write_bytes_per_launch"] if k1_counters else None,
                     "algorithmic_bytes": T,
                     "kernel": ("k1_gather" if cached and args.engine == "kernel" and not args.dev_alignment else
                                "k_scatter (host source)" if cached and args.engine == "kernel" else
                                "whole load on the caller's stream (events around sllm_load)"),
                     "kernel_ms": round(statistics.mean(kernel_ms), 3),
                     "peak_measured": None if h2d_peak is None else round(h2d_peak, 3),
                     "peak_measured_by_streams": h2d_by_streams,
                     "frac_measured": None if h2d_peak is None else round(achieved / h2d_peak, 4),
                     "tlp_ceiling": None if not (link and "tlp_ceiling_GBps" in link) else link["tlp_ceiling_GBps"],
                     "frac_tlp_ceiling": None if not (link and "tlp_ceiling_GBps" in link) else
                     round(achieved / link["tlp_ceiling_GBps"], 4),
                     "pcie": link,
                     "hbm_copy_measured": None if hbm_peak is None else round(hbm_peak, 1),
                     "link": next((f"{g['speed']} x{g['width']}" for g in gpu_links()), None)},
        "cpu_baseline": cpu,
        "parity": parity,
        "extras": extras,
    }
    print(json.dumps(out), flush=True)
    if cached:
        pool.evict(d)
    pool.close()
    if args.calib_copy:
        del buf
        calibration_copy(torch)


if __name__ == "__main__":
    main()
