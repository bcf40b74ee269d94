"""Every-byte check of a loaded device image against the input generator.

Not part of the load path: the tests and the benchmark use it to show that
a device image holds the generator's bytes of every tensor at the offsets
they are given, zeros in every other byte of ``[0, total)``, and nothing
else.  The offsets come from the caller (the tests take them from the
oracle's layout plan, the benchmark from the library's own index).

A tensor's digest is the xxh3-128 digest of the concatenated xxh3-128
digests of its generation blocks (``synth.BLOCK`` elements each, the last
one short; a tensor with no bytes has no blocks).  The blocks are hashed on
many threads, both as the generator makes them (so a checkpoint's digests
come out of its conversion for free) and as the device's bytes come back.
Two images with equal digests differ with probability about 2^-128 per
tensor; padding bytes are compared with zero directly.
"""

from __future__ import annotations

import os
from collections import deque
from concurrent.futures import ThreadPoolExecutor
from typing import Iterator, List, Optional, Sequence, Tuple

import numpy as np
import xxhash

from . import synth

DIGEST_FILE = "digests.xxh3"
DIGEST_BYTES = 16


def combine(block_digests: Sequence[bytes]) -> bytes:
    return xxhash.xxh3_128(b"".join(block_digests)).digest()


def _hash(a: np.ndarray) -> bytes:
    return xxhash.xxh3_128(memoryview(a)).digest()


def _fill_and_hash(spec, i: int, t, b: int, out: np.ndarray) -> bytes:
    synth.fill_block(spec, i, t, b, out)
    return _hash(out)


def _n_blocks(nbytes: int, step: int) -> int:
    return (nbytes + step - 1) // step


def generate(spec, threads: Optional[int] = None, indices: Optional[Sequence[int]] = None,
             lookahead: int = 1 << 30) -> Iterator[Tuple[int, object, np.ndarray, bytes]]:
    """Yield ``(i, spec_i, bytes_i, digest_i)`` in order.  Blocks of the next
    tensors are generated and hashed ahead, on a thread pool, while the
    caller consumes the current one (up to ``lookahead`` bytes in flight)."""
    idx = list(range(len(spec.tensors))) if indices is None else list(indices)
    pending: deque = deque()
    in_flight = 0
    nxt = 0
    with ThreadPoolExecutor(threads or synth.default_threads()) as pool:
        while nxt < len(idx) or pending:
            while nxt < len(idx) and (not pending or in_flight < lookahead):
                i = idx[nxt]
                nxt += 1
                t = spec.tensors[i]
                out = np.empty(t.nbytes, dtype=np.uint8)
                step = synth.block_size(t)
                futs = [pool.submit(_fill_and_hash, spec, i, t, b, out[b * step:(b + 1) * step])
                        for b in range(_n_blocks(t.nbytes, step))]
                pending.append((i, t, out, futs))
                in_flight += t.nbytes
            i, t, out, futs = pending.popleft()
            digest = combine([f.result() for f in futs])
            in_flight -= t.nbytes
            yield i, t, out, digest


def generated_digests(spec, threads: Optional[int] = None) -> List[bytes]:
    """Digests of every tensor, generated on a thread pool (no bytes kept)."""
    jobs = []
    for i, t in enumerate(spec.tensors):
        step = synth.block_size(t)
        for b in range(_n_blocks(t.nbytes, step)):
            jobs.append((i, b, min(step, t.nbytes - b * step)))

    def job(j):
        i, b, n = j
        out = np.empty(n, dtype=np.uint8)
        return _fill_and_hash(spec, i, spec.tensors[i], b, out)

    per: List[List[bytes]] = [[] for _ in spec.tensors]
    with ThreadPoolExecutor(threads or synth.default_threads()) as pool:
        for (i, _, _), d in zip(jobs, pool.map(job, jobs, chunksize=4)):
            per[i].append(d)
    return [combine(p) for p in per]


def save_digests(ckpt_dir: str, key: str, digests: Sequence[bytes]) -> None:
    path = os.path.join(ckpt_dir, DIGEST_FILE)
    with open(path + ".tmp", "wb") as f:
        f.write(key.encode() + b"\n")
        f.write(b"".join(digests))
    os.replace(path + ".tmp", path)


def load_digests(ckpt_dir: str, key: str, n: int) -> Optional[List[bytes]]:
    """The digests stored beside a converted checkpoint, if they belong to
    the same generator recipe (``key``) and tensor count."""
    path = os.path.join(ckpt_dir, DIGEST_FILE)
    try:
        blob = open(path, "rb").read()
    except OSError:
        return None
    head, _, body = blob.partition(b"\n")
    if head.decode(errors="replace") != key or len(body) != n * DIGEST_BYTES:
        return None
    return [body[k * DIGEST_BYTES:(k + 1) * DIGEST_BYTES] for k in range(n)]


class Mismatch(AssertionError):
    pass


def check_image(torch, buf, spec, offsets: Sequence[int], total: int, digests: Sequence[bytes],
                window: int = 512 << 20, threads: Optional[int] = None) -> dict:
    """Compare every byte of ``buf[0:total)`` (a uint8 device tensor) with
    the image the offsets define: tensor i of ``spec`` (its generator bytes,
    whose digest is ``digests[i]``) at ``offsets[i]``, zero everywhere else.
    Offsets must be in layout order with non-overlapping slots inside
    ``[0, total)``.

    The image comes back in windows that end at a tensor boundary, copied on
    a side stream into pinned host buffers while the previous window is
    hashed.  Raises :class:`Mismatch` naming the first wrong tensor (with its
    first differing bytes, from the regenerated tensor) or padding range.
    Returns counts of what was compared."""
    sizes = [t.nbytes for t in spec.tensors]
    n = len(sizes)
    if len(offsets) != n or len(digests) != n:
        raise ValueError("offsets, tensors and digests differ in length")
    prev_end = 0
    for i in range(n):
        if offsets[i] < prev_end or offsets[i] + sizes[i] > total:
            raise ValueError(f"tensor {i}: slot [{offsets[i]}, {offsets[i] + sizes[i]}) is out of order or past "
                             f"the image")
        prev_end = offsets[i] + sizes[i]
    if buf.numel() < total:
        raise ValueError(f"buffer holds {buf.numel()} bytes, the image {total}")

    # windows [start, end) covering [0, total): whole tensors and the padding after them
    wins: List[Tuple[int, int, int, int]] = []  # (start, end, first tensor, last tensor + 1)
    i = 0
    start = 0
    while i < n:
        j = i + 1
        while j < n and offsets[j] + sizes[j] - start <= window:
            j += 1
        end = offsets[j] if j < n else total
        wins.append((start, end, i, j))
        start, i = end, j
    if start < total or not wins:
        wins.append((start, total, n, n))
    cap = max(e - s for s, e, _, _ in wins)
    if cap == 0:
        return {"tensors": n, "bytes": 0, "padding_bytes": 0, "windows": 0}

    on_gpu = buf.device.type == "cuda"  # a CPU tensor is read in place (host-side tests of the checker)
    if on_gpu:
        host = [torch.empty(cap, dtype=torch.uint8, pin_memory=True) for _ in range(2)]
        done = [torch.cuda.Event(), torch.cuda.Event()]
        side = torch.cuda.Stream(device=buf.device)
        side.wait_stream(torch.cuda.current_stream(buf.device))
    pad_bytes = 0

    def fetch(k: int) -> None:
        if not on_gpu:
            return
        s, e, _, _ = wins[k]
        with torch.cuda.stream(side):
            host[k % 2][:e - s].copy_(buf[s:e], non_blocking=True)
            done[k % 2].record(side)

    def window_bytes(k: int) -> np.ndarray:
        s, e, _, _ = wins[k]
        if not on_gpu:
            return buf[s:e].numpy()
        done[k % 2].synchronize()
        if k + 1 < len(wins):  # the other buffer was consumed in the previous round
            fetch(k + 1)
        return host[k % 2].numpy()[:e - s]

    def fail_tensor(m: int, got: np.ndarray) -> None:
        want = synth.tensor_bytes(spec, m)
        bad = np.nonzero(got != want)[0]
        raise Mismatch(f"{spec.tensors[m].name}: device bytes at [{offsets[m]}, {offsets[m] + sizes[m]}) differ "
                       f"from the generator's ({bad.size} bytes, first at {bad[:4].tolist()})")

    with ThreadPoolExecutor(threads or synth.default_threads()) as pool:
        fetch(0)
        for k, (s, e, i0, i1) in enumerate(wins):
            h = window_bytes(k)
            jobs = []  # (tensor, block futures)
            gaps = []
            cur = s
            for m in range(i0, i1):
                a, z = offsets[m] - s, offsets[m] + sizes[m] - s
                if offsets[m] > cur:
                    gaps.append((cur - s, a))
                step = synth.block_size(spec.tensors[m])
                futs = [pool.submit(_hash, h[a + b * step:min(a + (b + 1) * step, z)])
                        for b in range(_n_blocks(sizes[m], step))]
                jobs.append((m, futs))
                cur = offsets[m] + sizes[m]
            if e > cur:
                gaps.append((cur - s, e - s))
            for a, z in gaps:
                pad_bytes += z - a
                nz = np.flatnonzero(h[a:z])
                if nz.size:
                    raise Mismatch(f"padding [{s + a}, {s + z}) holds {nz.size} non-zero bytes, first at "
                                   f"{s + a + int(nz[0])}")
            for m, futs in jobs:
                if combine([f.result() for f in futs]) != digests[m]:
                    fail_tensor(m, h[offsets[m] - s:offsets[m] + sizes[m] - s].copy())
    if on_gpu:
        torch.cuda.current_stream(buf.device).wait_stream(side)
    return {"tensors": n, "bytes": total, "padding_bytes": pad_bytes, "windows": len(wins)}
