"""CPU oracle for the loading-optimized checkpoint format and its loader.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the tests, the ``smoke()`` check and the benchmark's
CPU-baseline leg use it.  It shares no code with the GPU path (no kernels,
headers, helpers or tables) and imports nothing from the package.

It is the plain definition of what the method computes, written to be read
against the paper:

* Sec. 4.1 (loading-optimized checkpoints): a checkpoint is converted once
  into a per-GPU partition file that holds only the tensors' binary data,
  grouped for large sequential reads, plus a tensor index that maps each
  tensor name to (GPU id, offset, size).  Tensors sit at offsets aligned to a
  memory word size, so a tensor's device address is base + offset.
* Sec. 4.2 (multi-tier loading subsystem): the partition is read in
  fixed-size chunks and those chunks are copied into one GPU buffer.

Readings of points the paper leaves open (each one is listed with its reason
in the design notes of the repository):

1. Tensors keep the caller's order (the paper allows any order).
2. The alignment ``A`` is a parameter, a power of two >= 1.
3. Padding bytes are 0x00, in the file and on the device.
4. The partition file has no header: the first tensor starts at byte 0.
5. The file is zero-padded to ``F = align_up(T, 4096)`` bytes so that
   direct (O_DIRECT) reads of whole blocks stay inside it.
6. Chunk k covers bytes ``[kC, min(kC + C, T))``; the last chunk is short and
   tensors may straddle chunks.
7. The index also records dtype and shape (the paper keeps those in the model
   execution files); ``size`` is the unpadded byte size.
8. One partition (GPU id 0).
9. Zero-size tensors take no bytes and no padding; a 0-d tensor holds one
   element.
10. A device layout may use its own alignment ``A2``: the same closed form with
    ``A2`` in place of ``A``, zero padding.

Index encoding (all little-endian, packed)::

    magic "SLLMIDX1" | u32 version=1 | u32 n_partitions=1 | u64 A | u64 C |
    u64 T | u64 F | u64 n |
    n x ( u32 name_len | name (UTF-8) | u8 dtype | u8 ndim | u16 partition |
          i64 shape[ndim] | u64 offset | u64 nbytes ) |
    u32 CRC-32 (IEEE, as zlib.crc32) of every preceding byte

dtype codes: 0 f32, 1 f16, 2 bf16, 3 i8.
"""

from __future__ import annotations

import math
import os
import struct
import zlib
from dataclasses import dataclass
from typing import List, Sequence, Tuple

MAGIC = b"SLLMIDX1"
VERSION = 1
FILE_BLOCK = 4096           # reading 5: the data file is padded to a multiple of this
INDEX_NAME = "sllm.index"
DATA_NAME = "sllm.part0"    # partition 0: the only GPU of this loader
DTYPE_CODE = {"f32": 0, "f16": 1, "bf16": 2, "i8": 3}
CODE_DTYPE = {v: k for k, v in DTYPE_CODE.items()}
ITEMSIZE = {"f32": 4, "f16": 2, "bf16": 2, "i8": 1}
MAX_NDIM = 8
MAX_NAME = 65535


class OracleError(ValueError):
    pass


@dataclass(frozen=True)
class Entry:
    """One row of the tensor index (Sec. 4.1: name -> GPU id, offset, size)."""
    name: str
    dtype: str
    shape: Tuple[int, ...]
    partition: int
    offset: int
    nbytes: int


@dataclass(frozen=True)
class Index:
    alignment: int
    chunk_size: int
    total_bytes: int
    file_bytes: int
    entries: Tuple[Entry, ...]


# --------------------------------------------------------------------------
# layout (Sec. 4.1, "direct tensor addressing")
# --------------------------------------------------------------------------

def align_up(x: int, a: int) -> int:
    """Smallest multiple of ``a`` that is >= ``x``."""
    return -(-x // a) * a


def is_pow2(a: int) -> bool:
    return a >= 1 and (a & (a - 1)) == 0


def plan_layout(sizes: Sequence[int], alignment: int) -> Tuple[List[int], int]:
    """Offsets of tensors packed in order at ``alignment``-aligned offsets.

    Tensor i starts where the previous tensor's padded slot ends:
    ``o_i = sum_{j<i} align_up(s_j, A)``; the total is ``T = sum_i align_up(s_i, A)``.
    """
    if not is_pow2(alignment):
        raise OracleError(f"alignment {alignment} is not a power of two >= 1")
    offsets = []
    cursor = 0
    for s in sizes:
        if s < 0:
            raise OracleError("negative size")
        offsets.append(cursor)
        cursor += align_up(s, alignment)
    return offsets, cursor


def file_length(total: int) -> int:
    """Length of the partition file: T rounded up to whole 4 KiB blocks."""
    return align_up(total, FILE_BLOCK)


# --------------------------------------------------------------------------
# validation of the conversion input
# --------------------------------------------------------------------------

def _numel(shape: Sequence[int]) -> int:
    return math.prod(shape)


def validate(tensors, alignment: int, chunk_size: int) -> None:
    """``tensors``: sequence of (name, dtype, shape, data) with ``data`` bytes-like."""
    if not is_pow2(alignment):
        raise OracleError(f"alignment {alignment} is not a power of two >= 1")
    if chunk_size < 1:
        raise OracleError("chunk size must be >= 1")
    seen = set()
    for name, dtype, shape, data in tensors:
        raw = name.encode("utf-8")
        if not raw or len(raw) > MAX_NAME:
            raise OracleError(f"bad name length for {name!r}")
        if name in seen:
            raise OracleError(f"duplicate tensor name {name!r}")
        seen.add(name)
        if dtype not in DTYPE_CODE:
            raise OracleError(f"unknown dtype {dtype!r}")
        if len(shape) > MAX_NDIM or any(d < 0 for d in shape):
            raise OracleError(f"bad shape {shape!r} for {name!r}")
        if len(memoryview(data).cast("B")) != _numel(shape) * ITEMSIZE[dtype]:
            raise OracleError(f"size of {name!r} does not match its shape and dtype")


# --------------------------------------------------------------------------
# conversion (Sec. 4.1): partition file + tensor index
# --------------------------------------------------------------------------

def partition_bytes(tensors, alignment: int) -> bytearray:
    """The whole partition file ``P[0:F)``: each tensor's bytes at its offset,
    every other byte zero."""
    sizes = [len(memoryview(d).cast("B")) for _, _, _, d in tensors]
    offsets, total = plan_layout(sizes, alignment)
    P = bytearray(file_length(total))
    for (_, _, _, data), o, s in zip(tensors, offsets, sizes):
        P[o:o + s] = memoryview(data).cast("B")
    return P


def make_index(tensors, alignment: int, chunk_size: int) -> Index:
    sizes = [len(memoryview(d).cast("B")) for _, _, _, d in tensors]
    offsets, total = plan_layout(sizes, alignment)
    entries = tuple(Entry(n, dt, tuple(int(x) for x in sh), 0, o, s)
                    for (n, dt, sh, _), o, s in zip(tensors, offsets, sizes))
    return Index(alignment, chunk_size, total, file_length(total), entries)


def encode_index(index: Index) -> bytes:
    out = bytearray()
    out += MAGIC
    out += struct.pack("<II", VERSION, 1)
    out += struct.pack("<QQQQQ", index.alignment, index.chunk_size, index.total_bytes,
                       index.file_bytes, len(index.entries))
    for e in index.entries:
        raw = e.name.encode("utf-8")
        out += struct.pack("<I", len(raw)) + raw
        out += struct.pack("<BBH", DTYPE_CODE[e.dtype], len(e.shape), e.partition)
        out += struct.pack(f"<{len(e.shape)}q", *e.shape)
        out += struct.pack("<QQ", e.offset, e.nbytes)
    out += struct.pack("<I", zlib.crc32(bytes(out)) & 0xFFFFFFFF)
    return bytes(out)


def decode_index(blob: bytes) -> Index:
    if len(blob) < 60:
        raise OracleError("index too short")
    body, (crc,) = blob[:-4], struct.unpack("<I", blob[-4:])
    if zlib.crc32(body) & 0xFFFFFFFF != crc:
        raise OracleError("index CRC mismatch")
    if body[:8] != MAGIC:
        raise OracleError("bad magic")
    version, nparts = struct.unpack_from("<II", body, 8)
    if version != VERSION or nparts != 1:
        raise OracleError("unsupported version or partition count")
    A, C, T, F, n = struct.unpack_from("<QQQQQ", body, 16)
    pos = 56
    entries = []
    for _ in range(n):
        (ln,) = struct.unpack_from("<I", body, pos)
        pos += 4
        name = body[pos:pos + ln].decode("utf-8")
        pos += ln
        code, ndim, part = struct.unpack_from("<BBH", body, pos)
        pos += 4
        shape = struct.unpack_from(f"<{ndim}q", body, pos)
        pos += 8 * ndim
        off, nb = struct.unpack_from("<QQ", body, pos)
        pos += 16
        entries.append(Entry(name, CODE_DTYPE[code], tuple(shape), part, off, nb))
    if pos != len(body):
        raise OracleError("trailing bytes in index")
    return Index(A, C, T, F, tuple(entries))


def convert(tensors, out_dir: str, alignment: int, chunk_size: int) -> Index:
    """Write ``out_dir/sllm.part0`` and ``out_dir/sllm.index``."""
    validate(tensors, alignment, chunk_size)
    os.makedirs(out_dir, exist_ok=True)
    index = make_index(tensors, alignment, chunk_size)
    with open(os.path.join(out_dir, DATA_NAME), "wb") as f:
        f.write(partition_bytes(tensors, alignment))
    with open(os.path.join(out_dir, INDEX_NAME), "wb") as f:
        f.write(encode_index(index))
    return index


# --------------------------------------------------------------------------
# loading (Sec. 4.2): fixed-size chunks into one buffer
# --------------------------------------------------------------------------

def chunks(total: int, chunk_size: int) -> List[Tuple[int, int, int]]:
    """Chunk k covers ``[kC, min(kC + C, T))``: (k, start, end) for every chunk."""
    if chunk_size < 1:
        raise OracleError("chunk size must be >= 1")
    out = []
    k = 0
    while k * chunk_size < total:
        out.append((k, k * chunk_size, min((k + 1) * chunk_size, total)))
        k += 1
    return out


def read_index(ckpt_dir: str) -> Index:
    with open(os.path.join(ckpt_dir, INDEX_NAME), "rb") as f:
        return decode_index(f.read())


def read(ckpt_dir: str, chunk_size: int = 0, max_chunks: int = -1) -> Tuple[Index, bytearray]:
    """Reference reader: copy the partition into one buffer ``H`` chunk by chunk.

    ``H[0:T)`` equals the partition's first T bytes.  ``max_chunks >= 0`` stops
    after that many chunks (a bounded sample for timing); bytes past them stay 0.
    """
    index = read_index(ckpt_dir)
    C = chunk_size or index.chunk_size
    H = bytearray(index.total_bytes)
    view = memoryview(H)
    with open(os.path.join(ckpt_dir, DATA_NAME), "rb", buffering=0) as f:
        for k, start, end in chunks(index.total_bytes, C):
            if 0 <= max_chunks <= k:
                break
            f.seek(start)
            got = f.readinto(view[start:end])
            if got != end - start:
                raise OracleError(f"short read in chunk {k}")
    return index, H


def tensor_bytes(H, entry: Entry) -> bytes:
    """A tensor's view at base + offset (Sec. 4.1, direct tensor addressing)."""
    return bytes(H[entry.offset:entry.offset + entry.nbytes])


# --------------------------------------------------------------------------
# device layout with its own alignment A2 (reading 10)
# --------------------------------------------------------------------------

def device_layout(index: Index, dev_alignment: int) -> Tuple[List[int], int]:
    return plan_layout([e.nbytes for e in index.entries], dev_alignment)


def repack(H, index: Index, dev_alignment: int) -> bytearray:
    """Move every tensor from its file offset to its offset in the A2 layout."""
    d, total2 = device_layout(index, dev_alignment)
    D2 = bytearray(total2)
    for e, di in zip(index.entries, d):
        D2[di:di + e.nbytes] = H[e.offset:e.offset + e.nbytes]
    return D2


# --------------------------------------------------------------------------
# the invariants the format fixes
# --------------------------------------------------------------------------

def check_invariants(index: Index, P) -> None:
    """Raise if the partition/index pair breaks a property the format fixes."""
    A, T, F = index.alignment, index.total_bytes, index.file_bytes
    if not is_pow2(A):
        raise OracleError("alignment is not a power of two")
    if F % FILE_BLOCK or not 0 <= F - T < FILE_BLOCK or len(P) != F:
        raise OracleError("file length is not T rounded up to 4 KiB")
    padded = 0
    prev_end = 0
    gaps = []  # byte ranges that hold no tensor data
    for e in index.entries:
        if e.offset % A:
            raise OracleError(f"{e.name}: offset {e.offset} not aligned to {A}")
        if e.offset < prev_end:
            raise OracleError(f"{e.name}: overlaps the previous tensor or is out of order")
        if e.nbytes != _numel(e.shape) * ITEMSIZE[e.dtype]:
            raise OracleError(f"{e.name}: size does not match shape and dtype")
        gaps.append((prev_end, e.offset))
        prev_end = e.offset + e.nbytes
        padded += align_up(e.nbytes, A)
    if padded != T:
        raise OracleError("total is not the padded sum")
    if prev_end > T:
        raise OracleError("a tensor runs past T")
    gaps.append((prev_end, F))
    for a, b in gaps:
        if any(P[a:b]):
            raise OracleError(f"padding in [{a}, {b}) is not all zero")
