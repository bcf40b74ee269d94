"""Pins for the CPU oracle: each test checks it against something other than
its own formulas (hand-worked closed forms, brute force, library routines, the
independently computed workload sizes, invariants with planted mistakes)."""

import io
import math
import os
import random
import struct
import zlib

import numpy as np
import pytest

import oracle
from paper_2401_14351_amd import synth


def as_oracle_tensors(spec, data):
    return [(t.name, t.dtype, t.shape, d) for t, d in zip(spec.tensors, data)]


# ---------------------------------------------------------------------------
# layout: hand-worked cases of the aligned packing of Sec. 4.1
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("sizes,A,offsets,T", [
    # 5 bytes take an 8-byte slot at A=4; the empty tensor takes none; the last starts at 8
    ([5, 0, 3], 4, [0, 8, 8], 12),
    # dense packing at A=1
    ([5, 0, 3], 1, [0, 5, 5], 8),
    # one byte still takes a whole 4096-byte slot
    ([4096, 1, 4096], 4096, [0, 4096, 8192], 12288),
    # sizes that are already multiples of A need no padding
    ([256, 512, 768], 256, [0, 256, 768], 1536),
    # 255 and 257 bytes at A=256
    ([255, 257, 1], 256, [0, 256, 768], 1024),
    ([], 16, [], 0),
])
def test_layout_hand_worked(sizes, A, offsets, T):
    o, t = oracle.plan_layout(sizes, A)
    assert o == offsets and t == T
    assert oracle.file_length(t) == (0 if T == 0 else 4096 * ((T + 4095) // 4096))


def _brute_offsets(sizes, A):
    """Place each tensor at the first position after the previous one that is a
    multiple of A, found by stepping one byte at a time."""
    out, end = [], 0
    for s in sizes:
        x = end
        while x % A:
            x += 1
        out.append(x)
        end = x + s
    total = end
    while total % A:
        total += 1
    return out, total


@pytest.mark.parametrize("A", [1, 2, 16, 256, 4096])
def test_layout_matches_brute_force(A):
    rng = random.Random(A)
    for _ in range(200):
        sizes = [rng.choice([0, 1, A - 1 if A > 1 else 0, A, A + 1, rng.randrange(0, 3 * A + 5)])
                 for _ in range(rng.randrange(0, 9))]
        assert oracle.plan_layout(sizes, A) == _brute_offsets(sizes, A)


def test_layout_rejects_bad_alignment():
    for bad in (0, 3, 12, -4):
        with pytest.raises(oracle.OracleError):
            oracle.plan_layout([1], bad)


# ---------------------------------------------------------------------------
# workload sizes: totals computed independently from the model shapes
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("spec,n,T,F,max_bytes,min_bytes", [
    (synth.opt_125m(), 196, 250_478_592, 250_478_592, 77_217_792, 1_536),
    (synth.llama2("7b"), 291, 13_476_831_232, 13_476_831_232, 262_144_000, 8_192),
    (synth.llama2("13b"), 363, 26_031_728_640, 26_031_730_688, 327_680_000, 10_240),
    (synth.llama2("70b"), 723, 137_953_296_384, 137_953_296_384, 524_288_000, 16_384),
])
def test_workload_totals(spec, n, T, F, max_bytes, min_bytes):
    sizes = [t.nbytes for t in spec.tensors]
    assert len(sizes) == n and max(sizes) == max_bytes and min(sizes) == min_bytes
    _, total = oracle.plan_layout(sizes, spec.alignment)
    assert total == T
    assert oracle.file_length(total) == F
    assert total == sum(sizes)  # these model layouts need no padding at A = 256


@pytest.mark.parametrize("spec,C,count,last", [
    (synth.opt_125m(), 16 << 20, 15, None),
    (synth.llama2("7b"), 16 << 20, 804, 4_726_784),
    (synth.llama2("13b"), 4 << 20, 6207, None),
    (synth.llama2("13b"), 16 << 20, 1552, None),
    (synth.llama2("13b"), 64 << 20, 388, None),
    (synth.llama2("70b"), 64 << 20, 2056, None),
])
def test_workload_chunk_counts(spec, C, count, last):
    _, total = oracle.plan_layout([t.nbytes for t in spec.tensors], spec.alignment)
    ch = oracle.chunks(total, C)
    assert len(ch) == count
    if last is not None:
        assert ch[-1][2] - ch[-1][1] == last


# ---------------------------------------------------------------------------
# conversion: byte round trip and the format's invariants
# ---------------------------------------------------------------------------

def _independent_check(index, P, tensors):
    """The format's invariants, checked without the oracle's own checker."""
    A = index.alignment
    assert len(P) == index.file_bytes and index.file_bytes % 4096 == 0
    assert 0 <= index.file_bytes - index.total_bytes < 4096
    covered = np.zeros(len(P), dtype=np.int32)
    padded = 0
    for e, (name, dtype, shape, data) in zip(index.entries, tensors):
        assert e.name == name and e.dtype == dtype and e.shape == tuple(shape)
        assert e.offset % A == 0
        assert bytes(P[e.offset:e.offset + e.nbytes]) == bytes(memoryview(data).cast("B"))
        covered[e.offset:e.offset + e.nbytes] += 1
        padded += -(-e.nbytes // A) * A
    assert covered.max(initial=0) <= 1, "two tensors share a byte"
    starts = [e.offset for e in index.entries]
    assert starts == sorted(starts)
    assert padded == index.total_bytes
    arr = np.frombuffer(bytes(P), dtype=np.uint8)
    assert not arr[covered == 0].any(), "a padding byte is not zero"


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("A", [1, 2, 16, 256, 4096])
def test_convert_round_trip_tiny(tmp_path, seed, A):
    spec = synth.tiny(seed, alignment=A)
    tensors = as_oracle_tensors(spec, synth.materialize(spec, threads=1))
    d = tmp_path / "ck"
    index = oracle.convert(tensors, str(d), A, spec.chunk_size)
    P = (d / "sllm.part0").read_bytes()
    _independent_check(index, P, tensors)
    oracle.check_invariants(index, P)
    assert oracle.read_index(str(d)) == index


def test_convert_round_trip_opt125m(tmp_path):
    spec = synth.opt_125m()
    data = synth.materialize(spec)
    tensors = as_oracle_tensors(spec, data)
    index = oracle.convert(tensors, str(tmp_path), spec.alignment, spec.chunk_size)
    P = (tmp_path / "sllm.part0").read_bytes()
    _independent_check(index, P, tensors)
    oracle.check_invariants(index, P)
    idx, H = oracle.read(str(tmp_path))
    assert bytes(H) == P[:index.total_bytes]
    for e, dd in zip(idx.entries, data):
        assert oracle.tensor_bytes(H, e) == dd.tobytes()


# ---------------------------------------------------------------------------
# the oracle's checker catches planted mistakes
# ---------------------------------------------------------------------------

def _tiny_converted(A=16, seed=3):
    spec = synth.tiny(seed, alignment=A)
    tensors = as_oracle_tensors(spec, synth.materialize(spec, threads=1))
    index = oracle.make_index(tensors, A, spec.chunk_size)
    return index, oracle.partition_bytes(tensors, A)


def test_checker_accepts_good():
    index, P = _tiny_converted()
    oracle.check_invariants(index, P)


def test_checker_flags_dirty_padding():
    index, P = _tiny_converted()
    # first byte after the first non-aligned tensor's data
    e = next(e for e in index.entries if e.nbytes % index.alignment)
    P = bytearray(P)
    P[e.offset + e.nbytes] = 7
    with pytest.raises(oracle.OracleError):
        oracle.check_invariants(index, P)


def test_checker_flags_dirty_tail():
    index, P = _tiny_converted()
    P = bytearray(P)
    P[-1] = 1
    if index.total_bytes < len(P):
        with pytest.raises(oracle.OracleError):
            oracle.check_invariants(index, P)


def test_checker_flags_misaligned_and_overlap_and_total():
    import dataclasses
    index, P = _tiny_converted()
    ents = list(index.entries)
    i = next(k for k in range(1, len(ents)) if ents[k].nbytes)
    bad = dataclasses.replace(ents[i], offset=ents[i].offset + 1)
    with pytest.raises(oracle.OracleError):
        oracle.check_invariants(dataclasses.replace(index, entries=tuple(ents[:i] + [bad] + ents[i + 1:])), P)
    j = next(k for k in range(1, len(ents)) if ents[k - 1].nbytes > index.alignment)
    over = dataclasses.replace(ents[j], offset=ents[j - 1].offset)
    with pytest.raises(oracle.OracleError):
        oracle.check_invariants(dataclasses.replace(index, entries=tuple(ents[:j] + [over] + ents[j + 1:])), P)
    with pytest.raises(oracle.OracleError):
        oracle.check_invariants(dataclasses.replace(index, total_bytes=index.total_bytes + index.alignment), P)


# ---------------------------------------------------------------------------
# chunking: every chunk size on tiny checkpoints
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed,A", [(0, 1), (1, 16), (2, 256), (5, 4096)])
def test_every_chunk_size(tmp_path, seed, A):
    spec = synth.tiny(seed, alignment=A)
    tensors = as_oracle_tensors(spec, synth.materialize(spec, threads=1))
    index = oracle.convert(tensors, str(tmp_path), A, spec.chunk_size)
    P = (tmp_path / "sllm.part0").read_bytes()
    T, F = index.total_bytes, index.file_bytes
    for C in range(1, F + 2):
        ch = oracle.chunks(T, C)
        count = np.zeros(T, dtype=np.int32)
        for k, (kk, a, b) in enumerate(ch):
            assert kk == k and a == k * C and 0 < b - a <= C
            count[a:b] += 1
        assert (count == 1).all(), f"C={C}: chunks do not cover [0, T) exactly once"
        assert len(ch) * C >= T > (len(ch) - 1) * C or T == 0
        if C in (1, 2, 3, 7, 64, 4096, F, F + 1) or C % 97 == 0:
            _, H = oracle.read(str(tmp_path), C)
            assert bytes(H) == P[:T]


# ---------------------------------------------------------------------------
# index encoding
# ---------------------------------------------------------------------------

def test_index_fields_at_documented_positions():
    index, _ = _tiny_converted(A=256, seed=4)
    blob = oracle.encode_index(index)
    assert blob[:8] == b"SLLMIDX1"
    assert struct.unpack_from("<I", blob, 8)[0] == 1            # version
    assert struct.unpack_from("<I", blob, 12)[0] == 1           # one partition
    assert struct.unpack_from("<Q", blob, 16)[0] == 256         # A
    assert struct.unpack_from("<Q", blob, 24)[0] == index.chunk_size
    assert struct.unpack_from("<Q", blob, 32)[0] == index.total_bytes
    assert struct.unpack_from("<Q", blob, 40)[0] == index.file_bytes
    assert struct.unpack_from("<Q", blob, 48)[0] == len(index.entries)
    # CRC-32 trailer equals zlib's over everything before it
    assert struct.unpack("<I", blob[-4:])[0] == zlib.crc32(blob[:-4])
    # 60 bytes of header + trailer and 24 + 8*ndim + len(name) per tensor
    assert len(blob) == 60 + sum(24 + 8 * len(e.shape) + len(e.name.encode()) for e in index.entries)
    # walk the records by hand
    pos = 56
    for e in index.entries:
        ln = struct.unpack_from("<I", blob, pos)[0]
        assert blob[pos + 4:pos + 4 + ln].decode() == e.name
        pos += 4 + ln
        code, ndim, part = struct.unpack_from("<BBH", blob, pos)
        assert (code, ndim, part) == ({"f32": 0, "f16": 1, "bf16": 2, "i8": 3}[e.dtype], len(e.shape), 0)
        pos += 4 + 8 * ndim
        assert struct.unpack_from("<QQ", blob, pos) == (e.offset, e.nbytes)
        pos += 16
    assert pos == len(blob) - 4


def test_crc_is_the_ieee_polynomial():
    """The index trailer's CRC-32 is the IEEE 802.3 one (reflected 0xEDB88320,
    initial and final 0xFFFFFFFF): its published check value over the ASCII
    digits 1-9 is 0xCBF43926, and a bitwise long division written out here
    agrees with zlib.crc32 on random data."""
    assert zlib.crc32(b"123456789") == 0xCBF43926

    def crc_bitwise(data):
        c = 0xFFFFFFFF
        for byte in data:
            c ^= byte
            for _ in range(8):
                c = (c >> 1) ^ (0xEDB88320 if c & 1 else 0)
        return c ^ 0xFFFFFFFF

    rng = np.random.default_rng(9)
    for n in (0, 1, 7, 64, 1000):
        data = rng.integers(0, 256, n, dtype=np.uint8).tobytes()
        assert crc_bitwise(data) == zlib.crc32(data)


def test_index_round_trip_and_damage():
    index, _ = _tiny_converted(A=16, seed=7)
    blob = oracle.encode_index(index)
    assert oracle.decode_index(blob) == index
    for pos in (0, 9, 20, 60, len(blob) - 5, len(blob) - 1):
        bad = bytearray(blob)
        bad[pos] ^= 0x40
        with pytest.raises(oracle.OracleError):
            oracle.decode_index(bytes(bad))
    with pytest.raises(oracle.OracleError):
        oracle.decode_index(blob[:-1])


def test_golden_index_matches(tmp_path):
    """Regression fixture for the index encoding (written by the oracle-only
    script next to it)."""
    here = os.path.join(os.path.dirname(__file__), "golden")
    want = bytes.fromhex(open(os.path.join(here, "tiny_index.hex")).read().strip())
    from tests.golden.make_golden import golden_tensors, GOLDEN_A, GOLDEN_C
    index = oracle.make_index(golden_tensors(), GOLDEN_A, GOLDEN_C)
    assert oracle.encode_index(index) == want


# ---------------------------------------------------------------------------
# validation
# ---------------------------------------------------------------------------

def test_validation_rejects():
    ok = ("a", "f32", (2,), b"\0" * 8)
    oracle.validate([ok], 4, 1)
    for bad in (
        [ok, ok],                                   # duplicate name
        [("", "f32", (2,), b"\0" * 8)],            # empty name
        [("b", "f64", (2,), b"\0" * 16)],          # unknown dtype
        [("b", "f32", (3,), b"\0" * 8)],           # size does not match shape
        [("b", "i8", (1,) * 9, b"\0")],            # ndim > 8
        [("b", "i8", (-1,), b"")],                 # negative dim
    ):
        with pytest.raises(oracle.OracleError):
            oracle.validate(bad, 4, 1)
    with pytest.raises(oracle.OracleError):
        oracle.validate([ok], 6, 1)
    with pytest.raises(oracle.OracleError):
        oracle.validate([ok], 4, 0)


# ---------------------------------------------------------------------------
# device layout (A2) repack
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("A,A2", [(1, 16), (16, 256), (256, 16), (4096, 256), (16, 16), (1, 4096)])
def test_repack(A, A2):
    spec = synth.tiny(11, alignment=A)
    tensors = as_oracle_tensors(spec, synth.materialize(spec, threads=1))
    index = oracle.make_index(tensors, A, spec.chunk_size)
    P = oracle.partition_bytes(tensors, A)
    H = P[:index.total_bytes]
    D2 = oracle.repack(H, index, A2)
    if A2 == A:
        assert D2 == H                              # same alignment: nothing moves
    d, T2 = oracle.device_layout(index, A2)
    assert len(D2) == T2 == sum(-(-e.nbytes // A2) * A2 for e in index.entries)
    covered = np.zeros(T2, dtype=np.int32)
    for e, di, (_, _, _, data) in zip(index.entries, d, tensors):
        assert di % A2 == 0
        assert bytes(D2[di:di + e.nbytes]) == bytes(memoryview(data).cast("B"))
        covered[di:di + e.nbytes] += 1
    assert covered.max(initial=0) <= 1
    assert not np.frombuffer(bytes(D2), dtype=np.uint8)[covered == 0].any()


# ---------------------------------------------------------------------------
# the input generator (inputs only, but its rounding and determinism matter)
# ---------------------------------------------------------------------------

def test_bf16_round_to_nearest_even():
    from paper_2401_14351_amd.synth import _bits_of
    f = np.array([0x3F808000, 0x3F818000, 0x3F808001, 0x3F800000, 0xBF80FFFF], dtype=np.uint32).view(np.float32)
    got = _bits_of(f, "bf16").view(np.uint16).tolist()
    # 1+2^-8 is a tie -> even 0x3F80; 1+3*2^-8 is a tie -> even 0x3F82; just above a tie rounds up
    assert got == [0x3F80, 0x3F82, 0x3F81, 0x3F80, 0xBF81]


def test_generator_deterministic_and_thread_independent():
    spec = synth.llama2("7b")
    small = synth.CheckpointSpec("x", spec.seed, 256, 1 << 20,
                                 [synth.TensorSpec("a", "bf16", (3, synth.BLOCK + 5)),
                                  synth.TensorSpec("n", "bf16", (7,), init="ones")])
    a = synth.materialize(small, threads=1)
    b = synth.materialize(small, threads=4)
    assert all((x == y).all() for x, y in zip(a, b))
    assert a[1].view(np.uint16).tolist() == [0x3F80] * 7
    w = a[0].view(np.uint16).astype(np.uint32) << 16
    vals = w.view(np.float32)
    assert abs(float(vals.std()) - 0.02) < 1e-3 and abs(float(vals.mean())) < 1e-3
