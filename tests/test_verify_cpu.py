"""The every-byte image checker on the CPU, against images the oracle built:
it accepts the oracle's image in any window size, and it rejects a planted
mistake anywhere in it (a tensor byte, a padding byte, the tail before the
image's end, a shifted offset)."""

import numpy as np
import pytest
import torch
import xxhash

import oracle
from paper_2401_14351_amd import synth, verify


def multi_block_spec():
    """Tensors spanning several generation blocks (4 Mi elements each), next
    to small ones and a zero-size one, with padding between them."""
    t = [synth.TensorSpec("big.i8", "i8", (synth.BLOCK * 2 + 12345,), init="bytes"),
         synth.TensorSpec("small.f32", "f32", (7,)),
         synth.TensorSpec("empty.f16", "f16", (0, 3)),
         synth.TensorSpec("two.bf16", "bf16", (synth.BLOCK + 3,)),
         synth.TensorSpec("scalar.f16", "f16", ())]
    return synth.CheckpointSpec("multi-block", 77, alignment=4096, chunk_size=1 << 20, tensors=t)


def image_of(spec):
    tensors = [(t.name, t.dtype, t.shape, d) for t, d in zip(spec.tensors, synth.materialize(spec))]
    index = oracle.make_index(tensors, spec.alignment, spec.chunk_size)
    img = oracle.partition_bytes(tensors, spec.alignment)[:index.total_bytes]
    return tensors, index, img


def test_digest_is_the_block_digest_of_the_generator_bytes():
    spec = multi_block_spec()
    by_gen = verify.generated_digests(spec, threads=4)
    by_stream = [dg for _, _, _, dg in verify.generate(spec, threads=3, lookahead=1 << 20)]
    assert by_gen == by_stream
    for i, t in enumerate(spec.tensors):
        data = synth.tensor_bytes(spec, i)
        step = synth.BLOCK * synth.ITEMSIZE[t.dtype]
        blocks = [xxhash.xxh3_128(data[o:o + step].tobytes()).digest() for o in range(0, t.nbytes, step)]
        assert len(blocks) == -(-t.nbytes // step)
        assert by_gen[i] == xxhash.xxh3_128(b"".join(blocks)).digest()
    assert by_gen[2] == xxhash.xxh3_128(b"").digest()  # no bytes, no blocks


@pytest.mark.parametrize("window", [1, 4096, 5 << 20, 1 << 30])
def test_accepts_the_oracle_image(window):
    spec = multi_block_spec()
    _, index, img = image_of(spec)
    digests = verify.generated_digests(spec)
    buf = torch.frombuffer(bytearray(bytes(img) + b"\x5a" * 64), dtype=torch.uint8)
    got = verify.check_image(torch, buf, spec, [e.offset for e in index.entries], index.total_bytes, digests,
                             window=window)
    assert got["bytes"] == index.total_bytes and got["tensors"] == len(spec.tensors)
    assert got["padding_bytes"] == index.total_bytes - sum(t.nbytes for t in spec.tensors)


def test_accepts_repacked_images():
    spec = synth.stress(n=300, max_bytes=1 << 16, seed=9)
    _, index, img = image_of(spec)
    digests = verify.generated_digests(spec)
    for a2 in (16, 256, 8192):
        d2, t2 = oracle.device_layout(index, a2)
        out = oracle.repack(img, index, a2)
        buf = torch.frombuffer(bytearray(bytes(out)), dtype=torch.uint8)
        verify.check_image(torch, buf, spec, d2, t2, digests, window=100_000)


def test_rejects_planted_mistakes():
    spec = multi_block_spec()
    _, index, img = image_of(spec)
    digests = verify.generated_digests(spec)
    offs = [e.offset for e in index.entries]
    T = index.total_bytes

    def check(image, offsets=offs):
        buf = torch.frombuffer(bytearray(bytes(image)), dtype=torch.uint8)
        verify.check_image(torch, buf, spec, offsets, T, digests, window=3 << 20)

    check(img)
    for where, what in [(offs[0] + synth.BLOCK + 7, "big.i8"),        # inside the second block
                        (offs[0] + 2 * synth.BLOCK + 12344, "big.i8"),  # the tensor's last byte
                        (offs[3], "two.bf16"), (offs[4] + 1, "scalar.f16")]:
        bad = bytearray(img)
        bad[where] ^= 0x01
        with pytest.raises(verify.Mismatch, match=what):
            check(bad)
    for where in (offs[1] + 7 * 4, offs[0] + spec.tensors[0].nbytes, T - 1):  # padding and the image's tail
        bad = bytearray(img)
        bad[where] = 0x01
        with pytest.raises(verify.Mismatch, match="padding"):
            check(bad)
    # an offset off by one element: the tensor's bytes are not where the index says
    shifted = list(offs)
    shifted[3] += 2
    with pytest.raises(verify.Mismatch):
        check(img, shifted)
    with pytest.raises(ValueError):  # overlapping slots are refused outright
        check(img, [offs[0], offs[0] + 1] + offs[2:])
