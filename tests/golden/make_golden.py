"""Write the index-encoding regression fixture ``tiny_index.hex``.

The paper prints no worked example, byte layout or checksum of its converted
checkpoints (Sec. 4.1 describes the index only as name -> GPU id, offset,
size), so no stored value here comes from the paper.  This fixture only
freezes the oracle's encoding of a small fixed checkpoint so that an
accidental change to the format shows up; it calls nothing but the oracle.

Run from the repository root:  python -m tests.golden.make_golden
"""

import os

GOLDEN_A = 256
GOLDEN_C = 4096


def golden_tensors():
    # (name, dtype, shape, bytes): a 0-d f32, a zero-size bf16, a 3x5 f16, an i8 vector
    return [
        ("scalar", "f32", (), bytes([0, 0, 128, 63])),
        ("empty.bf16", "bf16", (0, 4), b""),
        ("w.f16", "f16", (3, 5), bytes(range(30))),
        ("layer.0.bias", "i8", (257,), bytes((i * 7) & 0xFF for i in range(257))),
    ]


def main():
    import oracle

    index = oracle.make_index(golden_tensors(), GOLDEN_A, GOLDEN_C)
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_index.hex")
    with open(path, "w") as f:
        f.write(oracle.encode_index(index).hex() + "\n")


if __name__ == "__main__":
    main()
