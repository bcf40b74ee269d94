"""The safetensors converter front-end (host-only): its output equals the
oracle's conversion of the same tensors in shard and file order, and it
rejects malformed or unsupported shards."""

import json
import os
import struct

import numpy as np
import pytest

import oracle
from paper_2401_14351_amd import binding, synth

torch = pytest.importorskip("torch")
st = pytest.importorskip("safetensors.torch")

TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16, "i8": torch.int8}


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("libsllm.so not built")
    return binding.lib()


def to_torch(t, data):
    if data.size == 0:
        return torch.empty(t.shape, dtype=TORCH_DT[t.dtype])
    return torch.from_numpy(data.copy()).view(TORCH_DT[t.dtype]).reshape(t.shape)


def file_order(path):
    """(name, dtype, shape, bytes) in data-offset order, read without the library."""
    raw = open(path, "rb").read()
    (n,) = struct.unpack_from("<Q", raw, 0)
    header = json.loads(raw[8:8 + n])
    header.pop("__metadata__", None)
    code = {"F32": "f32", "F16": "f16", "BF16": "bf16", "I8": "i8"}
    items = sorted(header.items(), key=lambda kv: kv[1]["data_offsets"][0])  # stable: JSON order breaks ties
    out = []
    for name, v in items:
        b, e = v["data_offsets"]
        out.append((name, code[v["dtype"]], tuple(v["shape"]), raw[8 + n + b:8 + n + e]))
    return out


def files(d):
    return open(os.path.join(d, "sllm.part0"), "rb").read(), open(os.path.join(d, "sllm.index"), "rb").read()


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("A", [1, 16, 256])
def test_matches_oracle(L, tmp_path, seed, A):
    spec = synth.tiny(seed, n=14, alignment=A)
    data = synth.materialize(spec, threads=1)
    path = str(tmp_path / "m.safetensors")
    st.save_file({t.name: to_torch(t, d) for t, d in zip(spec.tensors, data)}, path, metadata={"format": "pt"})
    binding.convert_safetensors([path], str(tmp_path / "b"), A, 64)
    oracle.convert(file_order(path), str(tmp_path / "o"), A, 64)
    assert files(tmp_path / "b") == files(tmp_path / "o")


def test_shards_and_lora_shapes(L, tmp_path):
    spec = synth.lora("7b", rank=4)
    data = synth.materialize(spec)
    half = len(spec.tensors) // 2
    paths = []
    for k, (lo, hi) in enumerate(((0, half), (half, len(spec.tensors)))):
        p = str(tmp_path / f"adapter-{k}.safetensors")
        st.save_file({t.name: to_torch(t, d) for t, d in zip(spec.tensors[lo:hi], data[lo:hi])}, p)
        paths.append(p)
    binding.convert_safetensors(paths, str(tmp_path / "b"), 256, 1 << 20)
    oracle.convert(file_order(paths[0]) + file_order(paths[1]), str(tmp_path / "o"), 256, 1 << 20)
    assert files(tmp_path / "b") == files(tmp_path / "o")


def _write_raw(path, header, payload=b""):
    h = json.dumps(header).encode()
    open(path, "wb").write(struct.pack("<Q", len(h)) + h + payload)


@pytest.mark.parametrize("header,payload,code", [
    ({"a": {"dtype": "F64", "shape": [1], "data_offsets": [0, 8]}}, b"\0" * 8, -1),      # unsupported dtype
    ({"a": {"dtype": "F32", "shape": [3], "data_offsets": [0, 8]}}, b"\0" * 8, -3),      # size != numel * 4
    ({"a": {"dtype": "F32", "shape": [2], "data_offsets": [0, 8]}}, b"\0" * 4, -3),      # data past the end
    ({"a": {"dtype": "I8", "shape": [4], "data_offsets": [0, 4]},
      "b": {"dtype": "I8", "shape": [4], "data_offsets": [2, 6]}}, b"\0" * 6, -3),       # overlap
    ({"a": {"dtype": "I8", "shape": [-1], "data_offsets": [0, 0]}}, b"", -3),            # negative dim
    ({"a": {"dtype": "I8", "shape": [1]}}, b"\0", -3),                                    # no offsets
    ({"a": {"dtype": "I8", "shape": [1, 1, 1, 1, 1, 1, 1, 1, 1], "data_offsets": [0, 1]}}, b"\0", -1),
])
def test_rejects(L, tmp_path, header, payload, code):
    p = str(tmp_path / "bad.safetensors")
    _write_raw(p, header, payload)
    with pytest.raises(binding.SllmError) as ei:
        binding.convert_safetensors([p], str(tmp_path / "o"), 256, 64)
    assert ei.value.code == code
    assert not os.path.exists(tmp_path / "o" / "sllm.part0")


def test_rejects_garbage_and_duplicates(L, tmp_path):
    p = str(tmp_path / "g.safetensors")
    open(p, "wb").write(struct.pack("<Q", 5) + b"{\"a\":")
    with pytest.raises(binding.SllmError) as ei:
        binding.convert_safetensors([p], str(tmp_path / "o"), 256, 64)
    assert ei.value.code == -3
    a = str(tmp_path / "a.safetensors")
    st.save_file({"x": torch.zeros(2)}, a)
    with pytest.raises(binding.SllmError) as ei:
        binding.convert_safetensors([a, a], str(tmp_path / "o"), 256, 64)
    assert ei.value.code == -1
    with pytest.raises(binding.SllmError) as ei:
        binding.convert_safetensors([str(tmp_path / "missing")], str(tmp_path / "o"), 256, 64)
    assert ei.value.code == -2
