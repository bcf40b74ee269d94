"""Host-side checks of the native library that need no GPU: the exported
symbols, the binding's struct layouts, the C++ converter against the oracle
(byte for byte) and the validation sllm_open performs before any HIP call."""

import ctypes as C
import os
import re
import shutil
import struct
import subprocess
import zlib

import numpy as np
import pytest

import oracle
from paper_2401_14351_amd import binding, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sllm.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("libsllm.so not built")
    return binding.lib()


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sllm_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(L):
    declared = header_functions()
    assert len(declared) >= 20
    assert sorted(binding.SIGNATURES) == declared
    out = subprocess.run(["nm", "-D", "--defined-only", binding.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (sllm_\w+)", out))
    assert set(declared) <= exported
    for name in declared:
        getattr(L, name)


def test_struct_layouts_match_header(tmp_path):
    probe = tmp_path / "probe.c"
    structs = {"sllm_src_tensor": binding.SrcTensor, "sllm_convert_opts": binding.ConvertOpts,
               "sllm_pool_info": binding.PoolInfo, "sllm_open_opts": binding.OpenOpts,
               "sllm_tensor_info": binding.TensorInfo, "sllm_stats": binding.Stats,
               "sllm_ipc_desc": binding.IpcDesc}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "sllm.h"', "int main(void) {"]
    for cname, py in structs.items():
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in py._fields_:
            lines.append(f'printf("{cname}.{f} %zu\\n", offsetof({cname}, {f}));')
    lines.append("return 0; }")
    probe.write_text("\n".join(lines))
    exe = tmp_path / "probe"
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", f"-I{ROOT}/include", str(probe), "-o", str(exe)], check=True)
    got = dict(l.rsplit(" ", 1) for l in subprocess.run([str(exe)], capture_output=True, text=True).stdout.splitlines())
    for cname, py in structs.items():
        assert int(got[f"{cname} size"]) == C.sizeof(py), cname
        for f, _ in py._fields_:
            assert int(got[f"{cname}.{f}"]) == getattr(py, f).offset, f"{cname}.{f}"


def test_strerror(L):
    assert L.sllm_strerror(0) == b"SLLM_OK"
    for code, name in binding.ERRORS.items():
        assert L.sllm_strerror(code).decode() == name


# ---------------------------------------------------------------------------
# converter parity with the oracle
# ---------------------------------------------------------------------------

def _tensors(spec):
    return [(t.name, t.dtype, t.shape, d) for t, d in zip(spec.tensors, synth.materialize(spec, threads=2))]


def _files(d):
    return (open(os.path.join(d, "sllm.part0"), "rb").read(), open(os.path.join(d, "sllm.index"), "rb").read())


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("A", [1, 2, 16, 256, 4096])
def test_convert_matches_oracle_tiny(L, tmp_path, seed, A):
    spec = synth.tiny(seed, alignment=A, chunk_size=64 + seed)
    tensors = _tensors(spec)
    oracle.convert(tensors, str(tmp_path / "o"), A, spec.chunk_size)
    binding.convert_array(tensors, str(tmp_path / "b"), A, spec.chunk_size)
    binding.convert(iter(tensors), str(tmp_path / "s"), A, spec.chunk_size)
    want = _files(tmp_path / "o")
    assert _files(tmp_path / "b") == want
    assert _files(tmp_path / "s") == want


def test_convert_matches_oracle_opt125m(L, tmp_path):
    spec = synth.opt_125m()
    tensors = _tensors(spec)
    oracle.convert(tensors, str(tmp_path / "o"), spec.alignment, spec.chunk_size)
    binding.convert(iter(tensors), str(tmp_path / "b"), spec.alignment, spec.chunk_size)
    assert _files(tmp_path / "b") == _files(tmp_path / "o")


def test_convert_stress_prefix(L, tmp_path):
    spec = synth.stress(n=300, max_bytes=1 << 16)
    tensors = _tensors(spec)
    oracle.convert(tensors, str(tmp_path / "o"), spec.alignment, spec.chunk_size)
    binding.convert(iter(tensors), str(tmp_path / "b"), spec.alignment, spec.chunk_size)
    assert _files(tmp_path / "b") == _files(tmp_path / "o")


def test_convert_empty_checkpoint(L, tmp_path):
    oracle.convert([], str(tmp_path / "o"), 256, 4096)
    binding.convert_array([], str(tmp_path / "b"), 256, 4096)
    assert _files(tmp_path / "b") == _files(tmp_path / "o")
    assert os.path.getsize(tmp_path / "b" / "sllm.part0") == 0


@pytest.mark.parametrize("bad", [
    [("a", "f32", (2,), b"\0" * 8), ("a", "f32", (2,), b"\0" * 8)],   # duplicate name
    [("", "f32", (2,), b"\0" * 8)],                                  # empty name
    [("a", "f32", (3,), b"\0" * 8)],                                 # nbytes != numel * itemsize
    [("a", "i8", (1,) * 9, b"\0")],                                  # ndim > 8
    [("a", "i8", (-1,), b"")],                                       # negative dim
])
def test_convert_rejects_and_cleans_up(L, tmp_path, bad):
    with pytest.raises(binding.SllmError) as ei:
        binding.convert_array(bad, str(tmp_path), 16, 64)
    assert ei.value.code == -1
    assert not os.path.exists(tmp_path / "sllm.part0")
    assert not os.path.exists(tmp_path / "sllm.index")


def test_convert_rejects_bad_alignment(L, tmp_path):
    with pytest.raises(binding.SllmError) as ei:
        binding.convert_array([("a", "i8", (1,), b"\1")], str(tmp_path), 3, 64)
    assert ei.value.code == -1


def test_writer_abort_removes_files(L, tmp_path):
    w = C.c_void_p()
    binding.check(L.sllm_writer_open(str(tmp_path).encode(), None, C.byref(w)))
    st, keep = binding._src_tensor("x", "i8", (3,), bytearray(b"abc"))
    binding.check(L.sllm_writer_add(w, C.byref(st)))
    L.sllm_writer_abort(w)
    assert os.listdir(tmp_path) == []


# ---------------------------------------------------------------------------
# sllm_open validation (every case fails before the first HIP call)
# ---------------------------------------------------------------------------

@pytest.fixture()
def ckpt(L, tmp_path):
    spec = synth.tiny(3, alignment=16)
    d = tmp_path / "ck"
    oracle.convert(_tensors(spec), str(d), 16, 64)
    return d


def _open_code(L, d):
    h = C.c_void_p()
    rc = L.sllm_open(str(d).encode(), None, C.byref(h))
    if rc == 0:
        L.sllm_close(h)
    return rc, L.sllm_last_error().decode()


def _rewrite_index(d, mutate):
    blob = bytearray(open(d / "sllm.index", "rb").read())
    mutate(blob)
    body = bytes(blob[:-4])
    blob[-4:] = struct.pack("<I", zlib.crc32(body))
    open(d / "sllm.index", "wb").write(bytes(blob))


def test_open_rejects_crc_damage(L, ckpt):
    blob = bytearray(open(ckpt / "sllm.index", "rb").read())
    blob[70] ^= 1
    open(ckpt / "sllm.index", "wb").write(bytes(blob))
    rc, msg = _open_code(L, ckpt)
    assert rc == -3 and "CRC" in msg


def test_open_rejects_bad_magic(L, ckpt):
    _rewrite_index(ckpt, lambda b: b.__setitem__(0, ord("X")))
    assert _open_code(L, ckpt)[0] == -3


def test_open_rejects_bad_version(L, ckpt):
    _rewrite_index(ckpt, lambda b: b.__setitem__(slice(8, 12), struct.pack("<I", 2)))
    assert _open_code(L, ckpt)[0] == -3


def test_open_rejects_wrong_total(L, ckpt):
    def m(b):
        T = struct.unpack_from("<Q", b, 32)[0]
        b[32:40] = struct.pack("<Q", T + 16)
    _rewrite_index(ckpt, m)
    rc, msg = _open_code(L, ckpt)
    assert rc == -3 and "padded sum" in msg


def test_open_rejects_moved_offset(L, ckpt):
    # shift the second tensor's offset by the alignment
    idx = oracle.read_index(str(ckpt))
    e = idx.entries[1]
    ents = list(idx.entries)
    import dataclasses
    ents[1] = dataclasses.replace(e, offset=e.offset + 16)
    blob = oracle.encode_index(dataclasses.replace(idx, entries=tuple(ents)))
    open(ckpt / "sllm.index", "wb").write(blob)
    rc, msg = _open_code(L, ckpt)
    assert rc == -3 and "offset" in msg


def test_open_rejects_duplicate_name(L, ckpt):
    import dataclasses
    idx = oracle.read_index(str(ckpt))
    ents = list(idx.entries)
    ents[1] = dataclasses.replace(ents[1], name=ents[0].name)
    open(ckpt / "sllm.index", "wb").write(oracle.encode_index(dataclasses.replace(idx, entries=tuple(ents))))
    rc, msg = _open_code(L, ckpt)
    assert rc == -3 and "duplicate" in msg


def test_open_rejects_size_shape_mismatch(L, ckpt):
    import dataclasses
    idx = oracle.read_index(str(ckpt))
    ents = list(idx.entries)
    i = next(k for k, e in enumerate(ents) if e.nbytes > 4)
    ents[i] = dataclasses.replace(ents[i], nbytes=ents[i].nbytes - 1)
    open(ckpt / "sllm.index", "wb").write(oracle.encode_index(dataclasses.replace(idx, entries=tuple(ents))))
    assert _open_code(L, ckpt)[0] == -3


def test_open_rejects_truncated_data(L, ckpt):
    p = ckpt / "sllm.part0"
    data = open(p, "rb").read()
    open(p, "wb").write(data[:-1])
    rc, msg = _open_code(L, ckpt)
    assert rc == -3 and "bytes" in msg


def test_open_rejects_truncated_index(L, ckpt):
    p = ckpt / "sllm.index"
    data = open(p, "rb").read()
    open(p, "wb").write(data[:40])
    assert _open_code(L, ckpt)[0] == -3


def test_close_is_safe_to_repeat(L, ckpt):
    """Closing nothing is a no-op for every handle type, and the binding's
    close() may run twice (the second call does nothing)."""
    assert L.sllm_close(None) == 0
    assert L.sllm_pool_destroy(None) == 0
    L.sllm_estimator_destroy(None)  # returns nothing; must not crash
    ck = binding.Checkpoint(str(ckpt), index_only=True)
    assert ck.total_bytes > 0
    ck.close()
    ck.close()
    with binding.Checkpoint(str(ckpt), index_only=True) as ck2:
        ck2.close()  # closed inside the block; leaving it closes nothing more


def test_open_missing_dir(L, tmp_path):
    assert _open_code(L, tmp_path / "nope")[0] == -2


def test_open_rejects_bad_options(L, ckpt):
    h = C.c_void_p()
    for kw in ({"engine": 7}, {"dev_alignment": 8}, {"dev_alignment": 48}, {"flags": 64}):
        o = binding.OpenOpts()
        for k, v in kw.items():
            setattr(o, k, v)
        assert L.sllm_open(str(ckpt).encode(), C.byref(o), C.byref(h)) == -1, kw


@pytest.mark.parametrize("A,A2", [(1, 0), (16, 0), (4096, 0), (1, 16), (16, 256), (4096, 256), (256, 4096)])
def test_index_only_open_matches_oracle_layout(L, tmp_path, A, A2):
    """An index-only handle needs no GPU; its offsets are the oracle's (file
    layout, or the A2 device layout planned on the host)."""
    spec = synth.tiny(9, alignment=A)
    tensors = _tensors(spec)
    oracle.convert(tensors, str(tmp_path), A, 64)
    index = oracle.read_index(str(tmp_path))
    want, total = (oracle.device_layout(index, A2) if A2 else
                   ([e.offset for e in index.entries], index.total_bytes))
    with binding.Checkpoint(str(tmp_path), index_only=True, dev_alignment=A2) as ck:
        got = ck.tensors()
        assert [t.offset for t in got] == want and ck.total_bytes == total
        assert [(t.name, t.dtype, t.shape, t.nbytes) for t in got] == \
            [(e.name, e.dtype, e.shape, e.nbytes) for e in index.entries]
        assert ck.find(index.entries[-1].name).offset == want[-1]
        with pytest.raises(binding.SllmError) as ei:
            ck.load(0, 1 << 30)
        assert ei.value.code == -1


@pytest.mark.skipif(not os.path.exists("/dev/full"), reason="no /dev/full")
def test_convert_reports_a_full_disk(L, tmp_path):
    """A write error (ENOSPC) ends the conversion with SLLM_E_IO and no files."""
    os.symlink("/dev/full", tmp_path / "sllm.part0")
    big = np.zeros(16 << 20, dtype=np.uint8)  # larger than the writer's staging buffer
    with pytest.raises(binding.SllmError) as ei:
        binding.convert([("w", "i8", (big.size,), big)], str(tmp_path), 256, 1 << 20)
    assert ei.value.code == -2 and "write" in ei.value.message
    assert not os.path.exists(tmp_path / "sllm.index")


def test_repack_noalloc_host_checks(L, tmp_path):
    """sllm_repack_noalloc refuses bad arguments before any HIP call (the
    device pointers below are never dereferenced)."""
    spec = synth.tiny(5, n=10, alignment=16)
    tensors = [(t.name, t.dtype, t.shape, d) for t, d in zip(spec.tensors, synth.materialize(spec))]
    d = str(tmp_path / "c")
    binding.convert(iter(tensors), d, 16, 64)
    index = oracle.make_index(tensors, 16, 64)
    T = index.total_bytes
    T2 = oracle.device_layout(index, 256)[1]
    src, dst = 1 << 40, 1 << 41  # 16-byte aligned, far apart
    with binding.Checkpoint(d, index_only=True) as ck:
        h = ck._h
        f = L.sllm_repack_noalloc
        assert f(None, 256, src, T, dst, T2, None) == -1
        assert f(h, 0, src, T, dst, T2, None) == -1           # no alignment given, none on the handle
        assert f(h, 8, src, T, dst, T2, None) == -1           # below 16
        assert f(h, 48, src, T, dst, T2, None) == -1          # not a power of two
        assert f(h, 256, src, T - 1, dst, T2, None) == -6     # source too small
        assert f(h, 256, src, T, dst, T2 - 1, None) == -6     # destination too small
        assert f(h, 256, src + 8, T, dst, T2, None) == -1     # misaligned
        assert f(h, 256, src, T, src + 16, T2, None) == -1    # overlap
        assert b"overlap" in L.sllm_last_error()
    empty = str(tmp_path / "e")
    binding.convert(iter([]), empty, 16, 64)
    with binding.Checkpoint(empty, index_only=True) as ck:
        assert L.sllm_repack_noalloc(ck._h, 256, src, 0, dst, 0, None) == 0  # nothing to move
    many = str(tmp_path / "m")
    binding.convert(iter((f"z{i}", "i8", (0,), np.zeros(0, np.uint8)) for i in range(65537)), many, 16, 64)
    with binding.Checkpoint(many, index_only=True) as ck:
        assert L.sllm_repack_noalloc(ck._h, 256, src, 64, dst, 64, None) == -6
        assert b"65536" in L.sllm_last_error()
