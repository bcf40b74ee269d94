"""Property tests (hypothesis, CPU): for arbitrary tensor lists (unicode
names, every dtype, 0-d, zero-size and odd shapes), alignments and chunk
sizes, the library's converters write files byte-identical to the oracle's,
and an index-only open reports the oracle's layout at any device alignment."""

import os
import shutil
import tempfile

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from paper_2401_14351_amd import binding

ITEMSIZE = {"f32": 4, "f16": 2, "bf16": 2, "i8": 1}

names = st.text(alphabet=st.characters(blacklist_categories=("Cs",), blacklist_characters="\x00"),
                min_size=1, max_size=24).filter(lambda s: 0 < len(s.encode()) <= 65535)
specs = st.lists(st.tuples(names, st.sampled_from(sorted(ITEMSIZE)),
                           st.lists(st.integers(0, 9), min_size=0, max_size=4).map(tuple)),
                 min_size=0, max_size=24, unique_by=lambda t: t[0])
alignments = st.sampled_from([1, 2, 4, 8, 16, 64, 256, 4096])


def materialize(spec, seed):
    rng = np.random.default_rng(seed)
    out = []
    for name, dt, shape in spec:
        n = int(np.prod(shape)) if shape else 1
        out.append((name, dt, shape, rng.integers(0, 256, n * ITEMSIZE[dt], dtype=np.uint8).tobytes()))
    return out


def files(d):
    return tuple(open(os.path.join(d, f), "rb").read() for f in ("sllm.part0", "sllm.index"))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("libsllm.so not built")
    return binding.lib()


@settings(max_examples=120, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(spec=specs, A=alignments, C=st.integers(1, 1 << 16), seed=st.integers(0, 2**32 - 1))
def test_converters_match_oracle(L, spec, A, C, seed):
    tensors = materialize(spec, seed)
    root = tempfile.mkdtemp()
    try:
        oracle.convert(tensors, os.path.join(root, "o"), A, C)
        binding.convert_array(tensors, os.path.join(root, "b"), A, C)
        binding.convert(iter(tensors), os.path.join(root, "s"), A, C)
        want = files(os.path.join(root, "o"))
        assert files(os.path.join(root, "b")) == want
        assert files(os.path.join(root, "s")) == want
    finally:
        shutil.rmtree(root, ignore_errors=True)


@settings(max_examples=120, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(spec=specs, A=alignments, A2=st.sampled_from([0, 16, 32, 256, 4096]), seed=st.integers(0, 2**32 - 1))
def test_index_only_open_matches_oracle_layout(L, spec, A, A2, seed):
    tensors = materialize(spec, seed)
    root = tempfile.mkdtemp()
    try:
        binding.convert(iter(tensors), root, A, 4096)
        index = oracle.make_index(tensors, A, 4096)
        offsets, total = oracle.device_layout(index, A2) if A2 else ([e.offset for e in index.entries],
                                                                    index.total_bytes)
        with binding.Checkpoint(root, index_only=True, dev_alignment=A2) as ck:
            got = ck.tensors()
            assert ck.total_bytes == total
            assert [t.offset for t in got] == offsets
            assert [(t.name, t.dtype, tuple(t.shape), t.nbytes) for t in got] == \
                [(e.name, e.dtype, tuple(e.shape), e.nbytes) for e in index.entries]
            for e in index.entries:
                assert ck.find(e.name).nbytes == e.nbytes
    finally:
        shutil.rmtree(root, ignore_errors=True)
