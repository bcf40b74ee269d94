"""ctypes binding of ``libsllm.so`` (the C ABI in ``include/sllm.h``).

The raw entry points keep their C names (``sllm_convert``, ``sllm_open``,
``sllm_load``, ``sllm_tensor_index`` ...) as attributes of :func:`lib`.  The
helpers below only marshal arguments: every byte a load moves is moved by the
library's HIP path.  torch is used for device memory, streams and the views
over the loaded buffer.  If the library has not been built the helpers raise:
there is no fallback.
"""

from __future__ import annotations

import ctypes as C
import functools
import os
import threading
from typing import Callable, Dict, Iterable, List, NamedTuple, Optional, Sequence, Tuple

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsllm.so")

SLLM_OK = 0
ERRORS = {-1: "SLLM_E_INVAL", -2: "SLLM_E_IO", -3: "SLLM_E_FORMAT", -4: "SLLM_E_NOMEM", -5: "SLLM_E_HIP",
          -6: "SLLM_E_RANGE", -7: "SLLM_E_BUSY", -8: "SLLM_E_NOTFOUND"}
DTYPE_CODE = {"f32": 0, "f16": 1, "bf16": 2, "i8": 3}
CODE_DTYPE = {v: k for k, v in DTYPE_CODE.items()}
ITEMSIZE = {0: 4, 1: 2, 2: 2, 3: 1}
ENGINE = {"kernel": 0, "sdma": 1}
OPEN_DIRECT_IO = 1
OPEN_TIMING = 2
OPEN_INDEX_ONLY = 4
OPEN_CACHE = 8
CONVERT_FSYNC = 1
MAX_NDIM = 8


class SrcTensor(C.Structure):
    _fields_ = [("name", C.c_char_p), ("dtype", C.c_uint32), ("ndim", C.c_uint32),
                ("shape", C.POINTER(C.c_int64)), ("data", C.c_void_p), ("nbytes", C.c_uint64)]


class ConvertOpts(C.Structure):
    _fields_ = [("alignment", C.c_uint64), ("chunk_size", C.c_uint64), ("flags", C.c_uint32), ("reserved", C.c_uint32)]


class PoolInfo(C.Structure):
    _fields_ = [("chunk_size", C.c_uint64), ("n_chunks", C.c_uint64), ("free_chunks", C.c_uint64),
                ("cached_checkpoints", C.c_uint64)]


class OpenOpts(C.Structure):
    _fields_ = [("chunk_size", C.c_uint64), ("dev_alignment", C.c_uint64), ("pool", C.c_void_p),
                ("io_threads", C.c_uint32), ("n_streams", C.c_uint32), ("ring_slots", C.c_uint32),
                ("engine", C.c_uint32), ("flags", C.c_uint32), ("device", C.c_int32)]


class TensorInfo(C.Structure):
    _fields_ = [("name", C.c_char_p), ("dtype", C.c_uint32), ("ndim", C.c_uint32),
                ("shape", C.c_int64 * MAX_NDIM), ("offset", C.c_uint64), ("nbytes", C.c_uint64)]


# below this many tensors load_with_views builds the views after the load
# (about 3 us per view on the host; starting a thread costs about 0.1 ms)
_THREADED_VIEWS_MIN = 1024

# the same layout as TensorInfo, for decoding a whole table with numpy
_TENSOR_INFO = np.dtype([("name", "<u8"), ("dtype", "<u4"), ("ndim", "<u4"), ("shape", "<i8", (MAX_NDIM,)),
                         ("offset", "<u8"), ("nbytes", "<u8")], align=True)
assert _TENSOR_INFO.itemsize == C.sizeof(TensorInfo)


class Stats(C.Structure):
    _fields_ = [("bytes_loaded", C.c_uint64), ("bytes_read", C.c_uint64), ("n_chunks", C.c_uint64),
                ("n_launches", C.c_uint64), ("engine", C.c_uint32), ("direct_io", C.c_uint32),
                ("from_cache", C.c_uint32), ("io_threads", C.c_uint32), ("open_s", C.c_double),
                ("load_s", C.c_double), ("read_wait_s", C.c_double), ("device_ms", C.c_double),
                ("bytes_bounced", C.c_uint64), ("reader_busy_s", C.c_double), ("reader_starved_s", C.c_double)]


class IpcDesc(C.Structure):
    _fields_ = [("mem_handle", C.c_uint8 * 64), ("event_handle", C.c_uint8 * 64), ("offset", C.c_uint64),
                ("bytes", C.c_uint64), ("device", C.c_int32), ("flags", C.c_uint32)]


# name -> (restype, argtypes); every symbol the header declares
SIGNATURES = {
    "sllm_convert": (C.c_int32, [C.POINTER(SrcTensor), C.c_uint64, C.c_char_p, C.POINTER(ConvertOpts)]),
    "sllm_writer_open": (C.c_int32, [C.c_char_p, C.POINTER(ConvertOpts), C.POINTER(C.c_void_p)]),
    "sllm_writer_add": (C.c_int32, [C.c_void_p, C.POINTER(SrcTensor)]),
    "sllm_writer_close": (C.c_int32, [C.c_void_p]),
    "sllm_writer_abort": (None, [C.c_void_p]),
    "sllm_convert_safetensors": (C.c_int32, [C.POINTER(C.c_char_p), C.c_uint64, C.c_char_p,
                                             C.POINTER(ConvertOpts)]),
    "sllm_pool_create": (C.c_int32, [C.c_uint64, C.c_uint64, C.c_int32, C.POINTER(C.c_void_p)]),
    "sllm_pool_destroy": (C.c_int32, [C.c_void_p]),
    "sllm_pool_query": (C.c_int32, [C.c_void_p, C.POINTER(PoolInfo)]),
    "sllm_pool_cache": (C.c_int32, [C.c_void_p, C.c_char_p, C.c_uint32, C.c_uint32]),
    "sllm_pool_evict": (C.c_int32, [C.c_void_p, C.c_char_p]),
    "sllm_open": (C.c_int32, [C.c_char_p, C.POINTER(OpenOpts), C.POINTER(C.c_void_p)]),
    "sllm_total_bytes": (C.c_uint64, [C.c_void_p]),
    "sllm_load": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_uint64, C.c_void_p]),
    "sllm_repack": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_uint64, C.c_void_p, C.c_uint64, C.c_void_p]),
    "sllm_repack_noalloc": (C.c_int32, [C.c_void_p, C.c_uint64, C.c_void_p, C.c_uint64, C.c_void_p, C.c_uint64,
                                        C.c_void_p]),
    "sllm_tensor_index": (C.c_int32, [C.c_void_p, C.POINTER(TensorInfo), C.c_uint64, C.POINTER(C.c_uint64)]),
    "sllm_tensor_find": (C.c_int32, [C.c_void_p, C.c_char_p, C.POINTER(TensorInfo)]),
    "sllm_get_stats": (C.c_int32, [C.c_void_p, C.POINTER(Stats)]),
    "sllm_close": (C.c_int32, [C.c_void_p]),
    "sllm_export_create": (C.c_int32, [C.c_void_p, C.c_uint64, C.c_int32, C.c_void_p, C.POINTER(IpcDesc),
                                       C.POINTER(C.c_void_p)]),
    "sllm_export_destroy": (C.c_int32, [C.c_void_p]),
    "sllm_import_open": (C.c_int32, [C.POINTER(IpcDesc), C.c_void_p, C.POINTER(C.c_void_p), C.POINTER(C.c_void_p)]),
    "sllm_import_close": (C.c_int32, [C.c_void_p]),
    "sllm_estimator_create": (C.c_int32, [C.c_double, C.c_double, C.c_double, C.POINTER(C.c_void_p)]),
    "sllm_estimator_destroy": (None, [C.c_void_p]),
    "sllm_estimator_query": (C.c_int32, [C.c_void_p, C.c_uint64, C.c_uint32, C.POINTER(C.c_double)]),
    "sllm_estimator_enqueue": (C.c_int32, [C.c_void_p, C.c_uint64, C.c_uint32, C.POINTER(C.c_uint64),
                                           C.POINTER(C.c_double)]),
    "sllm_estimator_complete": (C.c_int32, [C.c_void_p, C.c_uint64, C.c_double]),
    "sllm_estimator_complete_load": (C.c_int32, [C.c_void_p, C.c_uint64, C.c_void_p]),
    "sllm_estimator_bandwidth": (C.c_int32, [C.c_void_p, C.c_uint32, C.POINTER(C.c_double)]),
    "sllm_last_error": (C.c_char_p, []),
    "sllm_strerror": (C.c_char_p, [C.c_int32]),
}

_lib: Optional[C.CDLL] = None


def _hip_runtimes() -> List[str]:
    """Paths of the HIP runtime libraries mapped into this process."""
    paths = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                p = line.split()[-1]
                if "libamdhip64" in os.path.basename(p):
                    paths.add(os.path.realpath(p))
    except OSError:
        pass
    return sorted(paths)


def lib() -> C.CDLL:
    """The loaded library (raises if it has not been built).

    torch ships its own HIP runtime under the same soname.  It is imported
    first so that the library binds to that one runtime: stream handles and
    device pointers from torch are only meaningful to the runtime that made
    them, and a second runtime in the process finds no device."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with python -m paper_2401_14351_amd.build")
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        handle = C.CDLL(LIB_PATH)
        runtimes = _hip_runtimes()
        if len(runtimes) > 1:
            raise RuntimeError(f"two HIP runtimes are loaded ({', '.join(runtimes)}); load torch before "
                               f"{os.path.basename(LIB_PATH)}")
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


class SllmError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{ERRORS.get(code, code)}: {message}")
        self.code = code
        self.message = message


def check(rc: int) -> None:
    if rc != SLLM_OK:
        raise SllmError(rc, lib().sllm_last_error().decode(errors="replace"))


# ---------------------------------------------------------------------------
# conversion
# ---------------------------------------------------------------------------

def _src_tensor(name: str, dtype: str, shape: Sequence[int], data) -> Tuple[SrcTensor, tuple]:
    """Describe one tensor; returns the struct and the objects it points into."""
    mv = memoryview(data).cast("B") if not hasattr(data, "data_ptr") else None
    if mv is not None:
        nbytes = mv.nbytes
        ptr = C.addressof(C.c_char.from_buffer(mv)) if nbytes and not mv.readonly else None
        keep: tuple = (mv,)
        if nbytes and ptr is None:  # read-only buffer: borrow its address through a bytes copy
            buf = C.create_string_buffer(mv.tobytes(), nbytes)
            ptr, keep = C.addressof(buf), (buf,)
    else:  # a contiguous CPU torch tensor
        nbytes = data.numel() * data.element_size()
        ptr, keep = data.data_ptr(), (data,)
    shp = (C.c_int64 * max(1, len(shape)))(*[int(d) for d in shape])
    raw = name.encode("utf-8")
    st = SrcTensor(raw, DTYPE_CODE[dtype], len(shape), shp, ptr or None, nbytes)
    return st, keep + (shp, raw)


def convert(tensors: Iterable[Tuple[str, str, Sequence[int], object]], out_dir: str, alignment: int = 256,
            chunk_size: int = 16 << 20, fsync: bool = False) -> None:
    """``sllm_writer_*`` over an iterable of (name, dtype, shape, bytes-like).

    Tensors are written as they arrive, so a generator never has to hold the
    whole checkpoint in memory."""
    L = lib()
    opts = ConvertOpts(alignment, chunk_size, CONVERT_FSYNC if fsync else 0, 0)
    w = C.c_void_p()
    os.makedirs(out_dir, exist_ok=True)
    check(L.sllm_writer_open(out_dir.encode(), C.byref(opts), C.byref(w)))
    try:
        for name, dtype, shape, data in tensors:
            st, keep = _src_tensor(name, dtype, shape, data)
            check(L.sllm_writer_add(w, C.byref(st)))
            del keep
    except BaseException:
        L.sllm_writer_abort(w)
        raise
    check(L.sllm_writer_close(w))


def convert_array(tensors: Sequence[Tuple[str, str, Sequence[int], object]], out_dir: str, alignment: int = 256,
                  chunk_size: int = 16 << 20, fsync: bool = False) -> None:
    """``sllm_convert`` over a list held in memory."""
    L = lib()
    structs, keep = [], []
    for t in tensors:
        st, k = _src_tensor(*t)
        structs.append(st)
        keep.append(k)
    arr = (SrcTensor * max(1, len(structs)))(*structs)
    opts = ConvertOpts(alignment, chunk_size, CONVERT_FSYNC if fsync else 0, 0)
    os.makedirs(out_dir, exist_ok=True)
    check(L.sllm_convert(arr, len(structs), out_dir.encode(), C.byref(opts)))


def convert_safetensors(paths: Sequence[str], out_dir: str, alignment: int = 256,
                        chunk_size: int = 16 << 20) -> None:
    """``sllm_convert_safetensors`` over one or more shards."""
    arr = (C.c_char_p * max(1, len(paths)))(*[p.encode() for p in paths])
    opts = ConvertOpts(alignment, chunk_size, 0, 0)
    os.makedirs(out_dir, exist_ok=True)
    check(lib().sllm_convert_safetensors(arr, len(paths), out_dir.encode(), C.byref(opts)))


# ---------------------------------------------------------------------------
# pool, open, load
# ---------------------------------------------------------------------------

def _stream_ptr(stream) -> Optional[int]:
    if stream is None:
        return None
    return getattr(stream, "cuda_stream", stream)


class Pool:
    """The pinned host chunk pool (the DRAM tier)."""

    def __init__(self, chunk_size: int, n_chunks: int, device: int = 0):
        self._h = C.c_void_p()
        check(lib().sllm_pool_create(chunk_size, n_chunks, device, C.byref(self._h)))
        self.device = device

    @property
    def handle(self):
        return self._h

    def cache(self, ckpt_dir: str, io_threads: int = 4, direct_io: bool = False) -> None:
        check(lib().sllm_pool_cache(self._h, ckpt_dir.encode(), io_threads, OPEN_DIRECT_IO if direct_io else 0))

    def evict(self, ckpt_dir: str) -> None:
        check(lib().sllm_pool_evict(self._h, ckpt_dir.encode()))

    def info(self) -> Dict[str, int]:
        inf = PoolInfo()
        check(lib().sllm_pool_query(self._h, C.byref(inf)))
        return {f: getattr(inf, f) for f, _ in PoolInfo._fields_}

    def close(self) -> None:
        if self._h:
            check(lib().sllm_pool_destroy(self._h))
            self._h = C.c_void_p()

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


class Tensor(NamedTuple):
    """One entry of the tensor index: offset is o_i (or d_i with a device
    layout), nbytes the unpadded size."""

    name: str
    dtype: str
    shape: Tuple[int, ...]
    offset: int
    nbytes: int


class Checkpoint:
    """An open converted checkpoint (``sllm_open`` ... ``sllm_close``)."""

    def __init__(self, ckpt_dir: str, device: int = 0, pool: Optional[Pool] = None, chunk_size: int = 0,
                 dev_alignment: int = 0, io_threads: int = 4, n_streams: int = 2, ring_slots: int = 0,
                 engine: str = "kernel", direct_io: bool = False, timing: bool = False, index_only: bool = False,
                 cache: bool = False):
        """cache=True (SLLM_OPEN_CACHE): the first load streams into one chunk
        of ``pool`` per partition chunk and leaves the checkpoint cached there."""
        flags = (OPEN_DIRECT_IO if direct_io else 0) | (OPEN_TIMING if timing else 0) | \
            (OPEN_INDEX_ONLY if index_only else 0) | (OPEN_CACHE if cache else 0)
        opts = OpenOpts(chunk_size, dev_alignment, pool.handle if pool else None, io_threads, n_streams,
                        ring_slots, ENGINE[engine], flags, device)
        self._h = C.c_void_p()
        check(lib().sllm_open(ckpt_dir.encode(), C.byref(opts), C.byref(self._h)))
        self.device = device
        self.dir = ckpt_dir

    @property
    def total_bytes(self) -> int:
        return int(lib().sllm_total_bytes(self._h))

    def tensors(self) -> List[Tensor]:
        n = C.c_uint64()
        check(lib().sllm_tensor_index(self._h, None, 0, C.byref(n)))
        if n.value == 0:
            return []
        arr = (TensorInfo * n.value)()
        check(lib().sllm_tensor_index(self._h, arr, n.value, C.byref(n)))
        # decode the whole table at once (per-field ctypes access costs
        # microseconds per tensor, which adds up at 20,000 tensors)
        raw = np.frombuffer(arr, dtype=_TENSOR_INFO, count=n.value)
        names = [C.string_at(p).decode() for p in raw["name"].tolist()]
        return [Tensor(nm, CODE_DTYPE[dt], tuple(sh[:nd]), off, nb)
                for nm, dt, nd, sh, off, nb in zip(names, raw["dtype"].tolist(), raw["ndim"].tolist(),
                                                   raw["shape"].tolist(), raw["offset"].tolist(),
                                                   raw["nbytes"].tolist())]

    def find(self, name: str) -> Tensor:
        t = TensorInfo()
        check(lib().sllm_tensor_find(self._h, name.encode(), C.byref(t)))
        return Tensor(t.name.decode(), CODE_DTYPE[t.dtype], tuple(t.shape[:t.ndim]), t.offset, t.nbytes)

    def load(self, dst_ptr: int, dst_bytes: int, stream=None) -> None:
        check(lib().sllm_load(self._h, dst_ptr, dst_bytes, _stream_ptr(stream)))

    def load_into(self, buf, stream=None) -> None:
        """Load into a contiguous uint8 torch tensor on the handle's device
        (it may be a slice of a larger allocation)."""
        _check_buffer(buf)
        self.load(buf.data_ptr(), buf.numel(), stream)

    def load_with_views(self, buf, stream=None, after_load: Optional[Callable[[], None]] = None):
        """Load into ``buf`` while this thread builds the tensor views
        (``sllm_load`` runs on a helper thread; ctypes releases the GIL during
        the call) when there are many tensors, else load then build them.  ``after_load`` runs on that thread once the load is
        enqueued.  Returns ``{name: view}``; the data are ready once
        ``stream`` has been synchronized."""
        n = C.c_uint64()
        check(lib().sllm_tensor_index(self._h, None, 0, C.byref(n)))
        if n.value < _THREADED_VIEWS_MIN:  # a helper thread costs more than these views
            self.load_into(buf, stream)
            if after_load is not None:
                after_load()
            return views(buf, self.tensors())
        err: List[BaseException] = []

        def run():
            try:
                self.load_into(buf, stream)
                if after_load is not None:
                    after_load()
            except BaseException as e:  # re-raised on the calling thread
                err.append(e)

        th = threading.Thread(target=run, name="sllm-load")
        th.start()
        view_err = None
        try:
            out = views(buf, self.tensors())
        except BaseException as e:  # e.g. a buffer too small for the views
            view_err = e
        th.join()
        if err:  # the load's own error says more (SLLM_E_RANGE for a short buffer)
            raise err[0]
        if view_err is not None:
            raise view_err
        return out

    def repack(self, src, dst, stream=None) -> None:
        _check_buffer(src)
        _check_buffer(dst)
        check(lib().sllm_repack(self._h, src.data_ptr(), src.numel(), dst.data_ptr(), dst.numel(),
                                _stream_ptr(stream)))

    def repack_noalloc(self, src, dst, dev_alignment: int = 0, stream=None) -> None:
        """sllm_repack_noalloc: the repack into alignment ``dev_alignment``
        (0: the handle's) with no device allocation."""
        _check_buffer(src)
        _check_buffer(dst)
        check(lib().sllm_repack_noalloc(self._h, dev_alignment, src.data_ptr(), src.numel(), dst.data_ptr(),
                                        dst.numel(), _stream_ptr(stream)))

    def stats(self) -> Dict[str, float]:
        s = Stats()
        check(lib().sllm_get_stats(self._h, C.byref(s)))
        return {f: getattr(s, f) for f, _ in Stats._fields_}

    def close(self) -> None:
        if self._h:
            check(lib().sllm_close(self._h))
            self._h = C.c_void_p()

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def _check_buffer(buf) -> None:
    """Device buffers handed to the library are flat runs of bytes: the C ABI
    sees only data_ptr() and numel(), so anything else would be misread."""
    import torch

    if buf.dtype != torch.uint8 or buf.dim() != 1 or not buf.is_contiguous():
        raise ValueError(f"expected a contiguous 1-d uint8 tensor, got {buf.dtype} with shape "
                         f"{tuple(buf.shape)} and strides {buf.stride()}")


def views(buf, tensors: Sequence[Tensor]) -> Dict[str, object]:
    """torch views of each tensor at base + offset in ``buf`` (uint8).

    ``buf`` may start anywhere inside its storage (a slice of a larger
    allocation): offsets count from ``buf``'s first byte.  A tensor whose
    address is not a multiple of its element size (a dense file layout,
    A < itemsize, or a buffer that starts off that alignment) is returned as
    its raw uint8 bytes."""
    import torch

    _check_buffer(buf)
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16, "i8": torch.int8}
    typed = {}
    out = {}
    for t in tensors:
        isz = ITEMSIZE[DTYPE_CODE[t.dtype]]
        if buf.storage_offset() % isz or t.offset % isz:
            out[t.name] = buf[t.offset:t.offset + t.nbytes]
            continue
        base = typed.get(t.dtype)
        if base is None:
            base = buf[: (buf.numel() // isz) * isz].view(tdt[t.dtype])
            typed[t.dtype] = base
        # as_strided counts its offset from the start of the storage, not
        # from the start of the typed view
        out[t.name] = base.as_strided(t.shape, _contiguous_strides(t.shape),
                                      base.storage_offset() + t.offset // isz)
    return out


@functools.lru_cache(maxsize=4096)
def _contiguous_strides(shape: Tuple[int, ...]) -> Tuple[int, ...]:
    stride, acc = [], 1
    for d in reversed(shape):
        stride.append(acc)
        acc *= max(int(d), 1)
    return tuple(reversed(stride))


def load(ckpt_dir: str, device: int = 0, stream=None, pool: Optional[Pool] = None, **opts):
    """Open, load into a fresh uint8 device buffer, build views, synchronize.

    Returns ``(buffer, {name: tensor view})``; the data are ready on return."""
    import torch

    with Checkpoint(ckpt_dir, device=device, pool=pool, **opts) as ck:
        buf = torch.empty(max(ck.total_bytes, 1), dtype=torch.uint8, device=f"cuda:{device}")
        s = stream if stream is not None else torch.cuda.current_stream(device)
        out = ck.load_with_views(buf, s)
        s.synchronize()
    return buf, out


def device_tensor(ptr: int, nbytes: int, device: int = 0):
    """A uint8 torch tensor over device memory this process did not allocate
    (an imported buffer), through the CUDA array interface."""
    import torch

    class _Mem:
        __cuda_array_interface__ = {"shape": (nbytes,), "typestr": "|u1", "data": (ptr, False), "version": 3}

    return torch.as_tensor(_Mem(), device=f"cuda:{device}")


class Export:
    """Share a loaded uint8 device buffer with another process (``sllm_export_*``).

    The handoff event is recorded on ``stream`` after the work queued there,
    so export right after ``Checkpoint.load_into(buf, stream)``.  The whole
    device allocation holding ``buf`` is shared, so give the buffer its own
    allocation (a block of torch's caching allocator may sit inside a segment
    larger than ``SLLM_IPC_MAX_ALLOCATION``)."""

    def __init__(self, buf, stream=None, device: int = 0):
        self.desc = IpcDesc()
        self._h = C.c_void_p()
        check(lib().sllm_export_create(buf.data_ptr(), buf.numel(), device, _stream_ptr(stream), C.byref(self.desc),
                                       C.byref(self._h)))
        self._buf = buf  # the shared memory must outlive the export

    @property
    def desc_bytes(self) -> bytes:
        return bytes(self.desc)

    def close(self) -> None:
        if self._h:
            check(lib().sllm_export_destroy(self._h))
            self._h = C.c_void_p()
            self._buf = None


class Import:
    """Map a buffer exported by another process; ``stream`` waits for its load."""

    def __init__(self, desc: bytes, stream=None):
        if len(desc) != C.sizeof(IpcDesc):
            raise ValueError("not an sllm_ipc_desc")
        self.desc = IpcDesc.from_buffer_copy(desc)
        ptr, self._h = C.c_void_p(), C.c_void_p()
        check(lib().sllm_import_open(C.byref(self.desc), _stream_ptr(stream), C.byref(ptr), C.byref(self._h)))
        self.ptr = ptr.value

    def tensor(self):
        return device_tensor(self.ptr, self.desc.bytes, self.desc.device)

    def close(self) -> None:
        if self._h:
            check(lib().sllm_import_close(self._h))
            self._h = C.c_void_p()


TIER_DRAM = 1
TIER_STORAGE = 2


class Estimator:
    """Loading-time estimate q + n / b (``sllm_estimator_*``)."""

    def __init__(self, dram_bytes_per_s: float, storage_bytes_per_s: float, weight: float = 0.5):
        self._h = C.c_void_p()
        check(lib().sllm_estimator_create(dram_bytes_per_s, storage_bytes_per_s, weight, C.byref(self._h)))

    def query(self, nbytes: int, tiers: int) -> float:
        out = C.c_double()
        check(lib().sllm_estimator_query(self._h, int(nbytes), tiers, C.byref(out)))
        return out.value

    def enqueue(self, nbytes: int, tiers: int) -> Tuple[int, float]:
        task, eta = C.c_uint64(), C.c_double()
        check(lib().sllm_estimator_enqueue(self._h, int(nbytes), tiers, C.byref(task), C.byref(eta)))
        return task.value, eta.value

    def complete(self, task: int, seconds: float) -> None:
        check(lib().sllm_estimator_complete(self._h, task, seconds))

    def complete_load(self, task: int, ckpt: "Checkpoint") -> None:
        """Complete ``task`` with the time ``ckpt``'s last load took, from the
        handle's own counters (sllm_estimator_complete_load)."""
        check(lib().sllm_estimator_complete_load(self._h, task, ckpt._h))

    def bandwidth(self, tier: int) -> float:
        out = C.c_double()
        check(lib().sllm_estimator_bandwidth(self._h, tier, C.byref(out)))
        return out.value

    def close(self) -> None:
        if self._h:
            lib().sllm_estimator_destroy(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
