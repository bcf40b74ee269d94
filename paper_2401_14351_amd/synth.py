"""Seeded synthetic checkpoints shaped like the models the paper loads (Sec. 7.2).

This module produces *inputs only*: tensor names, dtypes, shapes and raw bytes.
It holds no part of the loading method's arithmetic (no offsets, alignment,
padding or chunk geometry) so that both the CPU oracle and the GPU path can be
fed from it without sharing any of the method's code.

Value recipe (the paper's checkpoints are real FP16 weights; load time depends
only on checkpoint size, Sec. 7.2, so synthetic values of the same shapes stand
in for them):

* Weights are N(0, 0.02) drawn as float32 from PCG64 and rounded to the stored
  dtype with IEEE round-to-nearest-even (fp16, bf16).
* Llama RMSNorm weights are exactly 1.0.
* The many-small-tensor stress set stores uniform random bytes, so its payload
  contains NaNs, infinities and signed zeros: compare it as bytes only.

Every tensor's bytes depend only on (seed, tensor position, block position):
element block ``b`` (``BLOCK`` elements) of tensor ``i`` is drawn from
``PCG64(SeedSequence([seed, i, b]))``, so generation can run on any number of
threads and still give the same bytes.
"""

from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Iterator, List, Optional, Sequence, Tuple

import numpy as np

#: element size in bytes of each stored dtype
ITEMSIZE = {"f32": 4, "f16": 2, "bf16": 2, "i8": 1}
DTYPES = tuple(ITEMSIZE)

#: elements per independently seeded generation block
BLOCK = 1 << 22

MiB = 1 << 20
KiB = 1 << 10


@dataclass(frozen=True)
class TensorSpec:
    name: str
    dtype: str
    shape: Tuple[int, ...]
    init: str = "normal"  # "normal" (N(0, 0.02)), "ones" or "bytes" (uniform random bytes)

    @property
    def numel(self) -> int:
        return math.prod(self.shape)  # a 0-d tensor holds one element

    @property
    def nbytes(self) -> int:
        return self.numel * ITEMSIZE[self.dtype]


@dataclass
class CheckpointSpec:
    """A synthetic checkpoint: ordered tensors plus the conversion parameters
    the workload names (file alignment A in bytes, load chunk size C in bytes)."""

    name: str
    seed: int
    alignment: int
    chunk_size: int
    tensors: List[TensorSpec] = field(default_factory=list)

    @property
    def payload_bytes(self) -> int:
        return sum(t.nbytes for t in self.tensors)


# ----------------------------------------------------------------------------
# model-shaped tensor lists (Hugging Face state-dict names and order)
# ----------------------------------------------------------------------------

def opt_125m(seed: int = 1001) -> CheckpointSpec:
    """OPT-125M: 12 layers, hidden 768, FFN 3072, vocab 50272, 2048 positions
    (+2 learned-position offset rows), fp16; lm_head is tied so it is not stored."""
    d, ffn, vocab, layers = 768, 3072, 50272, 12
    t: List[TensorSpec] = [
        TensorSpec("model.decoder.embed_tokens.weight", "f16", (vocab, d)),
        TensorSpec("model.decoder.embed_positions.weight", "f16", (2048 + 2, d)),
    ]
    for l in range(layers):
        p = f"model.decoder.layers.{l}."
        for proj in ("k_proj", "v_proj", "q_proj", "out_proj"):
            t.append(TensorSpec(p + f"self_attn.{proj}.weight", "f16", (d, d)))
            t.append(TensorSpec(p + f"self_attn.{proj}.bias", "f16", (d,)))
        t.append(TensorSpec(p + "self_attn_layer_norm.weight", "f16", (d,)))
        t.append(TensorSpec(p + "self_attn_layer_norm.bias", "f16", (d,)))
        t.append(TensorSpec(p + "fc1.weight", "f16", (ffn, d)))
        t.append(TensorSpec(p + "fc1.bias", "f16", (ffn,)))
        t.append(TensorSpec(p + "fc2.weight", "f16", (d, ffn)))
        t.append(TensorSpec(p + "fc2.bias", "f16", (d,)))
        t.append(TensorSpec(p + "final_layer_norm.weight", "f16", (d,)))
        t.append(TensorSpec(p + "final_layer_norm.bias", "f16", (d,)))
    t.append(TensorSpec("model.decoder.final_layer_norm.weight", "f16", (d,)))
    t.append(TensorSpec("model.decoder.final_layer_norm.bias", "f16", (d,)))
    return CheckpointSpec("opt-125m", seed, alignment=256, chunk_size=16 * MiB, tensors=t)


_LLAMA = {
    # size: (layers, d, query heads, kv heads, ffn)
    "7b": (32, 4096, 32, 32, 11008),
    "13b": (40, 5120, 40, 40, 13824),
    "70b": (80, 8192, 64, 8, 28672),
}
_LLAMA_SEED = {"7b": 1002, "13b": 1003, "70b": 1004}
_LLAMA_CHUNK = {"7b": 16 * MiB, "13b": 16 * MiB, "70b": 64 * MiB}


def llama2(size: str, seed: Optional[int] = None, chunk_size: Optional[int] = None) -> CheckpointSpec:
    """Llama-2-{7b,13b,70b}: bf16, head dim 128, vocab 32000, untied lm_head,
    RMSNorm weights 1.0.  70b uses grouped-query attention with 8 KV heads."""
    layers, d, nq, nkv, ffn = _LLAMA[size]
    vocab, hd = 32000, d // nq
    kv = nkv * hd
    t: List[TensorSpec] = [TensorSpec("model.embed_tokens.weight", "bf16", (vocab, d))]
    for l in range(layers):
        p = f"model.layers.{l}."
        t.append(TensorSpec(p + "self_attn.q_proj.weight", "bf16", (d, d)))
        t.append(TensorSpec(p + "self_attn.k_proj.weight", "bf16", (kv, d)))
        t.append(TensorSpec(p + "self_attn.v_proj.weight", "bf16", (kv, d)))
        t.append(TensorSpec(p + "self_attn.o_proj.weight", "bf16", (d, d)))
        t.append(TensorSpec(p + "mlp.gate_proj.weight", "bf16", (ffn, d)))
        t.append(TensorSpec(p + "mlp.up_proj.weight", "bf16", (ffn, d)))
        t.append(TensorSpec(p + "mlp.down_proj.weight", "bf16", (d, ffn)))
        t.append(TensorSpec(p + "input_layernorm.weight", "bf16", (d,), init="ones"))
        t.append(TensorSpec(p + "post_attention_layernorm.weight", "bf16", (d,), init="ones"))
    t.append(TensorSpec("model.norm.weight", "bf16", (d,), init="ones"))
    t.append(TensorSpec("lm_head.weight", "bf16", (vocab, d)))
    return CheckpointSpec(
        f"llama-2-{size}",
        _LLAMA_SEED[size] if seed is None else seed,
        alignment=256,
        chunk_size=_LLAMA_CHUNK[size] if chunk_size is None else chunk_size,
        tensors=t,
    )


def lora(size: str = "70b", rank: int = 32, seed: int = 1006) -> CheckpointSpec:
    """A LoRA adapter for a Llama-2 model (PEFT names): rank-`rank` A and B
    matrices on all seven linear modules of every layer, bf16 N(0, 0.02).
    For 70b at rank 32 this is 1,120 tensors and 0.83 GB, close to the 1 GB
    rank-32 LLaMA-70B adapter the paper loads (Sec. 7.2)."""
    layers, d, nq, nkv, ffn = _LLAMA[size]
    kv = nkv * (d // nq)
    dims = {"self_attn.q_proj": (d, d), "self_attn.k_proj": (d, kv), "self_attn.v_proj": (d, kv),
            "self_attn.o_proj": (d, d), "mlp.gate_proj": (d, ffn), "mlp.up_proj": (d, ffn),
            "mlp.down_proj": (ffn, d)}
    t: List[TensorSpec] = []
    for l in range(layers):
        for mod, (d_in, d_out) in dims.items():
            p = f"base_model.model.model.layers.{l}.{mod}."
            t.append(TensorSpec(p + "lora_A.weight", "bf16", (rank, d_in)))
            t.append(TensorSpec(p + "lora_B.weight", "bf16", (d_out, rank)))
    return CheckpointSpec(f"lora-{size}-r{rank}", seed, alignment=256, chunk_size=16 * MiB, tensors=t)


def huge_tensor(seed: int = 1007) -> CheckpointSpec:
    """One int8 tensor of 65,537 x 65,539 = 4,295,229,443 bytes (just over
    2^32) between small tensors of odd byte sizes, uniform random bytes,
    packed densely (A = 1): the tensor starts at an odd file offset, and
    bytes inside it lie more than 4 GiB from its start."""
    t = [TensorSpec("head.bias", "bf16", (1531,), "bytes"),
         TensorSpec("huge.weight", "i8", (65537, 65539), "bytes"),
         TensorSpec("tail.scale", "f32", (3,), "bytes"),
         TensorSpec("tail.weight", "f16", (4097, 3), "bytes")]
    return CheckpointSpec("huge-tensor", seed, alignment=1, chunk_size=16 * MiB, tensors=t)


def _prime_factors(n: int) -> List[int]:
    out, p = [], 2
    while p * p <= n:
        while n % p == 0:
            out.append(p)
            n //= p
        p += 1
    if n > 1:
        out.append(n)
    return out


def stress(n: int = 20000, seed: int = 1005, min_bytes: int = 256, max_bytes: int = 64 * MiB,
           cap_payload: Optional[int] = None) -> CheckpointSpec:
    """Many-small-tensor stress set: byte sizes log-uniform in [min_bytes, max_bytes],
    dtype uniform over f32/f16/bf16/i8, size rounded down to a whole number of
    elements (at least one), ndim uniform in 1..4 with the prime factors of
    numel spread at random over the dims, uniform random bytes, 4 KiB file
    alignment and 1 MiB chunks.

    ``cap_payload`` keeps only the leading tensors whose summed unpadded size
    stays within that many bytes (the same tensors and bytes as the full set).
    """
    meta = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0xFFFF_FFFF])))
    lo, hi = math.log(min_bytes), math.log(max_bytes)
    t: List[TensorSpec] = []
    total = 0
    for i in range(n):
        size = int(math.exp(meta.uniform(lo, hi)))
        dtype = DTYPES[int(meta.integers(0, len(DTYPES)))]
        isz = ITEMSIZE[dtype]
        numel = max(1, size // isz)
        ndim = int(meta.integers(1, 5))
        dims = [1] * ndim
        for f in _prime_factors(numel):
            dims[int(meta.integers(0, ndim))] *= f
        spec = TensorSpec(f"stress.{i:05d}", dtype, tuple(dims), init="bytes")
        if cap_payload is not None and total + spec.nbytes > cap_payload:
            break
        total += spec.nbytes
        t.append(spec)
    return CheckpointSpec("stress" if cap_payload is None else f"stress-cap{cap_payload}",
                          seed, alignment=4 * KiB, chunk_size=1 * MiB, tensors=t)


def tiny(seed: int, n: int = 12, alignment: int = 16, chunk_size: int = 64,
         max_bytes: int = 300) -> CheckpointSpec:
    """A small checkpoint for brute-force checks: random dtypes, 0-d tensors,
    zero-size tensors and sizes on both sides of the alignment."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0xFFFF_FFFE])))
    t: List[TensorSpec] = []
    for i in range(n):
        dtype = DTYPES[int(rng.integers(0, len(DTYPES)))]
        isz = ITEMSIZE[dtype]
        kind = int(rng.integers(0, 6))
        if kind == 0:
            shape: Tuple[int, ...] = ()                                  # 0-d: one element
        elif kind == 1:
            shape = (int(rng.integers(0, 3)), 0)                          # zero-size
        elif kind == 2:
            shape = (max(1, (alignment + int(rng.integers(-1, 2))) // isz),)   # near A
        else:
            numel = int(rng.integers(1, max(2, max_bytes // isz)))
            shape = (numel,) if kind == 3 else (1, numel) if kind == 4 else (numel, 1, 1)
        t.append(TensorSpec(f"t{i}.{dtype}", dtype, shape, init="bytes" if i % 3 == 0 else "normal"))
    return CheckpointSpec(f"tiny-{seed}", seed, alignment=alignment, chunk_size=chunk_size, tensors=t)


# ----------------------------------------------------------------------------
# value generation
# ----------------------------------------------------------------------------

def _bits_of(values_f32: np.ndarray, dtype: str) -> np.ndarray:
    """float32 values -> stored bit patterns (round-to-nearest-even)."""
    import torch

    if dtype == "f32":
        return values_f32
    src = torch.from_numpy(values_f32)
    if dtype == "f16":
        return src.to(torch.float16).view(torch.int16).numpy()
    if dtype == "bf16":
        return src.to(torch.bfloat16).view(torch.int16).numpy()
    raise ValueError(dtype)


def block_size(t: TensorSpec) -> int:
    """Bytes of one generation block of ``t`` (the last block may be shorter)."""
    return BLOCK * ITEMSIZE[t.dtype]


def fill_block(spec: CheckpointSpec, i: int, t: TensorSpec, b: int, out: np.ndarray) -> None:
    """Fill ``out`` (uint8 bytes of element block b of tensor i)."""
    isz = ITEMSIZE[t.dtype]
    n_el = out.size // isz
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([spec.seed, i, b])))
    if t.init == "bytes":
        out[:] = rng.integers(0, 256, size=out.size, dtype=np.uint8)
        return
    if t.init == "ones":
        vals = np.ones(n_el, dtype=np.float32)
    else:
        vals = rng.standard_normal(n_el, dtype=np.float32)
        vals *= np.float32(0.02)
    if t.dtype == "i8":
        # int8 weights: the N(0, 0.02) draw scaled to the int8 range and rounded
        q = np.clip(np.rint(vals * np.float32(127.0 / 0.1)), -128, 127).astype(np.int8)
        out[:] = q.view(np.uint8)
        return
    out[:] = _bits_of(vals, t.dtype).view(np.uint8)


def tensor_bytes(spec: CheckpointSpec, i: int, pool: Optional[ThreadPoolExecutor] = None) -> np.ndarray:
    """Raw little-endian bytes of tensor ``i`` as a fresh uint8 array."""
    t = spec.tensors[i]
    out = np.empty(t.nbytes, dtype=np.uint8)
    step = block_size(t)
    jobs = [(b, out[b * step:(b + 1) * step]) for b in range((t.nbytes + step - 1) // step)]
    if pool is None or len(jobs) <= 1:
        for b, o in jobs:
            fill_block(spec, i, t, b, o)
    else:
        list(pool.map(lambda job: fill_block(spec, i, t, job[0], job[1]), jobs))
    return out


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def iter_tensors(spec: CheckpointSpec, threads: Optional[int] = None,
                 indices: Optional[Sequence[int]] = None) -> Iterator[Tuple[int, TensorSpec, np.ndarray]]:
    """Yield ``(i, spec_i, bytes_i)`` in order, generating on a thread pool."""
    idx = range(len(spec.tensors)) if indices is None else indices
    with ThreadPoolExecutor(threads or default_threads()) as pool:
        for i in idx:
            yield i, spec.tensors[i], tensor_bytes(spec, i, pool)


def materialize(spec: CheckpointSpec, threads: Optional[int] = None) -> List[np.ndarray]:
    """All tensors' bytes in order (small checkpoints only)."""
    return [b for _, _, b in iter_tensors(spec, threads)]


def config(name: str) -> CheckpointSpec:
    """The five benchmark workloads by name, plus the capped stress variant
    (and that variant converted densely, for repacks whose shifts are not
    multiples of 16 bytes), the LoRA adapter and the checkpoint with one
    tensor over 4 GiB."""
    if name == "opt-125m":
        return opt_125m()
    if name.startswith("llama-2-"):
        return llama2(name[len("llama-2-"):])
    if name == "stress":
        return stress()
    if name == "stress-8g":
        return stress(cap_payload=8 << 30)
    if name == "stress-8g-dense":  # the same tensors packed with no alignment (A = 1)
        spec = stress(cap_payload=8 << 30)
        spec.name, spec.alignment = spec.name + "-dense", 1
        return spec
    if name == "lora-70b-r32":
        return lora("70b", 32)
    if name == "huge-tensor":
        return huge_tensor()
    raise KeyError(name)


WORKLOADS = ("opt-125m", "llama-2-7b", "llama-2-13b", "llama-2-70b", "stress")
