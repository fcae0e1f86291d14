"""Seeded synthetic workloads for the decode-maximal hybrid-batch layer.

This module is shared by the tests, the benchmark and the oracle's callers.
It draws random numbers and lays them out; it holds none of the layer's
arithmetic (no norm, projection, rotation or attention), so neither the HIP
path nor the oracle depends on the other through it.

Shapes follow the paper's model settings (Sec. 4.5: LLaMA-13B is 40 layers,
40 heads, hidden 5120; LLaMA-33B 60 layers, 52 heads, hidden 6656; GPT-3 96
layers, 96 heads, hidden 12288).  FFN widths, norm kind, activation and rotary
embedding are not in the paper; they are the public LLaMA / GPT-3 settings.

Recipe (the same for every workload):
  * numpy ``Generator(PCG64(seed))``, seed 0;
  * draw order: decode context lengths -> slot permutation -> X -> KV cache
    (slot by slot, K then V, valid positions only) -> W_qkv -> W_o -> W_up ->
    W_down -> g1 -> g2 (-> b1 -> b2 for LayerNorm);
  * weights 0.02 * N(0,1); norm gains 1 + 0.02 * N(0,1); LayerNorm biases
    0.02 * N(0,1); X and cached K/V N(0,1);
  * values are drawn in fp32 and, for bf16 workloads, rounded to bf16 with
    round-to-nearest-even, so both sides consume exactly the same numbers;
  * cache positions that hold no token yet carry a quiet-NaN sentinel, so an
    over-read poisons the outputs.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

BF16_NAN_BITS = np.uint16(0x7FC0)


@dataclass(frozen=True)
class LayerShape:
    """Decoder-layer shape.  ``norm`` in {"rms", "layer"}, ``act`` in
    {"swiglu", "gelu"}, ``dtype`` in {"f32", "bf16"}."""
    hidden: int
    n_heads: int
    head_dim: int
    ffn: int
    n_layers: int = 1
    norm: str = "rms"
    act: str = "swiglu"
    rope: bool = True
    rope_base: float = 10000.0
    eps: float = 1e-6
    dtype: str = "bf16"

    @property
    def up_rows(self) -> int:
        return 2 * self.ffn if self.act == "swiglu" else self.ffn


@dataclass(frozen=True)
class BatchSpec:
    """One decode-maximal batch: a chunk of ``chunk_len`` prompt tokens at
    ``chunk_offset`` plus ``n_decodes`` decodes whose context lengths are
    uniform integers in [ctx_lo, ctx_hi]."""
    chunk_len: int
    chunk_offset: int
    prompt_len: int
    n_decodes: int
    ctx_lo: int
    ctx_hi: int
    max_seq_len: int
    n_slots: int

    @property
    def n_tokens(self) -> int:
        return self.chunk_len + self.n_decodes


@dataclass(frozen=True)
class Workload:
    name: str
    shape: LayerShape
    batch: BatchSpec
    seed: int = 0
    steps: int = 1          # consecutive decode-maximal steps (model stack)
    description: str = ""


def _roundup(x: int, m: int) -> int:
    return (x + m - 1) // m * m


TINY = Workload(
    name="tiny-llama-layer-f32",
    shape=LayerShape(hidden=256, n_heads=4, head_dim=64, ffn=688, eps=1e-6, dtype="f32"),
    batch=BatchSpec(chunk_len=64, chunk_offset=128, prompt_len=256, n_decodes=8,
                    ctx_lo=32, ctx_hi=128, max_seq_len=256, n_slots=9),
    description="tiny LLaMA-style layer, fp32: H 256, 4x64 heads, SwiGLU 688; "
                "chunk 64 at offset 128 + 8 decodes, ctx U[32,128]",
)

LLAMA13B_LAYER = Workload(
    name="llama13b-layer-bf16-c256-b64",
    shape=LayerShape(hidden=5120, n_heads=40, head_dim=128, ffn=13824, dtype="bf16"),
    batch=BatchSpec(chunk_len=256, chunk_offset=512, prompt_len=1024, n_decodes=64,
                    ctx_lo=256, ctx_hi=1024, max_seq_len=1088, n_slots=65),
    description="LLaMA-13B-shaped layer, bf16: chunk 256 at offset 512 of a "
                "1024-token prompt + 64 decodes, ctx U[256,1024]",
)

LLAMA13B_STACK = Workload(
    name="llama13b-stack40-bf16-c256-b48",
    shape=LayerShape(hidden=5120, n_heads=40, head_dim=128, ffn=13824, n_layers=40, dtype="bf16"),
    batch=BatchSpec(chunk_len=256, chunk_offset=0, prompt_len=1024, n_decodes=48,
                    ctx_lo=512, ctx_hi=2048, max_seq_len=2112, n_slots=49),
    steps=4,
    description="LLaMA-13B-shaped 40-layer stack, bf16: 4 steps, each one 256-token "
                "chunk of a 1024 prompt + 48 decodes, ctx U[512,2048] (+1 per step)",
)


def llama33b_layer(chunk_len: int) -> Workload:
    return Workload(
        name=f"llama33b-layer-bf16-c{chunk_len}-b32",
        shape=LayerShape(hidden=6656, n_heads=52, head_dim=128, ffn=17920, dtype="bf16"),
        batch=BatchSpec(chunk_len=chunk_len, chunk_offset=2048, prompt_len=3072, n_decodes=32,
                        ctx_lo=1024, ctx_hi=3072, max_seq_len=3136, n_slots=33),
        description=f"LLaMA-33B-shaped layer, bf16: chunk {chunk_len} at offset 2048 + 32 "
                    "decodes, ctx U[1024,3072]",
    )


GPT3_LAYER = Workload(
    name="gpt3-layer-bf16-c256-b27",
    shape=LayerShape(hidden=12288, n_heads=96, head_dim=128, ffn=49152, norm="layer",
                     act="gelu", rope=False, eps=1e-5, dtype="bf16"),
    batch=BatchSpec(chunk_len=256, chunk_offset=1792, prompt_len=2048, n_decodes=27,
                    ctx_lo=1024, ctx_hi=2048, max_seq_len=2112, n_slots=28),
    description="GPT-3-175B-shaped layer, bf16: LayerNorm, GELU 49152, no RoPE; chunk 256 "
                "at offset 1792 + 27 decodes, ctx U[1024,2048]",
)

WORKLOADS = {w.name: w for w in
             [TINY, LLAMA13B_LAYER, LLAMA13B_STACK, llama33b_layer(128), llama33b_layer(256),
              llama33b_layer(512), GPT3_LAYER]}


def with_dtype(w: Workload, dtype: str) -> Workload:
    return dataclasses.replace(w, name=f"{w.name}@{dtype}",
                               shape=dataclasses.replace(w.shape, dtype=dtype))


# --------------------------------------------------------------------------- bf16 storage

def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns fp32
    holding exactly representable bf16 values.  NaN stays a quiet NaN."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # 32-bit arithmetic: the sum wraps only for bit patterns above 0xFFFF7FFF,
    # which are all NaNs (restored below)
    r = u + ((u >> 16) & np.uint32(1))
    r += np.uint32(0x7FFF)
    r &= np.uint32(0xFFFF0000)
    out = r.view(np.float32)
    nan = np.isnan(a)
    if nan.any():
        out = out.copy()
        out[nan] = np.float32(np.nan)
    return out


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 array holding bf16-exact values -> uint16 bf16 bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = (a.view(np.uint32) >> 16).astype(np.uint16)
    bits[np.isnan(a)] = BF16_NAN_BITS
    return bits


def bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns -> fp32 (exact)."""
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------- host instances

@dataclass
class Batch:
    """Concrete hybrid batch: rows 0..chunk_len-1 are the chunk (positions
    chunk_offset + r), then one row per decode in the given order."""
    prefill_slot: int
    chunk_offset: int
    chunk_len: int
    decode_slots: np.ndarray   # int32 [B]
    decode_ctx: np.ndarray     # int32 [B] tokens already cached per decode

    @property
    def n_decodes(self) -> int:
        return int(len(self.decode_slots))

    @property
    def n_tokens(self) -> int:
        return self.chunk_len + self.n_decodes


@dataclass
class MixedBatch:
    """Several prompt chunks plus decodes: chunks [(slot, offset, length)];
    rows are chunk 0 in position order, chunk 1, ..., then the decodes."""
    chunks: List[tuple]
    decode_slots: np.ndarray
    decode_ctx: np.ndarray

    @property
    def n_decodes(self) -> int:
        return int(len(self.decode_slots))

    @property
    def n_tokens(self) -> int:
        return sum(int(c[2]) for c in self.chunks) + self.n_decodes


@dataclass
class HostInstance:
    workload: Workload
    batch: Batch
    x: np.ndarray                        # [T, H] fp32 (bf16-exact for bf16)
    kv: np.ndarray                       # [L, n_slots, 2, nh, S, d] fp32, NaN where empty
    weights: List[dict] = field(default_factory=list)   # per layer, fp32 arrays

    @property
    def shape(self) -> LayerShape:
        return self.workload.shape


def _store(a: np.ndarray, dtype: str) -> np.ndarray:
    return round_to_bf16(a) if dtype == "bf16" else np.ascontiguousarray(a, dtype=np.float32)


def draw_batch(rng: np.random.Generator, spec: BatchSpec) -> Batch:
    ctx = rng.integers(spec.ctx_lo, spec.ctx_hi + 1, size=spec.n_decodes).astype(np.int32)
    perm = rng.permutation(spec.n_slots).astype(np.int32)
    return Batch(prefill_slot=int(perm[0]) if spec.chunk_len > 0 else -1,
                 chunk_offset=spec.chunk_offset, chunk_len=spec.chunk_len,
                 decode_slots=perm[1:1 + spec.n_decodes].copy(), decode_ctx=ctx)


def valid_lengths(batch, n_slots: int) -> np.ndarray:
    """Cached tokens per slot before the step (a chunk's slot: its offset)."""
    v = np.zeros(n_slots, dtype=np.int64)
    if isinstance(batch, MixedBatch):
        for s, o, _ in batch.chunks:
            v[int(s)] = int(o)
    elif batch.chunk_len > 0:
        v[batch.prefill_slot] = batch.chunk_offset
    for s, c in zip(batch.decode_slots, batch.decode_ctx):
        v[int(s)] = int(c)
    return v


def draw_weights(rng: np.random.Generator, shp: LayerShape) -> dict:
    H, nh, d, F = shp.hidden, shp.n_heads, shp.head_dim, shp.ffn
    f32 = np.float32
    w = {}
    w["w_qkv"] = _store(rng.standard_normal((3 * nh * d, H), dtype=f32) * f32(0.02), shp.dtype)
    w["w_o"] = _store(rng.standard_normal((H, nh * d), dtype=f32) * f32(0.02), shp.dtype)
    w["w_up"] = _store(rng.standard_normal((shp.up_rows, H), dtype=f32) * f32(0.02), shp.dtype)
    w["w_down"] = _store(rng.standard_normal((H, F), dtype=f32) * f32(0.02), shp.dtype)
    w["norm1_g"] = _store(1.0 + rng.standard_normal(H, dtype=f32) * f32(0.02), shp.dtype)
    w["norm2_g"] = _store(1.0 + rng.standard_normal(H, dtype=f32) * f32(0.02), shp.dtype)
    if shp.norm == "layer":
        w["norm1_b"] = _store(rng.standard_normal(H, dtype=f32) * f32(0.02), shp.dtype)
        w["norm2_b"] = _store(rng.standard_normal(H, dtype=f32) * f32(0.02), shp.dtype)
    return w


def generate(w: Workload, n_layers: Optional[int] = None, batch: Optional[Batch] = None) -> HostInstance:
    """Host-side instance of a workload (all layers' weights and KV).

    ``n_layers`` overrides the layer count (the 40-layer stack is generated on
    the device instead; see :func:`generate_stack_on_device`).  ``batch``
    replaces the drawn batch (the draws still happen, keeping the order)."""
    shp, spec = w.shape, w.batch
    L = shp.n_layers if n_layers is None else n_layers
    rng = np.random.Generator(np.random.PCG64(w.seed))
    drawn = draw_batch(rng, spec)
    b = drawn if batch is None else batch
    T = b.n_tokens
    x = _store(rng.standard_normal((T, shp.hidden), dtype=np.float32), shp.dtype)
    nh, d, S = shp.n_heads, shp.head_dim, spec.max_seq_len
    kv = np.full((L, spec.n_slots, 2, nh, S, d), np.nan, dtype=np.float32)
    valid = valid_lengths(b, spec.n_slots)
    for s in range(spec.n_slots):
        n = int(valid[s])
        for layer in range(L):
            if n:
                kv[layer, s, :, :, :n, :] = _store(
                    rng.standard_normal((2, nh, n, d), dtype=np.float32), shp.dtype)
    weights = [draw_weights(rng, shp) for _ in range(L)]
    return HostInstance(workload=w, batch=b, x=x, kv=kv, weights=weights)


def make_instance(shape: LayerShape, batch, max_seq_len: int, n_slots: int,
                  seed: int = 0, n_layers: int = 1, x_scale: float = 1.0) -> HostInstance:
    """Instance for an explicitly given batch (a Batch or a MixedBatch; tests
    of edge cases)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    T = batch.n_tokens
    x = _store(rng.standard_normal((T, shape.hidden), dtype=np.float32) * np.float32(x_scale), shape.dtype)
    nh, d = shape.n_heads, shape.head_dim
    kv = np.full((n_layers, n_slots, 2, nh, max_seq_len, d), np.nan, dtype=np.float32)
    valid = valid_lengths(batch, n_slots)
    for s in range(n_slots):
        n = int(valid[s])
        for layer in range(n_layers):
            if n:
                kv[layer, s, :, :, :n, :] = _store(
                    rng.standard_normal((2, nh, n, d), dtype=np.float32), shape.dtype)
    weights = [draw_weights(rng, shape) for _ in range(n_layers)]
    C = batch.n_tokens - batch.n_decodes
    off = 0 if isinstance(batch, MixedBatch) else batch.chunk_offset
    spec = BatchSpec(chunk_len=C, chunk_offset=off, prompt_len=off + C, n_decodes=batch.n_decodes,
                     ctx_lo=0, ctx_hi=0, max_seq_len=max_seq_len, n_slots=n_slots)
    wl = Workload(name="custom", shape=dataclasses.replace(shape, n_layers=n_layers), batch=spec, seed=seed)
    return HostInstance(workload=wl, batch=batch, x=x, kv=kv, weights=weights)
