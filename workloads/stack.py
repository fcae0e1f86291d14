"""On-device generation of a multi-layer stack workload (seeded torch RNG).

The 40-layer LLaMA-13B stack holds 25 GB of weights and, with every slot
sized for 2112 positions, 85 GB of KV cache; drawing that on the host is too
slow, so it is drawn on the device with torch's seeded generator.  Consumers
that need the values on the host (the oracle) copy the exact bytes back.
Like the rest of this package it holds no layer arithmetic: it draws numbers
(N(0,1) for X and cached K/V, 0.02 * N(0,1) for weights, 1 + 0.02 * N(0,1) for
norm gains), rounds them to bf16, and marks empty cache positions with NaN.
The batch (context lengths, slot permutation) is drawn on the host exactly as
in :func:`workloads.generate`.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List

import numpy as np

from . import Batch, Workload, draw_batch, valid_lengths


@dataclass
class DeviceStack:
    workload: Workload
    batch: Batch                 # step-0 batch
    x: "object"                  # torch bf16 [T, H]
    kv: "object"                 # torch bf16 [L, n_slots, 2, nh, S, d]
    weights: List[dict]          # per layer: name -> torch bf16 tensor

    def step_batch(self, step: int) -> Batch:
        """Batch of consecutive step `step`: the chunk advances by its length,
        every decode by one position (the KV grows in place)."""
        b = self.batch
        return Batch(prefill_slot=b.prefill_slot, chunk_offset=b.chunk_offset + step * b.chunk_len,
                     chunk_len=b.chunk_len, decode_slots=b.decode_slots.copy(),
                     decode_ctx=(b.decode_ctx + step).astype(np.int32))


def generate_stack_on_device(w: Workload) -> DeviceStack:
    import torch

    shp, spec = w.shape, w.batch
    rng = np.random.Generator(np.random.PCG64(w.seed))
    batch = draw_batch(rng, spec)
    g = torch.Generator(device="cuda")
    g.manual_seed(w.seed)
    L, H, nh, d, F, S = shp.n_layers, shp.hidden, shp.n_heads, shp.head_dim, shp.ffn, spec.max_seq_len
    bf = torch.bfloat16
    x = torch.empty((batch.n_tokens, H), dtype=bf, device="cuda").normal_(0.0, 1.0, generator=g)
    kv = torch.empty((L, spec.n_slots, 2, nh, S, d), dtype=bf, device="cuda")
    for layer in range(L):
        kv[layer].normal_(0.0, 1.0, generator=g)
    valid = valid_lengths(batch, spec.n_slots)
    for s in range(spec.n_slots):
        kv[:, s, :, :, int(valid[s]):, :] = float("nan")
    weights = []
    for _ in range(L):
        lw = {
            "w_qkv": torch.empty((3 * nh * d, H), dtype=bf, device="cuda").normal_(0.0, 0.02, generator=g),
            "w_o": torch.empty((H, nh * d), dtype=bf, device="cuda").normal_(0.0, 0.02, generator=g),
            "w_up": torch.empty((shp.up_rows, H), dtype=bf, device="cuda").normal_(0.0, 0.02, generator=g),
            "w_down": torch.empty((H, F), dtype=bf, device="cuda").normal_(0.0, 0.02, generator=g),
            "norm1_g": torch.empty(H, dtype=bf, device="cuda").normal_(1.0, 0.02, generator=g),
            "norm2_g": torch.empty(H, dtype=bf, device="cuda").normal_(1.0, 0.02, generator=g),
        }
        if shp.norm == "layer":
            lw["norm1_b"] = torch.empty(H, dtype=bf, device="cuda").normal_(0.0, 0.02, generator=g)
            lw["norm2_b"] = torch.empty(H, dtype=bf, device="cuda").normal_(0.0, 0.02, generator=g)
        weights.append(lw)
    return DeviceStack(workload=w, batch=batch, x=x, kv=kv, weights=weights)


@dataclass
class DeviceLayer:
    """One layer's weights and a KV cache on the device (for timing sweeps)."""
    shape: "object"
    kv: "object"                 # torch [1, n_slots, 2, nh, S, d]
    weights: dict


def generate_layer_on_device(shp, n_slots: int, max_seq_len: int, seed: int = 0) -> DeviceLayer:
    """Weights of one layer plus a KV cache whose every position holds a
    finite N(0,1) value (timing sweeps read prefixes written by nobody)."""
    import torch

    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    dt = torch.bfloat16 if shp.dtype == "bf16" else torch.float32
    H, nh, d, F = shp.hidden, shp.n_heads, shp.head_dim, shp.ffn
    kv = torch.empty((1, n_slots, 2, nh, max_seq_len, d), dtype=dt, device="cuda").normal_(0.0, 1.0, generator=g)
    lw = {
        "w_qkv": torch.empty((3 * nh * d, H), dtype=dt, device="cuda").normal_(0.0, 0.02, generator=g),
        "w_o": torch.empty((H, nh * d), dtype=dt, device="cuda").normal_(0.0, 0.02, generator=g),
        "w_up": torch.empty((shp.up_rows, H), dtype=dt, device="cuda").normal_(0.0, 0.02, generator=g),
        "w_down": torch.empty((H, F), dtype=dt, device="cuda").normal_(0.0, 0.02, generator=g),
        "norm1_g": torch.empty(H, dtype=dt, device="cuda").normal_(1.0, 0.02, generator=g),
        "norm2_g": torch.empty(H, dtype=dt, device="cuda").normal_(1.0, 0.02, generator=g),
    }
    if shp.norm == "layer":
        lw["norm1_b"] = torch.empty(H, dtype=dt, device="cuda").normal_(0.0, 0.02, generator=g)
        lw["norm2_b"] = torch.empty(H, dtype=dt, device="cuda").normal_(0.0, 0.02, generator=g)
    return DeviceLayer(shape=shp, kv=kv, weights=lw)


@dataclass
class DeviceModel:
    """Weights of ``n_layers`` layers and a KV cache on the device (timing)."""
    shape: "object"
    kv: "object"                 # torch [L, n_slots, 2, nh, S, d]
    weights: List[dict]


def generate_model_on_device(shp, n_layers: int, n_slots: int, max_seq_len: int, seed: int = 0) -> DeviceModel:
    """``n_layers`` layers of weights plus a KV cache whose every position
    holds a finite N(0,1) value, drawn with torch's seeded generator (the
    same distributions as :func:`generate_layer_on_device`)."""
    import torch

    layers = [generate_layer_on_device(shp, 1, 1, seed + 1000 * i).weights for i in range(n_layers)]
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    dt = torch.bfloat16 if shp.dtype == "bf16" else torch.float32
    kv = torch.empty((n_layers, n_slots, 2, shp.n_heads, max_seq_len, shp.head_dim), dtype=dt, device="cuda")
    for layer in range(n_layers):
        kv[layer].normal_(0.0, 1.0, generator=g)
    return DeviceModel(shape=shp, kv=kv, weights=layers)
