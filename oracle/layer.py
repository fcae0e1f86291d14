"""Float64 oracle of one decoder layer over a decode-maximal hybrid batch.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Every function names
the passage of the paper it follows; where the paper is silent the reading
taken is stated in the docstring.

Paper structure used throughout:
  * the decoder block is preproj -> attn -> postproj and ffn_ln1 -> ffn_ln2,
    plus "others" (norms, activation, residuals)  [Sec. 2.1, Table 1];
  * preproj is one matmul with a combined [H, 3H] weight  [Sec. 2.2];
  * a token's K and V are cached and every later token of the same request
    attends to them  [Sec. 2.2];
  * a prefill chunk's query q_i sees the keys (and values) of every token
    before it and none after it -- the same mask as the full prefill
    [Sec. 4.2, Figure "attention mask across chunk prefill iterations"];
  * a hybrid batch is one chunk plus decodes; the linear ops run over all
    rows, attention runs per request  [Sec. 4.3].
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np


@dataclass
class OracleBatch:
    """Hybrid batch [Sec. 4.3]: one chunk (slot, offset, length) then decodes.

    Rows 0..chunk_len-1 are the chunk at positions chunk_offset + r; row
    chunk_len + b is decode b at position decode_ctx[b] (the number of its
    tokens already cached, reading: a decode is a chunk of length 1)."""
    prefill_slot: int
    chunk_offset: int
    chunk_len: int
    decode_slots: Sequence[int]
    decode_ctx: Sequence[int]

    @property
    def n_tokens(self) -> int:
        return self.chunk_len + len(self.decode_slots)


@dataclass
class OracleMixedBatch:
    """Batch of several prompt chunks plus decodes (the iteration-level mixed
    batching that Sec. 5.2 compares against; the hybrid batch is the case of
    at most one chunk).  chunks: [(slot, offset, length)]; rows are chunk 0
    in position order, chunk 1, ..., then the decodes."""
    chunks: Sequence[Sequence[int]]
    decode_slots: Sequence[int]
    decode_ctx: Sequence[int]

    @property
    def n_tokens(self) -> int:
        return sum(int(c[2]) for c in self.chunks) + len(self.decode_slots)


@dataclass
class LayerOut:
    y: np.ndarray          # [T, H] layer output
    q: np.ndarray          # [T, nh, d] queries after rotation
    k_new: np.ndarray      # [T, nh, d] keys written to the cache (after rotation)
    v_new: np.ndarray      # [T, nh, d] values written to the cache
    o: np.ndarray          # [T, nh*d] attention output (before postproj)
    hres: np.ndarray       # [T, H] x + postproj(o)
    m: np.ndarray          # [T, F] FFN hidden activation
    slots: np.ndarray      # [T] slot of each row
    positions: np.ndarray  # [T] position of each row


# ----------------------------------------------------------------------------- "others"

def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """Root-mean-square norm of each row, times the gain.

    The paper lists normalisation among the "others" ops [Sec. 2.1]; the RMS
    form, with eps inside the square root, is the LLaMA reading."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(g, dtype=np.float64)


def layer_norm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm of each row (biased variance), times gain plus bias [Sec. 2.1,
    "layer normalization"]; used for the GPT-3 shape."""
    x = np.asarray(x, dtype=np.float64)
    mu = np.mean(x, axis=-1, keepdims=True)
    var = np.mean((x - mu) ** 2, axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * np.asarray(g, np.float64) + np.asarray(b, np.float64)


def silu(z: np.ndarray) -> np.ndarray:
    """z * sigmoid(z), the gate of the SwiGLU FFN (ffn_ln1's activation in
    the LLaMA reading of Sec. 2.1)."""
    z = np.asarray(z, dtype=np.float64)
    return z / (1.0 + np.exp(-z))


def gelu(z: np.ndarray) -> np.ndarray:
    """Exact GELU, z * Phi(z) with Phi the standard normal CDF (GPT-3
    reading of the activation among the "others" ops, Sec. 2.1)."""
    z = np.asarray(z, dtype=np.float64)
    erf = np.vectorize(math.erf, otypes=[np.float64])
    return 0.5 * z * (1.0 + erf(z / math.sqrt(2.0)))


# ----------------------------------------------------------------------------- linear ops

def linear(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """y = x W^T with W stored [out, in] (Table 1's [in, out] weight, kept
    transposed).  The hybrid batch runs each linear op as one matmul over all
    rows [Sec. 4.3]."""
    return np.asarray(x, np.float64) @ np.asarray(w, np.float64).T


# ----------------------------------------------------------------------------- rotary embedding

def rope_rotate(u: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotary position embedding (not in the paper; LLaMA reading).

    u: [..., n, d] with positions pos: [n].  Pairs (i, i + d/2) are rotated by
    angle pos * base^(-2i/d):  (a, b) -> (a cos - b sin, a sin + b cos)."""
    u = np.asarray(u, dtype=np.float64)
    d = u.shape[-1]
    half = d // 2
    i = np.arange(half, dtype=np.float64)
    theta = base ** (-2.0 * i / d)                                   # [half]
    ang = np.asarray(pos, dtype=np.float64)[:, None] * theta[None, :]  # [n, half]
    c, s = np.cos(ang), np.sin(ang)
    shape = (1,) * (u.ndim - 2) + ang.shape
    c, s = c.reshape(shape), s.reshape(shape)
    a, b = u[..., :half], u[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


# ----------------------------------------------------------------------------- attention

def attend(q: np.ndarray, keys: np.ndarray, values: np.ndarray) -> np.ndarray:
    """Softmax attention of one query per head over its request's keys.

    q [nh, d], keys/values [nh, n, d] -> [nh, d].  Scores q.k / sqrt(d)
    (scale: standard reading, the paper is silent); two-pass softmax."""
    q = np.asarray(q, np.float64)
    keys = np.asarray(keys, np.float64)
    values = np.asarray(values, np.float64)
    d = q.shape[-1]
    s = np.einsum("hd,hnd->hn", q, keys) / math.sqrt(d)
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    w = e / np.sum(e, axis=-1, keepdims=True)
    return np.einsum("hn,hnd->hd", w, values)


def token_positions(batch):
    """(slot, position) of every row of the batch: chunk rows at
    offset..offset+C-1 of their slot, then each decode at its context length
    [Sec. 4.2 chunk offsets; Sec. 4.3 row concatenation].  ``batch`` is an
    OracleBatch or an OracleMixedBatch."""
    if isinstance(batch, OracleMixedBatch):
        chunks = [(int(s), int(o), int(n)) for s, o, n in batch.chunks]
    else:
        chunks = [(batch.prefill_slot, batch.chunk_offset, batch.chunk_len)] if batch.chunk_len else []
    slots, pos = [], []
    for s, o, n in chunks:
        slots += [s] * n
        pos += [o + r for r in range(n)]
    slots += [int(s) for s in batch.decode_slots]
    pos += [int(c) for c in batch.decode_ctx]
    return np.asarray(slots, dtype=np.int64), np.asarray(pos, dtype=np.int64)


def chunk_visibility(prompt_len: int, chunk: int) -> List[np.ndarray]:
    """For a prompt split into chunks, the visibility matrix of each
    iteration: rows are the chunk's queries, columns all keys cached so far;
    True where the query may look [Sec. 4.2 and its mask figure]."""
    out = []
    for off in range(0, prompt_len, chunk):
        n = min(chunk, prompt_len - off)
        vis = np.zeros((n, off + n), dtype=bool)
        for r in range(n):
            vis[r, : off + r + 1] = True
        out.append(vis)
    return out


# ----------------------------------------------------------------------------- layer

def _get(w: dict, key: str) -> Optional[np.ndarray]:
    v = w.get(key)
    return None if v is None else np.asarray(v, dtype=np.float64)


def layer_forward(shape, w: dict, kv_layer: np.ndarray, batch: OracleBatch,
                  x: np.ndarray) -> LayerOut:
    """One pre-norm decoder layer over a hybrid batch.

    shape: object with hidden, n_heads, head_dim, ffn, norm ("rms"/"layer"),
      act ("swiglu"/"gelu"), rope (bool), rope_base, eps.
    w: weights of the layer, [out, in] matrices (w_qkv [3 nh d, H], w_o
      [H, nh d], w_up [2F or F, H] with gate rows first, w_down [H, F]) and
      norm gains/biases.
    kv_layer: this layer's cache [n_slots, 2, nh, S, d] (any float dtype);
      it is MODIFIED in place: the new tokens' K and V are written at their
      (slot, position).  Attention itself uses the float64 values of the new
      keys, and never reads a position past the row's own.
    x: [T, H] input rows.

    Steps, in the order of Sec. 2.1 / Table 1:
      1. norm_1; 2. preproj (one matmul over all T rows, Sec. 4.3);
      3. rotate q and k by absolute position; 4. write k, v to the cache
      (Sec. 4.5 "update respective KV pairs in place");
      5. attention of each row over keys 0..position of its own request
      (Sec. 4.2 mask, Sec. 4.3 separate attention);
      6. postproj + residual; 7. norm_2; 8. ffn_ln1 + activation;
      9. ffn_ln2 + residual.
    """
    H, nh, d, F = shape.hidden, shape.n_heads, shape.head_dim, shape.ffn
    x = np.asarray(x, dtype=np.float64)
    T = x.shape[0]
    assert T == batch.n_tokens and x.shape[1] == H
    slots, pos = token_positions(batch)

    def norm(v, g, b):
        if shape.norm == "rms":
            return rms_norm(v, g, shape.eps)
        return layer_norm(v, g, b, shape.eps)

    a = norm(x, _get(w, "norm1_g"), _get(w, "norm1_b"))
    qkv = linear(a, w["w_qkv"])                                   # [T, 3 nh d]
    q = qkv[:, 0:nh * d].reshape(T, nh, d)
    k = qkv[:, nh * d:2 * nh * d].reshape(T, nh, d)
    v = qkv[:, 2 * nh * d:3 * nh * d].reshape(T, nh, d)
    if shape.rope:
        # rotate per head: [nh, T, d] with positions [T]
        q = rope_rotate(q.transpose(1, 0, 2), pos, shape.rope_base).transpose(1, 0, 2)
        k = rope_rotate(k.transpose(1, 0, 2), pos, shape.rope_base).transpose(1, 0, 2)

    # Attention, request by request.  Each request's keys are its cached
    # tokens plus the ones this step adds; a row at position p looks at keys
    # 0..p inclusive (its own key included, as in the full causal prefill).
    o = np.zeros((T, nh * d), dtype=np.float64)
    for s in sorted(set(int(v_) for v_ in slots)):
        rows = [t for t in range(T) if slots[t] == s]
        n_max = max(int(pos[t]) for t in rows) + 1
        blk = np.array(kv_layer[s, :, :, :n_max, :], dtype=np.float64)   # [2, nh, n, d]
        for t in rows:
            blk[0, :, pos[t], :] = k[t]
            blk[1, :, pos[t], :] = v[t]
        for t in rows:
            n = int(pos[t]) + 1
            o[t] = attend(q[t], blk[0, :, :n, :], blk[1, :, :n, :]).reshape(nh * d)

    # In-place cache update at each new token's (slot, position).
    for t in range(T):
        kv_layer[slots[t], 0, :, pos[t], :] = k[t]
        kv_layer[slots[t], 1, :, pos[t], :] = v[t]

    hres = x + linear(o, w["w_o"])
    bn = norm(hres, _get(w, "norm2_g"), _get(w, "norm2_b"))
    up = linear(bn, w["w_up"])
    if shape.act == "swiglu":
        m = silu(up[:, :F]) * up[:, F:2 * F]
    else:
        m = gelu(up)
    y = hres + linear(m, w["w_down"])
    return LayerOut(y=y, q=q, k_new=k, v_new=v, o=o, hres=hres, m=m, slots=slots, positions=pos)


def model_step(shape, weights: List[dict], kv: np.ndarray, batch: OracleBatch,
               x: np.ndarray) -> List[LayerOut]:
    """L layers over the same hybrid batch, each feeding the next; layer l
    uses kv[l] (modified in place).  One iteration of the model [Sec. 4.5]."""
    outs = []
    h = np.asarray(x, dtype=np.float64)
    for layer, w in enumerate(weights):
        out = layer_forward(shape, w, kv[layer], batch, h)
        outs.append(out)
        h = out.y
    return outs
