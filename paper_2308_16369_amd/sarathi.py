"""ctypes binding of libsarathi.so (see include/sarathi.h for the contract).

Argument marshalling only: every step of the layer runs in the library's HIP
kernels.  The names mirror the C entry points.  Device memory is passed as
integer addresses (e.g. ``tensor.data_ptr()``) and streams as hipStream_t
handles (``torch.cuda.current_stream().cuda_stream``); PyTorch is not needed
to use this module.

If the library is missing, the first use raises :class:`SarathiLibraryMissing`
-- there is no other implementation to fall back to.
"""
from __future__ import annotations

import ctypes as ct
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsarathi.so")

OK, EINVAL, ERANGE, ENOSPC, EUNSUPPORTED, EHIP = 0, -1, -2, -3, -4, -5
NOALLOC_SCRATCH_BYTES = 160 << 20   # SARATHI_NOALLOC_SCRATCH_BYTES
F32, BF16 = 0, 1
NORM_RMS, NORM_LAYER = 0, 1
ACT_SWIGLU, ACT_GELU = 0, 1
LINEAR_PLAIN, LINEAR_RESID, LINEAR_RESID_F32IN, LINEAR_SWIGLU, LINEAR_GELU = 0, 1, 2, 3, 4
POLICY_DECODE_MAXIMAL, POLICY_PREFILL_DECODE, POLICY_MIXED = 0, 1, 2

_ERRNAMES = {EINVAL: "EINVAL", ERANGE: "ERANGE", ENOSPC: "ENOSPC", EUNSUPPORTED: "EUNSUPPORTED", EHIP: "EHIP"}


class SarathiLibraryMissing(RuntimeError):
    pass


class SarathiError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_ERRNAMES.get(code, code)}: {msg}")
        self.code = code


class sarathi_model_cfg(ct.Structure):
    _fields_ = [("hidden", ct.c_int), ("n_heads", ct.c_int), ("head_dim", ct.c_int), ("ffn", ct.c_int),
                ("n_layers", ct.c_int), ("norm", ct.c_int), ("act", ct.c_int), ("rope", ct.c_int),
                ("rope_base", ct.c_float), ("eps", ct.c_float), ("dtype", ct.c_int)]


class sarathi_layer_weights(ct.Structure):
    _fields_ = [(n, ct.c_void_p) for n in ("norm1_g", "norm1_b", "w_qkv", "w_o", "norm2_g", "norm2_b",
                                           "w_up", "w_down")]


class sarathi_hybrid_batch(ct.Structure):
    _fields_ = [("prefill_slot", ct.c_int), ("chunk_offset", ct.c_int), ("chunk_len", ct.c_int),
                ("n_decodes", ct.c_int), ("decode_slots", ct.POINTER(ct.c_int)),
                ("decode_ctx_lens", ct.POINTER(ct.c_int))]


class sarathi_mixed_batch(ct.Structure):
    _fields_ = [("n_chunks", ct.c_int), ("chunk_slots", ct.POINTER(ct.c_int)), ("chunk_offsets", ct.POINTER(ct.c_int)),
                ("chunk_lens", ct.POINTER(ct.c_int)), ("n_decodes", ct.c_int), ("decode_slots", ct.POINTER(ct.c_int)),
                ("decode_ctx_lens", ct.POINTER(ct.c_int))]


class sarathi_kv_strides(ct.Structure):
    _fields_ = [(n, ct.c_size_t) for n in ("layer", "slot", "kv", "head", "pos")]


class sarathi_ws_layout(ct.Structure):
    _fields_ = [(n, ct.c_size_t) for n in ("a", "qkv", "o", "hres", "m")] + [("ping", ct.c_size_t * 2),
                                                                             ("total", ct.c_size_t)]


class sarathi_attn_plan(ct.Structure):
    _fields_ = [("chunk_items", ct.c_int), ("decode_items", ct.c_int), ("partial_rows_written", ct.c_long),
                ("partial_rows_read", ct.c_long), ("combine_rows", ct.c_int)]


class sarathi_sched_cfg(ct.Structure):
    _fields_ = [(n, ct.c_int) for n in ("policy", "max_batch", "chunk", "max_chunks", "max_tokens", "n_slots",
                                        "max_seq_len")]


class sarathi_sched_step(ct.Structure):
    _fields_ = [("n_tokens", ct.c_int), ("n_chunks", ct.c_int)] + \
        [(n, ct.POINTER(ct.c_int)) for n in ("chunk_request", "chunk_slot", "chunk_offset", "chunk_len")] + \
        [("n_decodes", ct.c_int)] + \
        [(n, ct.POINTER(ct.c_int)) for n in ("decode_request", "decode_slot", "decode_ctx")]


class sarathi_sched_stats(ct.Structure):
    _fields_ = [(n, ct.c_longlong) for n in ("iterations", "prefill_tokens", "decode_tokens", "hybrid_iterations",
                                             "prefill_only_iterations", "decode_only_iterations")] + \
        [(n, ct.c_int) for n in ("submitted", "admitted", "finished", "resident")]


EXPORTS = {
    "sarathi_version": (ct.c_int, []),
    "sarathi_last_error": (ct.c_char_p, []),
    "sarathi_kv_bytes": (ct.c_size_t, [ct.POINTER(sarathi_model_cfg), ct.c_int, ct.c_int]),
    "sarathi_kv_alloc": (ct.c_int, [ct.POINTER(sarathi_model_cfg), ct.c_int, ct.c_int, ct.c_void_p, ct.c_size_t,
                                    ct.POINTER(ct.c_void_p)]),
    "sarathi_kv_free": (None, [ct.c_void_p]),
    "sarathi_kv_get_strides": (ct.c_int, [ct.c_void_p, ct.POINTER(sarathi_kv_strides)]),
    "sarathi_workspace_bytes": (ct.c_size_t, [ct.POINTER(sarathi_model_cfg), ct.c_int, ct.c_int, ct.c_int]),
    "sarathi_workspace_layout": (ct.c_int, [ct.POINTER(sarathi_model_cfg), ct.c_int, ct.c_int, ct.c_int,
                                            ct.POINTER(sarathi_ws_layout)]),
    "sarathi_hybrid_layer_forward": (ct.c_int, [ct.POINTER(sarathi_model_cfg), ct.POINTER(sarathi_layer_weights),
                                                ct.c_void_p, ct.c_int, ct.POINTER(sarathi_hybrid_batch),
                                                ct.c_void_p, ct.c_void_p, ct.c_void_p, ct.c_size_t, ct.c_void_p]),
    "sarathi_hybrid_layer_forward_noalloc": (ct.c_int, [ct.POINTER(sarathi_model_cfg),
                                                        ct.POINTER(sarathi_layer_weights), ct.c_void_p, ct.c_int,
                                                        ct.POINTER(sarathi_hybrid_batch), ct.c_void_p, ct.c_void_p,
                                                        ct.c_void_p]),
    "sarathi_model_step": (ct.c_int, [ct.POINTER(sarathi_model_cfg), ct.POINTER(sarathi_layer_weights),
                                      ct.c_void_p, ct.POINTER(sarathi_hybrid_batch), ct.c_void_p, ct.c_void_p,
                                      ct.c_void_p, ct.c_size_t, ct.c_void_p]),
    "sarathi_mixed_workspace_bytes": (ct.c_size_t, [ct.POINTER(sarathi_model_cfg), ct.c_int, ct.c_int, ct.c_int]),
    "sarathi_mixed_workspace_layout": (ct.c_int, [ct.POINTER(sarathi_model_cfg), ct.c_int, ct.c_int, ct.c_int,
                                                  ct.POINTER(sarathi_ws_layout)]),
    "sarathi_mixed_layer_forward": (ct.c_int, [ct.POINTER(sarathi_model_cfg), ct.POINTER(sarathi_layer_weights),
                                               ct.c_void_p, ct.c_int, ct.POINTER(sarathi_mixed_batch),
                                               ct.c_void_p, ct.c_void_p, ct.c_void_p, ct.c_size_t, ct.c_void_p]),
    "sarathi_mixed_model_step": (ct.c_int, [ct.POINTER(sarathi_model_cfg), ct.POINTER(sarathi_layer_weights),
                                            ct.c_void_p, ct.POINTER(sarathi_mixed_batch), ct.c_void_p, ct.c_void_p,
                                            ct.c_void_p, ct.c_size_t, ct.c_void_p]),
    "sarathi_profile_begin": (ct.c_int, [ct.c_int]),
    "sarathi_profile_end": (ct.c_int, [ct.POINTER(ct.c_double), ct.POINTER(ct.c_int)]),
    "sarathi_linear_scratch_bytes": (ct.c_size_t, [ct.c_int, ct.c_int]),
    "sarathi_linear": (ct.c_int, [ct.c_int, ct.c_int, ct.c_int, ct.c_int, ct.c_int, ct.c_void_p, ct.c_void_p,
                                  ct.c_void_p, ct.c_void_p, ct.c_void_p, ct.c_size_t, ct.c_void_p]),
    "sarathi_attention_plan": (ct.c_int, [ct.POINTER(sarathi_model_cfg), ct.POINTER(sarathi_hybrid_batch),
                                          ct.POINTER(sarathi_attn_plan)]),
    "sarathi_linear_plan": (ct.c_int, [ct.c_int, ct.c_int, ct.c_int, ct.c_int, ct.c_int, ct.c_size_t,
                                       ct.POINTER(ct.c_int), ct.POINTER(ct.c_int), ct.POINTER(ct.c_int)]),
    "sarathi_layer_split_scratch_bytes": (ct.c_size_t, [ct.POINTER(sarathi_model_cfg), ct.c_int]),
    "sarathi_linear_tile_count": (ct.c_int, []),
    "sarathi_linear_tile_shape": (ct.c_int, [ct.c_int, ct.POINTER(ct.c_int), ct.POINTER(ct.c_int)]),
    "sarathi_linear_tiled": (ct.c_int, [ct.c_int, ct.c_int, ct.c_int, ct.c_int, ct.c_void_p, ct.c_void_p,
                                        ct.c_void_p, ct.c_void_p, ct.c_void_p, ct.c_size_t, ct.c_int, ct.c_int,
                                        ct.c_void_p]),
    "sarathi_sched_create": (ct.c_int, [ct.POINTER(sarathi_sched_cfg), ct.POINTER(ct.c_void_p)]),
    "sarathi_sched_destroy": (None, [ct.c_void_p]),
    "sarathi_sched_submit": (ct.c_int, [ct.c_void_p, ct.c_int, ct.c_int, ct.POINTER(ct.c_int)]),
    "sarathi_sched_next": (ct.c_int, [ct.c_void_p, ct.POINTER(sarathi_sched_step)]),
    "sarathi_sched_commit": (ct.c_int, [ct.c_void_p]),
    "sarathi_sched_get_stats": (ct.c_int, [ct.c_void_p, ct.POINTER(sarathi_sched_stats)]),
}

_lib: Optional[ct.CDLL] = None


def lib() -> ct.CDLL:
    """Load libsarathi.so once; raise if it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise SarathiLibraryMissing(
                f"{LIB_PATH} not found: build it with `python -m paper_2308_16369_amd.build`")
        L = ct.CDLL(LIB_PATH)
        for name, (res, args) in EXPORTS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(rc: int) -> int:
    if rc != OK:
        raise SarathiError(rc, sarathi_last_error())
    return rc


# ---------------------------------------------------------------------------- thin wrappers

def sarathi_version() -> int:
    return lib().sarathi_version()


def sarathi_last_error() -> str:
    return (lib().sarathi_last_error() or b"").decode()


def make_cfg(hidden, n_heads, head_dim, ffn, n_layers=1, norm=NORM_RMS, act=ACT_SWIGLU, rope=1,
             rope_base=10000.0, eps=1e-6, dtype=BF16) -> sarathi_model_cfg:
    return sarathi_model_cfg(hidden, n_heads, head_dim, ffn, n_layers, norm, act, rope, rope_base, eps, dtype)


def sarathi_kv_bytes(cfg: sarathi_model_cfg, n_slots: int, max_seq_len: int) -> int:
    return lib().sarathi_kv_bytes(ct.byref(cfg), n_slots, max_seq_len)


class KV:
    """Host handle of a KV cache bound to caller-owned device memory."""

    def __init__(self, cfg: sarathi_model_cfg, n_slots: int, max_seq_len: int, dev_ptr: int, dev_bytes: int):
        h = ct.c_void_p()
        _check(lib().sarathi_kv_alloc(ct.byref(cfg), n_slots, max_seq_len, ct.c_void_p(dev_ptr), dev_bytes,
                                      ct.byref(h)))
        self.handle = h
        self.cfg = cfg
        self.n_slots, self.max_seq_len = n_slots, max_seq_len

    def strides(self) -> sarathi_kv_strides:
        st = sarathi_kv_strides()
        _check(lib().sarathi_kv_get_strides(self.handle, ct.byref(st)))
        return st

    def free(self):
        if self.handle:
            lib().sarathi_kv_free(self.handle)
            self.handle = ct.c_void_p()

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def sarathi_kv_alloc(cfg, n_slots, max_seq_len, dev_ptr, dev_bytes) -> KV:
    return KV(cfg, n_slots, max_seq_len, dev_ptr, dev_bytes)


def sarathi_workspace_bytes(cfg, max_tokens, max_decodes, max_seq_len) -> int:
    return lib().sarathi_workspace_bytes(ct.byref(cfg), max_tokens, max_decodes, max_seq_len)


def sarathi_workspace_layout(cfg, n_tokens, n_decodes, max_seq_len) -> sarathi_ws_layout:
    out = sarathi_ws_layout()
    _check(lib().sarathi_workspace_layout(ct.byref(cfg), n_tokens, n_decodes, max_seq_len, ct.byref(out)))
    return out


def make_batch(prefill_slot: int, chunk_offset: int, chunk_len: int, decode_slots: Sequence[int],
               decode_ctx: Sequence[int]):
    """Build the host batch struct; returns (struct, keepalive arrays)."""
    n = len(decode_slots)
    slots = (ct.c_int * max(n, 1))(*[int(s) for s in decode_slots])
    ctx = (ct.c_int * max(n, 1))(*[int(c) for c in decode_ctx])
    b = sarathi_hybrid_batch(int(prefill_slot), int(chunk_offset), int(chunk_len), n,
                             ct.cast(slots, ct.POINTER(ct.c_int)), ct.cast(ctx, ct.POINTER(ct.c_int)))
    return b, (slots, ctx)


def make_weights(ptrs: dict) -> sarathi_layer_weights:
    return sarathi_layer_weights(**{k: ct.c_void_p(int(ptrs[k])) if ptrs.get(k) else None
                                    for k, _ in sarathi_layer_weights._fields_})


def sarathi_hybrid_layer_forward(cfg, weights: sarathi_layer_weights, kv: KV, layer: int, batch, x_in: int,
                                 x_out: int, ws: int, ws_bytes: int, stream: int = 0, check: bool = True) -> int:
    rc = lib().sarathi_hybrid_layer_forward(ct.byref(cfg), ct.byref(weights), kv.handle, layer, ct.byref(batch),
                                            ct.c_void_p(x_in), ct.c_void_p(x_out), ct.c_void_p(ws), ws_bytes,
                                            ct.c_void_p(stream))
    return _check(rc) if check else rc


def sarathi_hybrid_layer_forward_noalloc(cfg, weights: sarathi_layer_weights, kv: KV, layer: int, batch, x_in: int,
                                         x_out: int, stream: int = 0, check: bool = True) -> int:
    rc = lib().sarathi_hybrid_layer_forward_noalloc(ct.byref(cfg), ct.byref(weights), kv.handle, layer,
                                                    ct.byref(batch), ct.c_void_p(x_in), ct.c_void_p(x_out),
                                                    ct.c_void_p(stream))
    return _check(rc) if check else rc


def sarathi_model_step(cfg, weights: Sequence[sarathi_layer_weights], kv: KV, batch, x_in: int, x_out: int,
                       ws: int, ws_bytes: int, stream: int = 0, check: bool = True) -> int:
    arr = (sarathi_layer_weights * len(weights))(*weights)
    rc = lib().sarathi_model_step(ct.byref(cfg), arr, kv.handle, ct.byref(batch), ct.c_void_p(x_in),
                                  ct.c_void_p(x_out), ct.c_void_p(ws), ws_bytes, ct.c_void_p(stream))
    return _check(rc) if check else rc


def sarathi_mixed_workspace_bytes(cfg, max_tokens, max_chunks, max_seq_len) -> int:
    return lib().sarathi_mixed_workspace_bytes(ct.byref(cfg), max_tokens, max_chunks, max_seq_len)


def sarathi_mixed_workspace_layout(cfg, n_tokens, n_chunks, max_seq_len) -> sarathi_ws_layout:
    out = sarathi_ws_layout()
    _check(lib().sarathi_mixed_workspace_layout(ct.byref(cfg), n_tokens, n_chunks, max_seq_len, ct.byref(out)))
    return out


def make_mixed_batch(chunks: Sequence[Sequence[int]], decode_slots: Sequence[int], decode_ctx: Sequence[int]):
    """Build a sarathi_mixed_batch from chunks [(slot, offset, len)] and
    decodes; returns (struct, keepalive arrays)."""
    k, n = len(chunks), len(decode_slots)
    arr = lambda vals, m: (ct.c_int * max(m, 1))(*[int(v) for v in vals])
    cs, co, cl = arr([c[0] for c in chunks], k), arr([c[1] for c in chunks], k), arr([c[2] for c in chunks], k)
    ds, dc = arr(decode_slots, n), arr(decode_ctx, n)
    P = lambda a: ct.cast(a, ct.POINTER(ct.c_int))
    b = sarathi_mixed_batch(k, P(cs), P(co), P(cl), n, P(ds), P(dc))
    return b, (cs, co, cl, ds, dc)


def sarathi_mixed_layer_forward(cfg, weights: sarathi_layer_weights, kv: KV, layer: int, batch, x_in: int,
                                x_out: int, ws: int, ws_bytes: int, stream: int = 0, check: bool = True) -> int:
    rc = lib().sarathi_mixed_layer_forward(ct.byref(cfg), ct.byref(weights), kv.handle, layer, ct.byref(batch),
                                           ct.c_void_p(x_in), ct.c_void_p(x_out), ct.c_void_p(ws), ws_bytes,
                                           ct.c_void_p(stream))
    return _check(rc) if check else rc


def sarathi_mixed_model_step(cfg, weights: Sequence[sarathi_layer_weights], kv: KV, batch, x_in: int, x_out: int,
                             ws: int, ws_bytes: int, stream: int = 0, check: bool = True) -> int:
    arr = (sarathi_layer_weights * len(weights))(*weights)
    rc = lib().sarathi_mixed_model_step(ct.byref(cfg), arr, kv.handle, ct.byref(batch), ct.c_void_p(x_in),
                                        ct.c_void_p(x_out), ct.c_void_p(ws), ws_bytes, ct.c_void_p(stream))
    return _check(rc) if check else rc


N_STAGES = 10
STAGE_NAMES = ["norm_1", "preproj", "rope_kv_append", "chunk_attention", "decode_attention", "attention_combine",
               "postproj", "norm_2",
               "ffn_ln1", "ffn_ln2"]


def sarathi_profile_begin(max_calls: int) -> int:
    return _check(lib().sarathi_profile_begin(max_calls))


def sarathi_profile_end():
    """Returns ({stage name: summed ms}, number of recorded layer calls)."""
    ms = (ct.c_double * N_STAGES)()
    n = ct.c_int()
    _check(lib().sarathi_profile_end(ms, ct.byref(n)))
    return dict(zip(STAGE_NAMES, list(ms))), n.value


def sarathi_linear_scratch_bytes(M: int, N: int) -> int:
    return lib().sarathi_linear_scratch_bytes(M, N)


def sarathi_linear(dtype, kind, M, N, K, x: int, w: int, resid: int, out: int, scratch: int = 0,
                   scratch_bytes: int = 0, stream: int = 0, check: bool = True) -> int:
    rc = lib().sarathi_linear(dtype, kind, M, N, K, ct.c_void_p(x), ct.c_void_p(w), ct.c_void_p(resid or None),
                              ct.c_void_p(out), ct.c_void_p(scratch or None), scratch_bytes, ct.c_void_p(stream))
    return _check(rc) if check else rc


def sarathi_attention_plan(cfg: sarathi_model_cfg, batch) -> dict:
    """Attention work items and key-split partial rows of a layer call."""
    out = sarathi_attn_plan()
    _check(lib().sarathi_attention_plan(ct.byref(cfg), ct.byref(batch), ct.byref(out)))
    return {k: getattr(out, k) for k, _ in sarathi_attn_plan._fields_}


def sarathi_linear_plan(dtype, kind, M, N, K, scratch_bytes: int = 0):
    """(bm, bn, n_split) that sarathi_linear would run the op with."""
    bm, bn, ns = ct.c_int(), ct.c_int(), ct.c_int()
    _check(lib().sarathi_linear_plan(dtype, kind, M, N, K, scratch_bytes, ct.byref(bm), ct.byref(bn), ct.byref(ns)))
    return bm.value, bn.value, ns.value


def sarathi_layer_split_scratch_bytes(cfg: sarathi_model_cfg, n_tokens: int) -> int:
    return int(lib().sarathi_layer_split_scratch_bytes(ct.byref(cfg), n_tokens))


def sarathi_linear_tile_count() -> int:
    return lib().sarathi_linear_tile_count()


def sarathi_linear_tile_shape(tile: int):
    bm, bn = ct.c_int(), ct.c_int()
    _check(lib().sarathi_linear_tile_shape(tile, ct.byref(bm), ct.byref(bn)))
    return bm.value, bn.value


def sarathi_linear_tiled(kind, M, N, K, x: int, w: int, resid: int, out: int, scratch: int, scratch_bytes: int,
                         tile: int, n_split: int, stream: int = 0, check: bool = True) -> int:
    rc = lib().sarathi_linear_tiled(kind, M, N, K, ct.c_void_p(x), ct.c_void_p(w), ct.c_void_p(resid or None),
                                    ct.c_void_p(out), ct.c_void_p(scratch or None), scratch_bytes, tile, n_split,
                                    ct.c_void_p(stream))
    return _check(rc) if check else rc


# ---------------------------------------------------------------------------- scheduler

class Step:
    """One iteration described by the scheduler (copied out of its arrays)."""

    def __init__(self, st: sarathi_sched_step):
        def arr(p, n):
            return [p[i] for i in range(n)]
        self.n_tokens = st.n_tokens
        self.chunk_request = arr(st.chunk_request, st.n_chunks)
        self.chunk_slot = arr(st.chunk_slot, st.n_chunks)
        self.chunk_offset = arr(st.chunk_offset, st.n_chunks)
        self.chunk_len = arr(st.chunk_len, st.n_chunks)
        self.decode_request = arr(st.decode_request, st.n_decodes)
        self.decode_slot = arr(st.decode_slot, st.n_decodes)
        self.decode_ctx = arr(st.decode_ctx, st.n_decodes)

    @property
    def n_chunks(self) -> int:
        return len(self.chunk_len)

    @property
    def n_decodes(self) -> int:
        return len(self.decode_ctx)

    def mixed_batch(self):
        """(sarathi_mixed_batch, keepalive) for any iteration."""
        return make_mixed_batch(list(zip(self.chunk_slot, self.chunk_offset, self.chunk_len)), self.decode_slot,
                                self.decode_ctx)

    def hybrid_batch(self):
        """(sarathi_hybrid_batch, keepalive) for an iteration of at most one chunk."""
        if self.n_chunks > 1:
            raise ValueError("an iteration with several chunks needs the mixed-batch entry points")
        if self.n_chunks == 1:
            return make_batch(self.chunk_slot[0], self.chunk_offset[0], self.chunk_len[0], self.decode_slot,
                              self.decode_ctx)
        return make_batch(-1, 0, 0, self.decode_slot, self.decode_ctx)


class Scheduler:
    """Owner of one sarathi_sched (include/sarathi_sched.h)."""

    def __init__(self, policy: int, max_batch: int, n_slots: int, max_seq_len: int, chunk: int = 0,
                 max_chunks: int = 0, max_tokens: int = 0):
        cfg = sarathi_sched_cfg(policy, max_batch, chunk, max_chunks, max_tokens, n_slots, max_seq_len)
        h = ct.c_void_p()
        _check(lib().sarathi_sched_create(ct.byref(cfg), ct.byref(h)))
        self._h = h

    def close(self):
        if self._h:
            lib().sarathi_sched_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def submit(self, prompt_len: int, decode_len: int) -> int:
        rid = ct.c_int()
        _check(lib().sarathi_sched_submit(self._h, prompt_len, decode_len, ct.byref(rid)))
        return rid.value

    def next(self) -> Step:
        st = sarathi_sched_step()
        _check(lib().sarathi_sched_next(self._h, ct.byref(st)))
        return Step(st)

    def commit(self):
        _check(lib().sarathi_sched_commit(self._h))

    def stats(self) -> dict:
        st = sarathi_sched_stats()
        _check(lib().sarathi_sched_get_stats(self._h, ct.byref(st)))
        return {n: getattr(st, n) for n, _ in sarathi_sched_stats._fields_}
