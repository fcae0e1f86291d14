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
F32, BF16 = 0, 1
NORM_RMS, NORM_LAYER = 0, 1
ACT_SWIGLU, ACT_GELU = 0, 1
LINEAR_PLAIN, LINEAR_RESID, LINEAR_RESID_F32IN, LINEAR_SWIGLU, LINEAR_GELU = 0, 1, 2, 3, 4

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


class sarathi_kv_strides(ct.Structure):
    _fields_ = [(n, ct.c_size_t) for n in ("layer", "slot", "kv", "head", "pos")]


class sarathi_ws_layout(ct.Structure):
    _fields_ = [(n, ct.c_size_t) for n in ("a", "qkv", "o", "hres", "m")] + [("ping", ct.c_size_t * 2),
                                                                             ("total", ct.c_size_t)]


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
    "sarathi_model_step": (ct.c_int, [ct.POINTER(sarathi_model_cfg), ct.POINTER(sarathi_layer_weights),
                                      ct.c_void_p, ct.POINTER(sarathi_hybrid_batch), ct.c_void_p, ct.c_void_p,
                                      ct.c_void_p, ct.c_size_t, ct.c_void_p]),
    "sarathi_profile_begin": (ct.c_int, [ct.c_int]),
    "sarathi_profile_end": (ct.c_int, [ct.POINTER(ct.c_double), ct.POINTER(ct.c_int)]),
    "sarathi_linear_scratch_bytes": (ct.c_size_t, [ct.c_int, ct.c_int]),
    "sarathi_linear": (ct.c_int, [ct.c_int, ct.c_int, ct.c_int, ct.c_int, ct.c_int, ct.c_void_p, ct.c_void_p,
                                  ct.c_void_p, ct.c_void_p, ct.c_void_p, ct.c_size_t, ct.c_void_p]),
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


def sarathi_model_step(cfg, weights: Sequence[sarathi_layer_weights], kv: KV, batch, x_in: int, x_out: int,
                       ws: int, ws_bytes: int, stream: int = 0, check: bool = True) -> int:
    arr = (sarathi_layer_weights * len(weights))(*weights)
    rc = lib().sarathi_model_step(ct.byref(cfg), arr, kv.handle, ct.byref(batch), ct.c_void_p(x_in),
                                  ct.c_void_p(x_out), ct.c_void_p(ws), ws_bytes, ct.c_void_p(stream))
    return _check(rc) if check else rc


N_STAGES = 9
STAGE_NAMES = ["norm_1", "preproj", "rope_kv_append", "chunk_attention", "decode_attention", "postproj", "norm_2",
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
