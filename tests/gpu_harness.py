"""Helpers of the GPU tests: upload a host instance, run the library through
its C-ABI, read results back, and compare with the oracle.

PyTorch is used only for device memory, streams and copies."""
from __future__ import annotations

import sys
import time
from dataclasses import dataclass
from typing import List, Optional

import numpy as np
import torch

import oracle
import workloads as wl
from paper_2308_16369_amd import sarathi as S

TOL = {"f32": 1e-4, "bf16": 2e-2}


def log(msg: str):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


def cfg_of(shape: wl.LayerShape, n_layers: Optional[int] = None) -> S.sarathi_model_cfg:
    return S.make_cfg(hidden=shape.hidden, n_heads=shape.n_heads, head_dim=shape.head_dim, ffn=shape.ffn,
                      n_layers=shape.n_layers if n_layers is None else n_layers,
                      norm=S.NORM_RMS if shape.norm == "rms" else S.NORM_LAYER,
                      act=S.ACT_SWIGLU if shape.act == "swiglu" else S.ACT_GELU,
                      rope=1 if shape.rope else 0, rope_base=shape.rope_base, eps=shape.eps,
                      dtype=S.BF16 if shape.dtype == "bf16" else S.F32)


def to_dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(wl.bf16_bits(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def from_dev(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> fp32 numpy (exact for bf16)."""
    if t.dtype == torch.bfloat16:
        return wl.bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16))
    return t.float().cpu().numpy()


def bits_of(t: torch.Tensor) -> np.ndarray:
    """Raw bit patterns (uint16 for bf16, uint32 for fp32)."""
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.view(torch.int32).cpu().numpy().view(np.uint32)


def rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    ref = np.asarray(ref, np.float64)
    got = np.asarray(got, np.float64)
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / den) if den > 0 else float(np.max(np.abs(got)))


def half_ulp_bf16(v: np.ndarray) -> np.ndarray:
    """Half a bf16 ulp at |v| (8 significant bits)."""
    a = np.maximum(np.abs(np.asarray(v, np.float64)), np.finfo(np.float32).tiny)
    return np.ldexp(1.0, (np.floor(np.log2(a)) - 8).astype(np.int64))


def delta_err(got: np.ndarray, ref_total: np.ndarray, ref_delta: np.ndarray, out_dtype: str) -> float:
    """Error of an output y = base + delta, measured on the delta's scale
    after allowing for the rounding of y itself to its storage type:
    max(|got - ref| - half_ulp(y)) / max|delta|  (bf16 storage), or plain
    max|got - ref| / max|delta| for fp32 storage."""
    got = np.asarray(got, np.float64)
    ref_total = np.asarray(ref_total, np.float64)
    diff = np.abs(got - ref_total)
    if out_dtype == "bf16":
        diff = np.maximum(diff - half_ulp_bf16(np.maximum(np.abs(got), np.abs(ref_total))), 0.0)
    den = np.max(np.abs(ref_delta))
    return float(np.max(diff) / den) if den > 0 else float(np.max(diff))


WKEYS = ("norm1_g", "norm1_b", "w_qkv", "w_o", "norm2_g", "norm2_b", "w_up", "w_down")


class DeviceModel:
    """Weights, KV and workspace of an instance on the GPU."""

    def __init__(self, inst: wl.HostInstance, max_tokens: Optional[int] = None, max_chunks: int = 1):
        self.inst = inst
        shp = inst.shape
        self.dtype = shp.dtype
        self.L = inst.kv.shape[0]
        self.cfg = cfg_of(shp, self.L)
        self.tdtype = torch.bfloat16 if shp.dtype == "bf16" else torch.float32
        self.w_dev = [{k: to_dev(w[k], shp.dtype) for k in WKEYS if k in w} for w in inst.weights]
        self.w_abi = [S.make_weights({k: t.data_ptr() for k, t in wd.items()}) for wd in self.w_dev]
        spec = inst.workload.batch
        self.S = inst.kv.shape[4]
        self.n_slots = inst.kv.shape[1]
        self.kv_dev = to_dev(inst.kv, shp.dtype)
        self.kv = S.sarathi_kv_alloc(self.cfg, self.n_slots, self.S, self.kv_dev.data_ptr(),
                                     self.kv_dev.numel() * self.kv_dev.element_size())
        T = max_tokens or inst.batch.n_tokens
        self.ws_bytes = S.sarathi_mixed_workspace_bytes(self.cfg, T, max_chunks, self.S)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device="cuda")

    def batch_abi(self, b: wl.Batch):
        return S.make_batch(b.prefill_slot, b.chunk_offset, b.chunk_len, list(b.decode_slots), list(b.decode_ctx))

    def layer(self, layer: int, b: wl.Batch, x: torch.Tensor) -> torch.Tensor:
        out = torch.empty_like(x)
        bb, keep = self.batch_abi(b)
        S.sarathi_hybrid_layer_forward(self.cfg, self.w_abi[layer], self.kv, layer, bb, x.data_ptr(),
                                       out.data_ptr(), self.ws.data_ptr(), self.ws_bytes,
                                       torch.cuda.current_stream().cuda_stream)
        return out

    def mixed_layer(self, layer: int, b: wl.MixedBatch, x: torch.Tensor) -> torch.Tensor:
        out = torch.empty_like(x)
        mb, keep = S.make_mixed_batch(b.chunks, list(b.decode_slots), list(b.decode_ctx))
        S.sarathi_mixed_layer_forward(self.cfg, self.w_abi[layer], self.kv, layer, mb, x.data_ptr(), out.data_ptr(),
                                      self.ws.data_ptr(), self.ws_bytes, torch.cuda.current_stream().cuda_stream)
        return out

    def mixed_step(self, b: wl.MixedBatch, x: torch.Tensor) -> torch.Tensor:
        out = torch.empty_like(x)
        mb, keep = S.make_mixed_batch(b.chunks, list(b.decode_slots), list(b.decode_ctx))
        S.sarathi_mixed_model_step(self.cfg, self.w_abi, self.kv, mb, x.data_ptr(), out.data_ptr(),
                                   self.ws.data_ptr(), self.ws_bytes, torch.cuda.current_stream().cuda_stream)
        return out

    def step(self, b: wl.Batch, x: torch.Tensor) -> torch.Tensor:
        out = torch.empty_like(x)
        bb, keep = self.batch_abi(b)
        S.sarathi_model_step(self.cfg, self.w_abi, self.kv, bb, x.data_ptr(), out.data_ptr(), self.ws.data_ptr(),
                             self.ws_bytes, torch.cuda.current_stream().cuda_stream)
        return out

    def intermediates(self, b: wl.Batch) -> dict:
        """Views of the workspace intermediates of the last call."""
        T = b.n_tokens
        lay = S.sarathi_workspace_layout(self.cfg, T, b.n_decodes, self.S)
        shp = self.inst.shape
        QD = shp.n_heads * shp.head_dim
        es = 2 if self.dtype == "bf16" else 4

        def view(off, n, dt):
            nbytes = n * (2 if dt == torch.bfloat16 else 4)
            return self.ws[off:off + nbytes].view(dt)

        return {
            "qkv": view(lay.qkv, T * 3 * QD, self.tdtype).view(T, 3 * QD),
            "o": view(lay.o, T * QD, self.tdtype).view(T, QD),
            "hres": view(lay.hres, T * shp.hidden, torch.float32).view(T, shp.hidden),
            "m": view(lay.m, T * shp.ffn, self.tdtype).view(T, shp.ffn),
        }


def oracle_batch(b):
    if isinstance(b, wl.MixedBatch):
        return oracle.OracleMixedBatch(chunks=[tuple(int(v) for v in c) for c in b.chunks],
                                       decode_slots=[int(s) for s in b.decode_slots],
                                       decode_ctx=[int(c) for c in b.decode_ctx])
    return oracle.OracleBatch(prefill_slot=b.prefill_slot, chunk_offset=b.chunk_offset, chunk_len=b.chunk_len,
                              decode_slots=[int(s) for s in b.decode_slots],
                              decode_ctx=[int(c) for c in b.decode_ctx])


@dataclass
class Check:
    name: str
    err: float
    tol: float

    @property
    def ok(self) -> bool:
        return self.err <= self.tol


def compare_layer(dm: DeviceModel, layer: int, b: wl.Batch, x_host: np.ndarray, y_dev: torch.Tensor,
                  kv_before_bits: np.ndarray, kv_host_layer: np.ndarray, ref: oracle.LayerOut,
                  check_intermediates: bool = True) -> List[Check]:
    """Compare one layer call with the oracle: outputs and intermediates to
    the tolerance, K/V written at exactly the oracle's (slot, position) and
    every other KV element bit-identical to its value before the call."""
    tol = TOL[dm.dtype]
    shp = dm.inst.shape
    nh, hd = shp.n_heads, shp.head_dim
    checks = []
    y = from_dev(y_dev)
    checks.append(Check("y", rel_err(y, ref.y), tol))
    checks.append(Check("y - hres (beyond y rounding)", delta_err(y, ref.y, ref.y - ref.hres, dm.dtype), tol))
    if check_intermediates:
        it = dm.intermediates(b)
        o = from_dev(it["o"])
        hres = from_dev(it["hres"])
        q = from_dev(it["qkv"])[:, :nh * hd].reshape(-1, nh, hd)
        checks.append(Check("q", rel_err(q, ref.q), tol))
        checks.append(Check("o", rel_err(o, ref.o), tol))
        checks.append(Check("hres - x", rel_err(hres.astype(np.float64) - x_host, ref.hres - x_host), tol))
        checks.append(Check("m (ffn_ln1 activation)", rel_err(from_dev(it["m"]), ref.m), tol))
    # KV: written values
    kv_after = bits_of(dm.kv_dev)
    kv_after_f = wl.bits_to_f32(kv_after) if dm.dtype == "bf16" else kv_after.view(np.float32)
    written = np.zeros(kv_after.shape, dtype=bool)
    kn, vn = [], []
    for t, (s, p) in enumerate(zip(ref.slots, ref.positions)):
        written[layer, s, :, :, p, :] = True
        kn.append(kv_after_f[layer, s, 0, :, p, :])
        vn.append(kv_after_f[layer, s, 1, :, p, :])
    checks.append(Check("k_new", rel_err(np.stack(kn), ref.k_new), tol))
    checks.append(Check("v_new", rel_err(np.stack(vn), ref.v_new), tol))
    untouched_same = np.array_equal(kv_after[~written], kv_before_bits[~written])
    checks.append(Check("kv untouched bit-identical", 0.0 if untouched_same else 1.0, 0.0))
    return checks


def assert_checks(checks: List[Check], label: str):
    for c in checks:
        log(f"  {label}: {c.name:28s} err {c.err:.3e}  tol {c.tol:.0e}  {'ok' if c.ok else 'FAIL'}")
    bad = [c for c in checks if not c.ok]
    assert not bad, f"{label}: " + ", ".join(f"{c.name} {c.err:.3e} > {c.tol:.0e}" for c in bad)
