#!/usr/bin/env python3
"""Benchmark of the decode-maximal hybrid-batch decoder layer on one MI355X.

A step is one pass of the whole hot path -- one decoder layer over one
hybrid batch (norm_1, preproj, rotary embedding + KV append, chunk and
decode attention, postproj, norm_2, ffn_ln1, ffn_ln2), through the C-ABI --
over synthetic, seeded inputs already resident in HBM.  Default workload:
a LLaMA-13B-shaped layer, chunk 256 at offset 512 + 64 decodes with context
uniform in [256, 1024] (T = 320 rows), bf16.

Prints ONE JSON line: hybrid tokens/s (value), the decode accounting of the
paper (Sec. 5.1.1) from prefill-only and decode-only runs of the same rows,
per-stage times from HIP events recorded on the launch stream inside the
timed region, the roofline of the dominant kernel and the oracle timed on
the host cores (cpu_baseline).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBPS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama13b-layer-bf16-c256-b64")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-compare", action="store_true", help="skip the prefill-only / decode-only runs")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB elementwise copy kernel (for HBM counter scaling)")
    ap.add_argument("--no-stack", action="store_true",
                    help="skip the 40-layer model-step measurement (the 'stack' object)")
    ap.add_argument("--stack-steps", type=int, default=5)
    ap.add_argument("--stack-only", action="store_true",
                    help="measure only the 40-layer model step and print its object (for kernel traces of it)")
    return ap.parse_args()


def bench_stack(steps: int, warmup: int, cpu_baseline: bool = True):
    """Model step of the 40-layer LLaMA-13B-shaped stack (chunk 256 + 48
    decodes of context U[512, 2048], KV for 49 slots x 2112 positions):
    time per step, per layer, and the decode accounting of Sec. 5.1.1 against
    prefill-only and decode-only steps of the same rows."""
    import numpy as np
    import torch

    import workloads as wl
    from workloads.stack import generate_stack_on_device
    from paper_2308_16369_amd import sarathi as S
    from paper_2308_16369_amd import accounting

    w = wl.LLAMA13B_STACK
    shp = w.shape
    st = generate_stack_on_device(w)
    L = shp.n_layers
    cfg = S.make_cfg(hidden=shp.hidden, n_heads=shp.n_heads, head_dim=shp.head_dim, ffn=shp.ffn, n_layers=L,
                     rope_base=shp.rope_base, eps=shp.eps, dtype=S.BF16)
    kv = S.sarathi_kv_alloc(cfg, st.kv.shape[1], st.kv.shape[4], st.kv.data_ptr(), st.kv.numel() * 2)
    wabi = [S.make_weights({k: t.data_ptr() for k, t in lw.items()}) for lw in st.weights]
    b = st.batch
    T, C, B = b.n_tokens, b.chunk_len, b.n_decodes
    ws_bytes = S.sarathi_workspace_bytes(cfg, T, B, st.kv.shape[4])
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    def run(batch, x, steps_, warmup_):
        bb, keep = S.make_batch(batch.prefill_slot, batch.chunk_offset, batch.chunk_len, list(batch.decode_slots),
                                list(batch.decode_ctx))
        y = torch.empty_like(x)
        call = lambda: S.sarathi_model_step(cfg, wabi, kv, bb, x.data_ptr(), y.data_ptr(), ws.data_ptr(), ws_bytes,
                                            stream.cuda_stream)
        for _ in range(warmup_):
            call()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps_):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps_

    ms = run(b, st.x, steps, warmup)
    bp = wl.Batch(b.prefill_slot, b.chunk_offset, C, np.zeros(0, np.int32), np.zeros(0, np.int32))
    bd = wl.Batch(-1, 0, 0, b.decode_slots, b.decode_ctx)
    ms_p = run(bp, st.x[:C].clone(), steps, 1)
    ms_d = run(bd, st.x[C:].clone(), steps, 1)
    t_h = accounting.decode_time_per_token_hybrid(ms, ms_p, B)
    t_b = accounting.decode_time_per_token_baseline(ms_d, B)
    out = {"workload": w.name, "layers": L, "rows": T, "ms_per_step": round(ms, 4),
           "tokens_per_s": round(T / (ms * 1e-3), 1), "ms_per_layer": round(ms / L, 5),
           "prefill_only_ms_per_step": round(ms_p, 4), "decode_only_ms_per_step": round(ms_d, 4),
           "decode_tokens_per_s_hybrid": round(1e3 / t_h, 1) if t_h > 0 else None,
           "decode_tokens_per_s_hybrid_accounting": "Sec. 5.1.1: B / (t_hybrid - t_prefill_only)",
           "decode_tokens_per_s_decode_only": round(1e3 / t_b, 1),
           "decode_speedup": round(t_b / t_h, 3) if t_h > 0 else None}
    out["decode_tokens_per_s_plain"] = round(B / (ms * 1e-3), 1)
    del st, ws
    torch.cuda.empty_cache()
    if cpu_baseline:
        import oracle
        out["cpu_baseline"] = oracle_stack_baseline(oracle, shp, b, L)
    return out


def per_call_ms(make_call, stream, steps):
    """Time of each of ``steps`` consecutive calls, from HIP events recorded
    between them on the launch stream (one event per call boundary)."""
    import torch
    call, keep = make_call()
    call()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(steps):
        call()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    return [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]


def cold_call_ms(make_call, stream, steps, flush_bytes=1 << 30):
    """Time of each of ``steps`` calls made with cold caches: before each
    call a 1 GiB buffer is read on the same stream (more than the 256 MB
    memory-side cache and the L2s hold; a read leaves clean lines behind,
    so no write-back lands inside the call), then HIP events bracket the
    call alone."""
    import torch
    call, keep = make_call()
    buf = torch.ones(flush_bytes // 4, dtype=torch.float32, device="cuda")
    call()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    for i in range(steps):
        buf.sum()
        ev[i][0].record(stream)
        call()
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    del buf
    return [a.elapsed_time(b) for a, b in ev]


def oracle_cpu_baseline(oracle, shp, w, kv_layer, ob, x, T, budget_s=25.0, one_core_max_s=45.0):
    """The oracle on the host cores: one full layer call of the workload,
    one untimed warm-up, then the median of up to 3 calls within budget_s
    with every BLAS thread, and one call limited to a single thread (skipped
    when it would take longer than one_core_max_s)."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits
    kv = kv_layer.copy()          # the oracle writes the new K/V rows in place (same values every call)
    run = lambda: oracle.layer_forward(shp, w, kv, ob, x)
    run()
    times = []
    t0 = time.perf_counter()
    while len(times) < 3 and time.perf_counter() - t0 < budget_s:
        t1 = time.perf_counter()
        run()
        times.append(time.perf_counter() - t1)
    blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = int(max([i.get("num_threads", 1) for i in blas], default=1))
    lib = ", ".join(f"{i.get('internal_api')} {i.get('version')}" for i in blas) or "none"
    t_cpu = float(np.median(times))
    one = None
    if t_cpu * threads <= one_core_max_s:
        with threadpool_limits(limits=1, user_api="blas"):
            t1 = time.perf_counter()
            run()
            one = time.perf_counter() - t1
    return {"value": round(T / t_cpu, 2), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"one full layer call of the same workload ({T} rows), float64 NumPy, median of "
                      f"{len(times)} runs of {t_cpu:.2f}s after one warm-up; host affinity "
                      f"{len(os.sched_getaffinity(0))} cpus",
            "blas": lib, "one_core_value": round(T / one, 2) if one else None}


class _SlotKV:
    """One layer's KV cache as the oracle indexes it ([slot, kv, head, pos,
    d]), holding only positions [0, n) of the slots a batch touches."""

    def __init__(self, need: dict, nh: int, d: int):
        self.blk = {s: np.full((2, nh, n, d), 0.5, np.float32) for s, n in need.items()}

    def __getitem__(self, idx):
        return self.blk[int(idx[0])][tuple(idx[1:])]

    def __setitem__(self, idx, val):
        self.blk[int(idx[0])][tuple(idx[1:])] = val


def oracle_stack_baseline(oracle, shp, b, n_layers: int, budget_s: float = 8.0):
    """The oracle on the host cores for the 40-layer stack: one layer of the
    stack's step-0 batch (same rows, chunk and decode contexts; constant
    weights and cache values of the same shapes -- the time of the plain
    NumPy arithmetic does not depend on the values), timed after one
    warm-up call (median of the calls that fit budget_s, at least one), then
    multiplied by the layer count and labelled as extrapolated."""
    from threadpoolctl import threadpool_info
    rng = np.random.default_rng(0)
    H, nh, d, F = shp.hidden, shp.n_heads, shp.head_dim, shp.ffn
    f32 = lambda *sh: np.full(sh, 0.01, np.float32)
    w = {"w_qkv": f32(3 * nh * d, H), "w_o": f32(H, nh * d), "w_up": f32(shp.up_rows, H), "w_down": f32(H, F),
         "norm1_g": np.ones(H, np.float32), "norm2_g": np.ones(H, np.float32)}
    need = {}
    if b.chunk_len:
        need[int(b.prefill_slot)] = int(b.chunk_offset) + int(b.chunk_len)
    for s_, c in zip(b.decode_slots, b.decode_ctx):
        need[int(s_)] = int(c) + 1
    ob = oracle.OracleBatch(b.prefill_slot, b.chunk_offset, b.chunk_len, list(b.decode_slots), list(b.decode_ctx))
    x = rng.random((b.n_tokens, H), dtype=np.float32) - 0.5
    kv = _SlotKV(need, nh, d)
    run = lambda: oracle.layer_forward(shp, w, kv, ob, x)
    run()
    times = []
    t0 = time.perf_counter()
    while len(times) < 3 and time.perf_counter() - t0 < budget_s:
        t1 = time.perf_counter()
        run()
        times.append(time.perf_counter() - t1)
    blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = int(max([i.get("num_threads", 1) for i in blas], default=1))
    t_layer = float(np.median(times))
    t_step = t_layer * n_layers
    return {"value": round(b.n_tokens / t_step, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "extrapolated": True,
            "sample": f"one layer of the stack's step-0 batch ({b.n_tokens} rows), float64 NumPy, median of "
                      f"{len(times)} runs of {t_layer:.2f}s after one warm-up, times {n_layers} layers "
                      f"(extrapolated, not run); host affinity {len(os.sched_getaffinity(0))} cpus",
            "ms_per_step": round(t_step * 1e3, 1)}


def stage_work(shp, b):
    """Algorithmic FLOPs and HBM bytes of each stage of one layer call --
    only what the method itself must compute and move (Sec. 4.3's fused
    linear ops and separate attention): weights once, KV read once per query
    set, activations once in and once out, attention output rows counted
    with the attention that produces them; FLOPs count 2 per multiply-add,
    attention pairs only where the mask allows them.  The combine of
    attention key-splits is implementation overhead (no method bytes)."""
    T, C, B = b.n_tokens, b.chunk_len, b.n_decodes
    H, nh, hd, F = shp.hidden, shp.n_heads, shp.head_dim, shp.ffn
    QD = nh * hd
    es = 2 if shp.dtype == "bf16" else 4
    up_rows = 2 * F if shp.act == "swiglu" else F
    ctx = [int(c) for c in b.decode_ctx]
    dec_keys = sum(c + 1 for c in ctx)
    pre_pairs = C * b.chunk_offset + C * (C + 1) // 2
    pre_keys = b.chunk_offset + C if C else 0
    w = {}
    w["norm_1"] = (0.0, 2 * T * H * es + T * H * 4)
    w["preproj"] = (2.0 * T * H * 3 * QD, 3 * QD * H * es + T * H * es + T * 3 * QD * es)
    w["rope_kv_append"] = (0.0, 2 * T * 3 * QD * es + T * QD * es)
    w["chunk_attention"] = (4.0 * pre_pairs * hd * nh, pre_keys * 2 * QD * es + 2 * C * QD * es)
    w["decode_attention"] = (4.0 * dec_keys * hd * nh, dec_keys * 2 * QD * es + 2 * B * QD * es)
    w["attention_combine"] = (0.0, 0.0)
    w["postproj"] = (2.0 * T * QD * H, H * QD * es + T * QD * es + T * H * es + T * H * 4)
    w["norm_2"] = (0.0, T * H * 4 + T * H * es + T * H * 4)
    w["ffn_ln1"] = (2.0 * T * H * up_rows, up_rows * H * es + T * H * es + T * F * es)
    w["ffn_ln2"] = (2.0 * T * F * H, H * F * es + T * F * es + T * H * 4 + T * H * es)
    return w


def stage_overhead(shp, b, attn_plan, split_counts=None):
    """HBM bytes each stage moves beyond the method's own (stage_work): the
    fp32 key-split partials of the attention (hd + 4 floats per row and head;
    attn_plan: the library's sarathi_attention_plan of the batch -- the rows
    each attention kernel writes and the combine pass reads back, plus the
    output rows the combine writes), and the fp32 split-K partials of
    postproj and ffn_ln2 (split_counts: stage -> K-splits of its matmul),
    written by the matmul and read back by its reduction pass."""
    T = b.n_tokens
    H, nh, hd = shp.hidden, shp.n_heads, shp.head_dim
    es = 2 if shp.dtype == "bf16" else 4
    part_bytes = nh * (hd + 4) * 4
    dec_rows = attn_plan["decode_items"]
    o = {k: 0.0 for k in BOUND}
    o["chunk_attention"] = (attn_plan["partial_rows_written"] - dec_rows) * part_bytes
    o["decode_attention"] = dec_rows * part_bytes
    o["attention_combine"] = (attn_plan["partial_rows_read"] * part_bytes
                              + attn_plan["combine_rows"] * nh * hd * es)
    for st, ns in (split_counts or {}).items():
        if ns > 1:
            o[st] += 2.0 * ns * T * H * 4
    return o


def counter_traffic(stage: str, workload: str):
    """HBM bytes per launch of a stage's kernel from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE record (profiles/traffic_<stage>_<workload>.json),
    or None when there is no record or the kernel's source changed since."""
    import hashlib
    p = os.path.join(ROOT, "profiles", f"traffic_{stage}_{workload}.json")
    if not os.path.exists(p):
        return None
    rec = json.load(open(p))
    src = os.path.join(ROOT, rec["source"])
    if not os.path.exists(src):
        return None
    if hashlib.sha256(open(src, "rb").read()).hexdigest()[:16] != rec["source_sha256_16"]:
        return None
    return round(rec["traffic_bytes"])


# The bar the fused linear ops of a hybrid batch are held to: 60% of dense
# MFMA peak over C + B rows (the premise of Sec. 4.3 that the linear ops,
# fused over the chunk and the decodes, run near the compute roof).
LINEAR_MFMA_TARGET = 0.60

BOUND = {"norm_1": "hbm", "preproj": "mfma", "rope_kv_append": "hbm", "chunk_attention": "mfma",
         "decode_attention": "hbm", "attention_combine": "overhead", "postproj": "mfma", "norm_2": "hbm",
         "ffn_ln1": "mfma", "ffn_ln2": "mfma"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the hot path runs on a single MI355X and has no multi-GPU mode "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import workloads as wl
    from paper_2308_16369_amd import sarathi as S
    from paper_2308_16369_amd import accounting

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.stack_only:
        print(json.dumps(bench_stack(args.stack_steps, 2, cpu_baseline=not args.no_cpu_baseline)), flush=True)
        return
    w = wl.WORKLOADS[args.workload]
    shp = w.shape
    t0 = time.time()
    inst = wl.generate(w)
    print(f"# generated {w.name} in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    b = inst.batch
    T, C, B = b.n_tokens, b.chunk_len, b.n_decodes

    def dev(a):
        if shp.dtype == "bf16":
            return torch.from_numpy(wl.bf16_bits(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()

    cfg = S.make_cfg(hidden=shp.hidden, n_heads=shp.n_heads, head_dim=shp.head_dim, ffn=shp.ffn, n_layers=1,
                     norm=S.NORM_RMS if shp.norm == "rms" else S.NORM_LAYER,
                     act=S.ACT_SWIGLU if shp.act == "swiglu" else S.ACT_GELU, rope=int(shp.rope),
                     rope_base=shp.rope_base, eps=shp.eps, dtype=S.BF16 if shp.dtype == "bf16" else S.F32)
    wdev = {k: dev(v) for k, v in inst.weights[0].items()}
    wabi = S.make_weights({k: t.data_ptr() for k, t in wdev.items()})
    kv_t = dev(inst.kv)
    Sx = kv_t.shape[4]
    kv = S.sarathi_kv_alloc(cfg, kv_t.shape[1], Sx, kv_t.data_ptr(), kv_t.numel() * kv_t.element_size())
    ws_bytes = S.sarathi_workspace_bytes(cfg, T, B, Sx)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    x = dev(inst.x)
    y = torch.empty_like(x)
    stream = torch.cuda.current_stream()
    print(f"# uploaded in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    def run(batch, xin, xout, steps, warmup, profile=False):
        bb, keep = S.make_batch(batch.prefill_slot, batch.chunk_offset, batch.chunk_len,
                                list(batch.decode_slots), list(batch.decode_ctx))
        call = lambda: S.sarathi_hybrid_layer_forward(cfg, wabi, kv, 0, bb, xin.data_ptr(), xout.data_ptr(),
                                                      ws.data_ptr(), ws_bytes, stream.cuda_stream)
        for _ in range(warmup):
            call()
        torch.cuda.synchronize()
        if profile:
            S.sarathi_profile_begin(steps)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t_wall = time.perf_counter()
        e0.record(stream)
        for _ in range(steps):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t_wall
        stages = None
        if profile:
            stages, n = S.sarathi_profile_end()
            stages = {k: v / n for k, v in stages.items()}
        return e0.elapsed_time(e1) / steps, wall / steps * 1e3, stages

    def run_once(batch, xin, xout):
        bb, keep = S.make_batch(batch.prefill_slot, batch.chunk_offset, batch.chunk_len,
                                list(batch.decode_slots), list(batch.decode_ctx))
        return lambda: S.sarathi_hybrid_layer_forward(cfg, wabi, kv, 0, bb, xin.data_ptr(), xout.data_ptr(),
                                                      ws.data_ptr(), ws_bytes, stream.cuda_stream), keep

    # ---- timed region: K hybrid steps, with per-stage HIP events on the launch stream
    ms, wall_ms, stages = run(b, x, y, args.steps, args.warmup, profile=True)
    # ---- same steps without the stage events (the events' own cost)
    ms_plain, _, _ = run(b, x, y, args.steps, 2)
    print(f"# hybrid: {ms:.4f} ms/step with stage events, {ms_plain:.4f} without", file=sys.stderr, flush=True)
    # ---- spread: the same steps with one event between consecutive calls
    per_call = per_call_ms(lambda: run_once(b, x, y), stream, args.steps)
    # ---- cold caches: each call after a 1 GiB write (outside the timed region above)
    cold = cold_call_ms(lambda: run_once(b, x, y), stream, max(args.steps, 10))

    # ---- decode accounting (Sec. 5.1.1): prefill-only and decode-only batches of the same rows
    extra = {}
    if not args.no_compare and C > 0 and B > 0:
        bp = wl.Batch(b.prefill_slot, b.chunk_offset, C, np.zeros(0, np.int32), np.zeros(0, np.int32))
        bd = wl.Batch(-1, 0, 0, b.decode_slots, b.decode_ctx)
        xp, yp = x[:C].clone(), torch.empty_like(x[:C])
        xd, yd = x[C:].clone(), torch.empty_like(x[C:])
        ms_p, _, _ = run(bp, xp, yp, args.steps, 2)
        ms_d, _, _ = run(bd, xd, yd, args.steps, 2)
        t_dec_h = accounting.decode_time_per_token_hybrid(ms_plain, ms_p, B)
        t_dec_b = accounting.decode_time_per_token_baseline(ms_d, B)
        extra = {
            "prefill_only_ms": round(ms_p, 5), "decode_only_ms": round(ms_d, 5),
            "decode_tokens_per_s_hybrid": round(1e3 / t_dec_h, 1) if t_dec_h > 0 else None,
            "decode_tokens_per_s_hybrid_accounting": "Sec. 5.1.1: B / (t_hybrid - t_prefill_only)",
            "decode_tokens_per_s_plain": round(B / (ms_plain * 1e-3), 1),
            "decode_tokens_per_s_decode_only": round(1e3 / t_dec_b, 1),
            "decode_speedup": round(t_dec_b / t_dec_h, 3) if t_dec_h > 0 else None,
        }

    if args.copy_calibration:
        a = torch.empty(1 << 29, dtype=torch.float16, device="cuda").fill_(1.0)   # 1 GiB
        c = torch.empty_like(a)
        for _ in range(3):
            torch.mul(a, 1.0, out=c)
        torch.cuda.synchronize()
        del a, c

    # ---- rooflines per stage (method FLOPs and bytes), with each stage's
    # implementation overhead traffic reported beside them
    work = stage_work(shp, b)
    dt_abi = S.BF16 if shp.dtype == "bf16" else S.F32
    split_scratch = S.sarathi_layer_split_scratch_bytes(cfg, T)
    QD = shp.n_heads * shp.head_dim
    splits = {"postproj": S.sarathi_linear_plan(dt_abi, S.LINEAR_RESID, T, shp.hidden, QD, split_scratch)[2],
              "ffn_ln2": S.sarathi_linear_plan(dt_abi, S.LINEAR_RESID_F32IN, T, shp.hidden, shp.ffn,
                                               split_scratch)[2]}
    bb_plan, keep_plan = S.make_batch(b.prefill_slot, b.chunk_offset, C, list(b.decode_slots), list(b.decode_ctx))
    over = stage_overhead(shp, b, S.sarathi_attention_plan(cfg, bb_plan), splits)
    peak_flops = PEAK_BF16_TFLOPS if shp.dtype == "bf16" else PEAK_F32_TFLOPS
    kernels = {}
    for name, t in stages.items():
        fl, by = work[name]
        sec = t * 1e-3
        if sec <= 0:
            continue
        tf = fl / sec / 1e12
        gb = by / sec / 1e9
        kernels[name] = {"ms": round(t, 5), "tflops": round(tf, 2), "gbps": round(gb, 1),
                         "mfma_frac": round(tf / peak_flops, 4), "hbm_frac": round(gb / PEAK_HBM_GBPS, 4),
                         "bound": BOUND[name], "overhead_bytes": round(over[name]),
                         "gbps_with_overhead": round((by + over[name]) / sec / 1e9, 1)}
        if name in splits:
            kernels[name]["k_splits"] = splits[name]
    dom = max((k for k in kernels if kernels[k]["bound"] != "overhead"), key=lambda k: kernels[k]["ms"])
    dk = kernels[dom]
    if dk["bound"] == "mfma":
        roof = {"bound": "mfma", "achieved": dk["tflops"], "peak": peak_flops, "unit": "TFLOP/s",
                "frac": dk["mfma_frac"]}
    else:
        roof = {"bound": "hbm", "achieved": dk["gbps"], "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                "frac": dk["hbm_frac"]}
    roof["kernel"] = dom
    roof["traffic"] = counter_traffic(dom, w.name)
    # layer roofline: every stage at the larger of its MFMA and HBM times
    roof_ms = sum(max(fl / (peak_flops * 1e12), by / (PEAK_HBM_GBPS * 1e9)) for fl, by in work.values()) * 1e3
    over_total = sum(over.values())
    lin = ["preproj", "postproj", "ffn_ln1", "ffn_ln2"]
    lin_ms = sum(kernels[k]["ms"] for k in lin if k in kernels)
    lin_flops = sum(work[k][0] for k in lin)
    lin_bytes = sum(work[k][1] for k in lin)

    # ---- oracle on the host cores, bounded sample: one full layer call (all T rows)
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        ob = oracle.OracleBatch(b.prefill_slot, b.chunk_offset, C, list(b.decode_slots), list(b.decode_ctx))
        cpu = oracle_cpu_baseline(oracle, shp, inst.weights[0], inst.kv[0], ob, inst.x, T)

    stack = None
    if not args.no_stack:
        del kv_t, wdev, ws
        torch.cuda.empty_cache()
        t_s = time.time()
        stack = bench_stack(args.stack_steps, 2, cpu_baseline=not args.no_cpu_baseline)
        print(f"# stack measured in {time.time() - t_s:.1f}s: {stack['ms_per_step']} ms per step",
              file=sys.stderr, flush=True)

    value = T / (ms_plain * 1e-3)
    lin_mfma = lin_flops / (lin_ms * 1e-3) / 1e12 / peak_flops
    line = {
        "metric": "hybrid-batch tokens/s per layer (C+B rows per layer forward)",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_plain, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": shp.dtype,
        "data": "synthetic (seeded N(0,1) activations/KV, N(0,0.02) weights; no trained weights)",
        "config": {"workload": w.name, "hidden": shp.hidden, "heads": shp.n_heads, "head_dim": shp.head_dim,
                   "ffn": shp.ffn, "chunk_len": C, "chunk_offset": b.chunk_offset, "n_decodes": B,
                   "ctx_range": [w.batch.ctx_lo, w.batch.ctx_hi], "rows": T, "parallelism": "none (1 GPU)"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "layer_roofline": {"ms": round(roof_ms, 5), "frac": round(roof_ms / ms_plain, 4),
                           "overhead_bytes": round(over_total)},
        "ms_per_call_p10_p50_p90": [round(float(np.percentile(per_call, q)), 5) for q in (10, 50, 90)],
        "cold": {"ms_per_call_p10_p50_p90": [round(float(np.percentile(cold, q)), 5) for q in (10, 50, 90)],
                 "tokens_per_s_p50": round(T / (float(np.median(cold)) * 1e-3), 1),
                 "calls": len(cold), "note": "each call timed alone after a 1 GiB read that evicts the "
                                             "memory-side cache and the L2s"},
        "ms_per_step_with_stage_events": round(ms, 5),
        "wall_ms_per_step": round(wall_ms, 5),
        "linear_ops": {"ms": round(lin_ms, 5), "mfma_frac": round(lin_mfma, 4),
                       "weight_stream_hbm_frac": round(lin_bytes / (lin_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
                       "target_mfma_frac": LINEAR_MFMA_TARGET, "target_met": bool(lin_mfma >= LINEAR_MFMA_TARGET)},
        "kernels": kernels,
        **extra,
        "stack": stack,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
