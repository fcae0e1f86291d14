"""Chunk-size ablation and tile-quantization sweep of the hybrid-batch layer.

Effects of the chunk size the paper measures (Sec. 4.4, tile quantization;
Sec. 5.4, ablation of chunked prefills), taken here on this library's kernels
through the C-ABI:

* tile quantization: the fused linear ops run whole output tiles over the
  T = C + B rows of a batch, so the layer time rises in steps just past the
  row-tile multiples (the paper's advice: choose the chunk so that chunk plus
  piggybacked decodes fills whole tiles);
* chunking overhead: a prompt of P tokens prefilled as P / c chunks of c
  tokens costs more than one full prefill -- the matmuls are smaller and each
  chunk re-reads the KV of every earlier chunk.  The overhead is reported for
  the attention alone and for the whole layer, c from 64 to 512;
* decode piggybacking: for a chunk of c tokens and B decodes, the decode time
  per token of the hybrid batch (hybrid minus prefill-only time, over B)
  against a decode-only batch (the accounting of Sec. 5.1.1);
* the per-token prefill and decode times of Sec. 4.3's table, re-run on the
  whole 40-layer LLaMA-13B model: a prefill-only iteration of 1024 tokens, a
  decode-only iteration of 4 decodes at sequence length 1024, and a
  decode-maximal iteration of one 1021-token chunk plus 3 decodes, each split
  into linear-op, attention and other time;
* a tile sweep of the four linear ops of a workload's layer: every
  producer/consumer tile shape (and, for the residual ops, the split-K count
  the planner would use) timed alone through sarathi_linear_tiled, next to
  the planner's pick.

Inputs are seeded synthetic tensors drawn on the device (weights
0.02 * N(0,1), activations and cached K/V N(0,1)); only timing is measured
here -- the same kernels' results are checked against the oracle by the
parity tests.

Command line (one GPU):
    python -m paper_2308_16369_amd.ablation --json out.json --md out.md
"""
from __future__ import annotations

import argparse
import json
import sys
import time
from dataclasses import dataclass
from typing import Callable, Dict, List, Optional, Sequence, Tuple

LINEAR_STAGES = ("preproj", "postproj", "ffn_ln1", "ffn_ln2")
ATTENTION_STAGES = ("chunk_attention", "decode_attention", "attention_combine")

# Sec. 4.3's table (LLaMA-13B, A6000): total ms of one iteration of the whole
# model, linear / attention / total, for the three batch kinds (context only).
PAPER_TABLE2_A6000 = {"prefill_only": (224.8, 10.0, 234.8), "decode_only": (44.28, 5.68, 49.96),
                      "decode_maximal": (223.2, 15.2, 238.4)}


def chunk_plan(prompt_len: int, chunk: int) -> List[Tuple[int, int]]:
    """(offset, length) of each chunk when a prompt of ``prompt_len`` tokens
    is prefilled ``chunk`` tokens at a time (the last chunk may be shorter)."""
    if prompt_len < 1 or chunk < 1:
        raise ValueError("prompt_len and chunk must be positive")
    return [(o, min(chunk, prompt_len - o)) for o in range(0, prompt_len, chunk)]


def tile_lengths(lo: int, hi: int, step: int, tiles: Sequence[int]) -> List[int]:
    """Row counts for the tile-quantization sweep: every ``step`` rows in
    [lo, hi] plus each tile multiple m in range and m +- 1."""
    pts = set(range(lo, hi + 1, step))
    for t in tiles:
        for m in range(t, hi + 2, t):
            pts.update(v for v in (m - 1, m, m + 1) if lo <= v <= hi)
    return sorted(pts)


@dataclass
class Batch:
    prefill_slot: int
    chunk_offset: int
    chunk_len: int
    decode_slots: List[int]
    decode_ctx: List[int]

    @property
    def n_tokens(self) -> int:
        return self.chunk_len + len(self.decode_slots)


class LayerRunner:
    """One layer on the device, a KV cache of ``n_slots`` x ``max_seq_len``
    positions, and a workspace for up to ``max_tokens`` rows."""

    def __init__(self, shape, n_slots: int, max_seq_len: int, max_tokens: int, max_decodes: int, seed: int = 0,
                 max_chunks: int = 1):
        import torch

        from workloads.stack import generate_layer_on_device
        from . import sarathi as S

        self.S, self.torch, self.shape = S, torch, shape
        self.dev = generate_layer_on_device(shape, n_slots, max_seq_len, seed)
        self.cfg = S.make_cfg(hidden=shape.hidden, n_heads=shape.n_heads, head_dim=shape.head_dim, ffn=shape.ffn,
                              n_layers=1, norm=S.NORM_RMS if shape.norm == "rms" else S.NORM_LAYER,
                              act=S.ACT_SWIGLU if shape.act == "swiglu" else S.ACT_GELU, rope=int(shape.rope),
                              rope_base=shape.rope_base, eps=shape.eps,
                              dtype=S.BF16 if shape.dtype == "bf16" else S.F32)
        kvt = self.dev.kv
        self.kv = S.sarathi_kv_alloc(self.cfg, n_slots, max_seq_len, kvt.data_ptr(),
                                     kvt.numel() * kvt.element_size())
        self.w = S.make_weights({k: t.data_ptr() for k, t in self.dev.weights.items()})
        self.ws_bytes = S.sarathi_mixed_workspace_bytes(self.cfg, max_tokens, max_chunks, max_seq_len)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device="cuda")
        g = torch.Generator(device="cuda")
        g.manual_seed(seed + 1)
        self.x = torch.empty((max_tokens, shape.hidden), dtype=kvt.dtype, device="cuda").normal_(0.0, 1.0,
                                                                                                generator=g)
        self.y = torch.empty_like(self.x)
        self.stream = torch.cuda.current_stream()

    def call(self, b: Batch) -> Callable[[], None]:
        """A zero-argument launcher of one layer call on batch ``b``."""
        bb, keep = self.S.make_batch(b.prefill_slot, b.chunk_offset, b.chunk_len, list(b.decode_slots),
                                     list(b.decode_ctx))
        S, x, y = self.S, self.x, self.y

        def launch(bb=bb, keep=keep):   # the closure keeps the host arrays alive
            S.sarathi_hybrid_layer_forward(self.cfg, self.w, self.kv, 0, bb, x.data_ptr(), y.data_ptr(),
                                           self.ws.data_ptr(), self.ws_bytes, self.stream.cuda_stream)
        return launch

    def call_mixed(self, chunks, decode_slots, decode_ctx) -> Callable[[], None]:
        """A launcher of one layer call on a mixed batch: chunks [(slot, offset, length)]."""
        mb, keep = self.S.make_mixed_batch(chunks, list(decode_slots), list(decode_ctx))
        S, x, y = self.S, self.x, self.y

        def launch(mb=mb, keep=keep):
            S.sarathi_mixed_layer_forward(self.cfg, self.w, self.kv, 0, mb, x.data_ptr(), y.data_ptr(),
                                          self.ws.data_ptr(), self.ws_bytes, self.stream.cuda_stream)
        return launch

    def time(self, calls: Sequence[Callable[[], None]], iters: int = 20, warmup: int = 3) -> float:
        """Milliseconds for one pass over ``calls`` (launched back to back)."""
        torch = self.torch
        for _ in range(warmup):
            for c in calls:
                c()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(self.stream)
        for _ in range(iters):
            for c in calls:
                c()
        e1.record(self.stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters

    def stages(self, calls: Sequence[Callable[[], None]], iters: int = 5) -> Dict[str, float]:
        """Per-stage milliseconds summed over one pass of ``calls`` (HIP events
        on the launch stream around each stage)."""
        S, torch = self.S, self.torch
        for c in calls:
            c()
        torch.cuda.synchronize()
        S.sarathi_profile_begin(iters * len(calls))
        for _ in range(iters):
            for c in calls:
                c()
        torch.cuda.synchronize()
        st, n = S.sarathi_profile_end()
        return {k: v / iters for k, v in st.items()}


def tile_quantization(r: LayerRunner, lengths: Sequence[int], iters: int = 20) -> List[dict]:
    """Prefill-only layer calls of T rows (chunk at offset 0): total and
    linear-op milliseconds per call, and microseconds per row."""
    out = []
    for T in lengths:
        calls = [r.call(Batch(0, 0, T, [], []))]
        ms = r.time(calls, iters)
        st = r.stages(calls, 3)
        lin = sum(st[k] for k in LINEAR_STAGES)
        out.append({"rows": T, "ms": round(ms, 5), "linear_ms": round(lin, 5),
                    "us_per_row": round(ms * 1e3 / T, 4),
                    **{f"{k}_ms": round(st[k], 5) for k in LINEAR_STAGES}})
    return out


def chunking_overhead(r: LayerRunner, prompts: Sequence[int], chunks: Sequence[int], iters: int = 10) -> List[dict]:
    """For each prompt length P and chunk size c: the time of the whole chunk
    sequence (P / c prefill-only calls, each attending to every earlier
    chunk) against one full prefill of P rows, for the attention stage and the
    whole layer.  A chunk size of P is the full prefill itself."""
    out = []
    for P in prompts:
        full_calls = [r.call(Batch(0, 0, P, [], []))]
        full_ms = r.time(full_calls, iters)
        full_attn = r.stages(full_calls, 3)["chunk_attention"]
        for c in sorted(set(c for c in chunks if c < P) | {P}):
            calls = [r.call(Batch(0, o, n, [], [])) for o, n in chunk_plan(P, c)]
            ms = r.time(calls, iters)
            st = r.stages(calls, 3)
            out.append({"prompt": P, "chunk": c, "n_chunks": len(calls), "ms": round(ms, 4),
                        "attn_ms": round(st["chunk_attention"], 4), "full_ms": round(full_ms, 4),
                        "full_attn_ms": round(full_attn, 4), "overhead": round(ms / full_ms, 3),
                        "attn_overhead": round(st["chunk_attention"] / full_attn, 3)})
    return out


def piggyback(r: LayerRunner, chunks: Sequence[int], decodes: Sequence[int], ctx: int, offset: int,
              iters: int = 20) -> List[dict]:
    """Hybrid batches of one chunk (c tokens at ``offset``) plus B decodes of
    context ``ctx``: step time, decode time per token against a decode-only
    batch of the same decodes (Sec. 5.1.1), and rows T = c + B."""
    out = []
    for c in chunks:
        for B in decodes:
            slots = list(range(1, B + 1))
            ctxs = [ctx] * B
            t_h = r.time([r.call(Batch(0, offset, c, slots, ctxs))], iters)
            t_p = r.time([r.call(Batch(0, offset, c, [], []))], iters)
            t_d = r.time([r.call(Batch(-1, 0, 0, slots, ctxs))], iters)
            dec_h = (t_h - t_p) / B
            dec_b = t_d / B
            out.append({"chunk": c, "decodes": B, "rows": c + B, "hybrid_ms": round(t_h, 5),
                        "prefill_only_ms": round(t_p, 5), "decode_only_ms": round(t_d, 5),
                        "decode_us_per_token_hybrid": round(dec_h * 1e3, 3),
                        "decode_us_per_token_decode_only": round(dec_b * 1e3, 3),
                        "decode_speedup": round(dec_b / dec_h, 3) if dec_h > 0 else None})
    return out


def table2_batches(seq_len: int = 1024, decodes: int = 4):
    """The three iterations of Sec. 4.3's table at sequence length
    ``seq_len``: prefill-only (one prompt of seq_len tokens, slot 0),
    decode-only (``decodes`` decodes whose new token sits at position
    seq_len - 1, slots 1..decodes) and decode-maximal (a chunk of
    seq_len - (decodes - 1) tokens plus decodes - 1 of those decodes, seq_len
    rows in all)."""
    dec = decodes - 1
    return {"prefill_only": Batch(0, 0, seq_len, [], []),
            "decode_only": Batch(-1, 0, 0, list(range(1, decodes + 1)), [seq_len - 1] * decodes),
            "decode_maximal": Batch(0, 0, seq_len - dec, list(range(1, dec + 1)), [seq_len - 1] * dec),
            "prefill_only_chunk": Batch(0, 0, seq_len - dec, [], [])}


def table2(shape, n_layers: int = 40, seq_len: int = 1024, decodes: int = 4, iters: int = 10) -> dict:
    """Per-token prefill and decode time of the whole model (Sec. 4.3's
    table), with each iteration split into linear ops, attention and the rest
    from per-stage HIP events (summed over layers; the events add a few
    microseconds per stage, so the split is of the profiled run and the
    total of an unprofiled one).  Decode time per token follows Sec. 5.1.1:
    decode-only time / batch, and (decode-maximal - prefill-only) / decodes."""
    import torch

    from workloads.stack import generate_model_on_device
    from . import sarathi as S

    dm = generate_model_on_device(shape, n_layers, decodes + 1, seq_len)
    cfg = S.make_cfg(hidden=shape.hidden, n_heads=shape.n_heads, head_dim=shape.head_dim, ffn=shape.ffn,
                     n_layers=n_layers, norm=S.NORM_RMS if shape.norm == "rms" else S.NORM_LAYER,
                     act=S.ACT_SWIGLU if shape.act == "swiglu" else S.ACT_GELU, rope=int(shape.rope),
                     rope_base=shape.rope_base, eps=shape.eps, dtype=S.BF16 if shape.dtype == "bf16" else S.F32)
    kv = S.sarathi_kv_alloc(cfg, decodes + 1, seq_len, dm.kv.data_ptr(), dm.kv.numel() * dm.kv.element_size())
    wabi = [S.make_weights({k: t.data_ptr() for k, t in lw.items()}) for lw in dm.weights]
    ws_bytes = S.sarathi_workspace_bytes(cfg, seq_len, decodes, seq_len)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    x = torch.empty((seq_len, shape.hidden), dtype=dm.kv.dtype, device="cuda").normal_(0.0, 1.0)
    y = torch.empty_like(x)
    stream = torch.cuda.current_stream()
    out = {}
    for name, b in table2_batches(seq_len, decodes).items():
        bb, keep = S.make_batch(b.prefill_slot, b.chunk_offset, b.chunk_len, b.decode_slots, b.decode_ctx)
        call = lambda: S.sarathi_model_step(cfg, wabi, kv, bb, x.data_ptr(), y.data_ptr(), ws.data_ptr(), ws_bytes,
                                            stream.cuda_stream)
        for _ in range(2):
            call()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(iters):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        total = e0.elapsed_time(e1) / iters
        S.sarathi_profile_begin(3 * n_layers)
        for _ in range(3):
            call()
        torch.cuda.synchronize()
        st, n = S.sarathi_profile_end()
        st = {k: v / 3 for k, v in st.items()}
        lin = sum(st[k] for k in LINEAR_STAGES)
        att = sum(st[k] for k in ATTENTION_STAGES)
        out[name] = {"rows": b.n_tokens, "prefill_tokens": b.chunk_len, "decode_tokens": len(b.decode_slots),
                     "total_ms": round(total, 4), "linear_ms": round(lin, 4), "attention_ms": round(att, 4),
                     "other_ms": round(sum(st.values()) - lin - att, 4),
                     "profiled_total_ms": round(sum(st.values()), 4)}
    p, d, h, pc = (out[k]["total_ms"] for k in ("prefill_only", "decode_only", "decode_maximal",
                                                 "prefill_only_chunk"))
    dec = decodes - 1
    out["per_token_ms"] = {
        "prefill": round(p / seq_len, 5),
        "decode_baseline": round(d / decodes, 5),
        "decode_hybrid": round((h - p) / dec, 5),
        "decode_hybrid_same_chunk": round((h - pc) / dec, 5),
    }
    out["decode_speedup"] = round((d / decodes) / ((h - p) / dec), 3) if h > p else None
    out["decode_speedup_same_chunk"] = round((d / decodes) / ((h - pc) / dec), 3) if h > pc else None
    out["layers"], out["seq_len"], out["decodes"] = n_layers, seq_len, decodes
    del ws, dm
    torch.cuda.empty_cache()
    return out


def table2_markdown(t: dict) -> str:
    rows = [("prefill_only", f"prefill-only ({t['seq_len']} tokens)"),
            ("decode_only", f"decode-only ({t['decodes']} decodes at {t['seq_len']})"),
            ("decode_maximal", f"decode-maximal ({t['seq_len'] - t['decodes'] + 1} + {t['decodes'] - 1})"),
            ("prefill_only_chunk", f"prefill-only ({t['seq_len'] - t['decodes'] + 1} tokens)")]
    L = [f"## Per-token prefill and decode time, whole {t['layers']}-layer model (Sec. 4.3's table)", "",
         "Linear = preproj + postproj + ffn_ln1 + ffn_ln2 (split-K reductions included), attention = chunk + "
         "decode attention + combine, other = norms and the rotary/KV append when it runs alone; the split is "
         "from a run with per-stage events (a few us each), the total from one without.  The paper's A6000 "
         "values are context, not a target.", "",
         "| iteration | rows | linear ms | attention ms | other ms | total ms | paper A6000 linear / attn / total ms |",
         "|---|---|---|---|---|---|---|"]
    for k, label in rows:
        e = t[k]
        pap = PAPER_TABLE2_A6000.get(k)
        ps = " / ".join(f"{v:g}" for v in pap) if pap else "—"
        L.append(f"| {label} | {e['rows']} | {e['linear_ms']:.3f} | {e['attention_ms']:.3f} | {e['other_ms']:.3f} | "
                 f"{e['total_ms']:.3f} | {ps} |")
    pt = t["per_token_ms"]
    L += ["", "| per-token time | this GPU (ms) | paper A6000 (ms) |", "|---|---|---|",
          f"| prefill (prefill-only time / {t['seq_len']}) | {pt['prefill']:.5f} | 0.229 |",
          f"| decode, decode-only batch (time / {t['decodes']}) | {pt['decode_baseline']:.4f} | 12.49 |",
          f"| decode, decode-maximal batch ((decode-maximal - prefill-only {t['seq_len']}) / "
          f"{t['decodes'] - 1}) | {pt['decode_hybrid']:.4f} | 1.2 |",
          f"| decode, decode-maximal batch ((decode-maximal - prefill-only {t['seq_len'] - t['decodes'] + 1}) / "
          f"{t['decodes'] - 1}) | {pt['decode_hybrid_same_chunk']:.4f} | — |",
          "", f"Decode speedup: {t['decode_speedup']} (paper: 12.49 / 1.2 = 10.4); against the prefill-only time of "
              f"the same {t['seq_len'] - t['decodes'] + 1}-token chunk: {t['decode_speedup_same_chunk']}.", ""]
    return "\n".join(L) + "\n"


def to_markdown(res: dict) -> str:
    L = [f"# Chunk-size ablation and tile quantization: {res['workload']}", "",
         f"Command: `{res['command']}`", "", "## Tile quantization (prefill-only layer call of T rows)", "",
         "| T | layer ms | linear ms | us/row | preproj | postproj | ffn_ln1 | ffn_ln2 |",
         "|---|---|---|---|---|---|---|---|"]
    for e in res["tile_quantization"]:
        L.append(f"| {e['rows']} | {e['ms']:.4f} | {e['linear_ms']:.4f} | {e['us_per_row']:.3f} | "
                 f"{e['preproj_ms']:.4f} | {e['postproj_ms']:.4f} | {e['ffn_ln1_ms']:.4f} | {e['ffn_ln2_ms']:.4f} |")
    L += ["", "## Chunked prefill against one full prefill (Sec. 5.4)", "",
          "| prompt | chunk | chunks | layer ms | overhead | attention ms | attention overhead |",
          "|---|---|---|---|---|---|---|"]
    for e in res["chunking_overhead"]:
        L.append(f"| {e['prompt']} | {e['chunk']} | {e['n_chunks']} | {e['ms']:.3f} | {e['overhead']:.3f} | "
                 f"{e['attn_ms']:.3f} | {e['attn_overhead']:.3f} |")
    L += ["", f"## Decode piggybacking (decodes of context {res['piggyback_ctx']}, chunk at offset "
              f"{res['piggyback_offset']})", "",
          "| chunk | decodes | T | hybrid ms | prefill-only ms | decode-only ms | decode us/token hybrid | "
          "decode-only | speedup |", "|---|---|---|---|---|---|---|---|---|"]
    for e in res["piggyback"]:
        L.append(f"| {e['chunk']} | {e['decodes']} | {e['rows']} | {e['hybrid_ms']:.4f} | {e['prefill_only_ms']:.4f} | "
                 f"{e['decode_only_ms']:.4f} | {e['decode_us_per_token_hybrid']:.2f} | "
                 f"{e['decode_us_per_token_decode_only']:.2f} | {e['decode_speedup']} |")
    out = "\n".join(L) + "\n"
    if res.get("table2"):
        out += "\n" + table2_markdown(res["table2"])
    return out


def tile_sweep(shape, T: int, iters: int = 20) -> List[dict]:
    """Every producer/consumer tile of the four linear ops over T rows, each op
    alone (split reductions included), with the planner's pick."""
    import torch

    from . import sarathi as S

    def _time(fn: Callable[[], None], n: int) -> float:   # ms per call, events on the null stream fn uses
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    H, nh, d, F = shape.hidden, shape.n_heads, shape.head_dim, shape.ffn
    QD = nh * d
    dt = torch.bfloat16
    up_kind = S.LINEAR_SWIGLU if shape.act == "swiglu" else S.LINEAR_GELU
    ops = [("preproj", S.LINEAR_PLAIN, 3 * QD, H, 3 * QD), ("postproj", S.LINEAR_RESID, H, QD, H),
           ("ffn_ln1", up_kind, F, H, shape.up_rows), ("ffn_ln2", S.LINEAR_RESID_F32IN, H, F, H)]
    scratch_bytes = S.sarathi_linear_scratch_bytes(T, max(H, F))
    scratch = torch.empty(scratch_bytes // 4 + 1, dtype=torch.float32, device="cuda")
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    out: List[dict] = []
    for name, kind, N, K, w_rows in ops:
        x = (torch.randn(T, K, generator=g, device="cuda") * 0.5).to(dt)
        w = (torch.randn(w_rows, K, generator=g, device="cuda") * 0.02).to(dt)
        resid_dt = torch.float32 if kind == S.LINEAR_RESID_F32IN else dt
        out_dt = torch.float32 if kind == S.LINEAR_RESID else dt
        resid = torch.randn(T, N, generator=g, device="cuda").to(resid_dt)
        y = torch.empty(T, N, dtype=out_dt, device="cuda")
        pick = S.sarathi_linear_plan(S.BF16, kind, T, N, K, scratch_bytes)
        splits = sorted({1, pick[2]}) if kind in (S.LINEAR_RESID, S.LINEAR_RESID_F32IN) else [1]
        if K % 64 != 0:
            # no tile choice for a K off the 64-wide k-tiles: the op's one kernel, as the planner runs it
            run = lambda: S.sarathi_linear(S.BF16, kind, T, N, K, x.data_ptr(), w.data_ptr(), resid.data_ptr(),
                                           y.data_ptr(), scratch.data_ptr(), scratch_bytes)
            for _ in range(3):
                run()
            ms = _time(run, iters)
            out.append({"op": name, "T": T, "N": N, "K": K, "bm": pick[0], "bn": pick[1], "n_split": pick[2],
                        "us": ms * 1e3, "tflops": 2.0 * T * w_rows * K / (ms * 1e-3) / 1e12, "picked": True})
            del x, w, resid, y
            continue
        for tile in range(S.sarathi_linear_tile_count()):
            bm, bn = S.sarathi_linear_tile_shape(tile)
            if bm == 64 and T > 64:
                continue
            for ns in splits:
                run = lambda: S.sarathi_linear_tiled(kind, T, N, K, x.data_ptr(), w.data_ptr(), resid.data_ptr(),
                                                     y.data_ptr(), scratch.data_ptr(), scratch_bytes, tile, ns)
                for _ in range(3):
                    run()
                ms = _time(run, iters)
                out.append({"op": name, "T": T, "N": N, "K": K, "bm": bm, "bn": bn, "n_split": ns, "us": ms * 1e3,
                            "tflops": 2.0 * T * w_rows * K / (ms * 1e-3) / 1e12,
                            "picked": (bm, bn, ns) == tuple(pick)})
        del x, w, resid, y
    return out


def tile_sweep_markdown(workload: str, rows: List[dict]) -> str:
    lines = [f"## Linear-op tile sweep: {workload} (T = {rows[0]['T']} rows)\n",
             "Each op alone through `sarathi_linear_tiled` (split-K reductions included), mean of 20 calls after "
             "3 warm-ups; weights re-read every call (a 256 MB memory-side cache can hold one "
             "op's weights between calls, so these times can be below the in-layer ones); preproj without its "
             "RoPE + KV-append epilogue.  * = the planner's pick.\n",
             "| op | N x K | tile (BM x BN) | K-splits | us | TFLOP/s | |", "|---|---|---|---|---|---|---|"]
    for e in rows:
        mark = "*" if e["picked"] else ""
        lines.append(f"| {e['op']} | {e['N']} x {e['K']} | {e['bm']} x {e['bn']} | {e['n_split']} | {e['us']:.1f} | "
                     f"{e['tflops']:.0f} | {mark} |")
    return "\n".join(lines) + "\n"


def main(argv: Optional[Sequence[str]] = None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", default="llama13b", choices=["llama13b", "tiny"])
    ap.add_argument("--json", default=None)
    ap.add_argument("--md", default=None)
    ap.add_argument("--quick", action="store_true", help="a few points of each sweep")
    ap.add_argument("--table2-only", action="store_true", help="only the whole-model per-token table")
    ap.add_argument("--no-table2", action="store_true", help="skip the whole-model per-token table")
    ap.add_argument("--tile-sweep", nargs="+", default=None, metavar="WORKLOAD",
                    help="only the linear-op tile sweep of these workloads (names in workloads.WORKLOADS)")
    args = ap.parse_args(argv)

    import torch

    import workloads as wl

    assert torch.cuda.is_available(), "the ablation runs on a GPU"
    if args.tile_sweep:
        cmd = "python -m paper_2308_16369_amd.ablation " + " ".join(argv if argv is not None else sys.argv[1:])
        res = {"command": cmd, "tile_sweep": {}}
        md = [f"# Linear-op tile sweeps\n\nCommand: `{cmd}`\n"]
        for name in args.tile_sweep:
            w = wl.WORKLOADS[name]
            T = w.batch.chunk_len + w.batch.n_decodes
            rows = tile_sweep(w.shape, T)
            res["tile_sweep"][name] = rows
            md.append(tile_sweep_markdown(name, rows))
            print(f"# {name}: {len(rows)} points", file=sys.stderr, flush=True)
        if args.json:
            with open(args.json, "w") as f:
                json.dump(res, f, indent=1)
        if args.md:
            with open(args.md, "w") as f:
                f.write("\n".join(md))
        return 0
    if args.workload == "llama13b":
        shape = wl.LLAMA13B_LAYER.shape
        prompts = [1024, 2048] if args.quick else [1024, 2048, 3072]
        chunks = [64, 128, 256, 512]
        lengths = [128, 129, 256, 257] if args.quick else tile_lengths(32, 512, 32, [64, 96, 128, 160])
        pig_chunks = [128, 256] if args.quick else [64, 128, 192, 256, 320, 384, 512]
        pig_dec = [32, 64] if args.quick else [16, 32, 63, 64, 96, 128]
        ctx, offset = 1024, 1024
    else:
        shape = wl.with_dtype(wl.TINY, "bf16").shape
        prompts, chunks = [256], [64, 128]
        lengths = [64, 65, 128]
        pig_chunks, pig_dec = [64], [4]
        ctx, offset = 100, 64
    max_seq = max(max(prompts), ctx + 2, offset + max(pig_chunks))
    n_slots = 1 + max(pig_dec)
    max_tokens = max(max(prompts), max(lengths), max(pig_chunks) + max(pig_dec))
    t0 = time.time()
    r = LayerRunner(shape, n_slots, max_seq, max_tokens, max(pig_dec))
    log = lambda m: print(f"# {m} ({time.time() - t0:.1f}s)", file=sys.stderr, flush=True)
    log("inputs on the device")
    res = {"workload": f"{args.workload}-layer-{shape.dtype}", "command":
           "python -m paper_2308_16369_amd.ablation " + " ".join(argv if argv is not None else sys.argv[1:])}
    if args.table2_only:
        del r
        torch.cuda.empty_cache()
        res["table2"] = table2(shape, n_layers=40 if args.workload == "llama13b" else 2)
        log("table 2 done")
        if args.json:
            with open(args.json, "w") as f:
                json.dump(res, f, indent=1)
        if args.md:
            with open(args.md, "w") as f:
                f.write(f"# Per-token prefill and decode time: {res['workload']}\n\nCommand: `{res['command']}`\n\n"
                        + table2_markdown(res["table2"]))
        print(json.dumps(res["table2"]["per_token_ms"]))
        return 0
    res["tile_quantization"] = tile_quantization(r, lengths)
    log("tile quantization done")
    res["chunking_overhead"] = chunking_overhead(r, prompts, chunks)
    log("chunking overhead done")
    res["piggyback_ctx"], res["piggyback_offset"] = ctx, offset
    res["piggyback"] = piggyback(r, pig_chunks, pig_dec, ctx, offset)
    log("piggyback done")
    if not args.no_table2:
        del r
        torch.cuda.empty_cache()
        res["table2"] = table2(shape, n_layers=40 if args.workload == "llama13b" else 2)
        log("table 2 done")
    if args.json:
        with open(args.json, "w") as f:
            json.dump(res, f, indent=1)
    if args.md:
        with open(args.md, "w") as f:
            f.write(to_markdown(res))
    print(json.dumps({"workload": res["workload"], "points": {k: len(v) for k, v in res.items()
                                                             if isinstance(v, list)}}))
    return 0


if __name__ == "__main__":
    sys.exit(main())
