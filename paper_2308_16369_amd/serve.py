"""End-to-end serving loop: the host scheduler (include/sarathi_sched.h)
driving sarathi_model_step, and the throughput study of Sec. 5.1.

Each request is a prompt of P tokens followed by D decode iterations.  There
is no embedding, LM head or sampling: a row's input hidden state stands in
for its token.  In timing mode every iteration reads the same synthetic
input rows; in recording mode (used by the parity tests) each (request,
position) has its own input row and the final hidden state of every token is
kept, so the outputs can be compared across policies and with a one-shot
causal forward of each request.

Throughput = (prompt tokens + decode tokens) / wall time of the GPU work,
measured with events on the launch stream around the whole schedule; the
scheduler runs ahead of the GPU (its decisions never wait for model
outputs).  Decode-maximal batching (chunk C, batch B) is compared with the
prefill-only / decode-only baseline on the same requests; Sec. 5.1.3 puts
the peak gain at P:D = C / (B - 1).

Command line (one GPU):
    python -m paper_2308_16369_amd.serve --json out.json --md out.md
"""
from __future__ import annotations

import argparse
import json
import sys
import time
from typing import List, Optional, Sequence, Tuple

from . import accounting
from . import sarathi as S

POLICY_NAMES = {S.POLICY_DECODE_MAXIMAL: "decode-maximal", S.POLICY_PREFILL_DECODE: "prefill/decode",
                S.POLICY_MIXED: "mixed"}


class ServeModel:
    """L layers of weights, a KV cache of n_slots x max_seq_len positions and
    a workspace for max_tokens rows, all on the current device.  Weights come
    from host arrays (``weights``: list of per-layer dicts) or are drawn on
    the device (0.02 * N(0,1); gains 1 + 0.02 * N(0,1))."""

    def __init__(self, shape, n_layers: int, n_slots: int, max_seq_len: int, max_tokens: int,
                 weights: Optional[List[dict]] = None, seed: int = 0, max_chunks: int = 1):
        import numpy as np
        import torch

        self.torch, self.shape, self.L = torch, shape, n_layers
        self.tdt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        self.cfg = S.make_cfg(hidden=shape.hidden, n_heads=shape.n_heads, head_dim=shape.head_dim, ffn=shape.ffn,
                              n_layers=n_layers, norm=S.NORM_RMS if shape.norm == "rms" else S.NORM_LAYER,
                              act=S.ACT_SWIGLU if shape.act == "swiglu" else S.ACT_GELU, rope=int(shape.rope),
                              rope_base=shape.rope_base, eps=shape.eps,
                              dtype=S.BF16 if shape.dtype == "bf16" else S.F32)
        H, nh, d, F = shape.hidden, shape.n_heads, shape.head_dim, shape.ffn
        dims = {"w_qkv": (3 * nh * d, H), "w_o": (H, nh * d), "w_up": (shape.up_rows, H), "w_down": (H, F),
                "norm1_g": (H,), "norm2_g": (H,)}
        if shape.norm == "layer":
            dims.update(norm1_b=(H,), norm2_b=(H,))
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        self.w = []
        for layer in range(n_layers):
            lw = {}
            for k, dim in dims.items():
                if weights is not None:
                    a = np.ascontiguousarray(weights[layer][k], np.float32)
                    lw[k] = torch.from_numpy(a).to(self.tdt).cuda()
                else:
                    mean, std = (1.0, 0.02) if k.endswith("_g") else (0.0, 0.02)
                    lw[k] = torch.empty(dim, dtype=self.tdt, device="cuda").normal_(mean, std, generator=g)
            self.w.append(lw)
        self.wabi = (S.sarathi_layer_weights * n_layers)(
            *[S.make_weights({k: t.data_ptr() for k, t in lw.items()}) for lw in self.w])
        self.kv_t = torch.zeros((n_layers, n_slots, 2, nh, max_seq_len, d), dtype=self.tdt, device="cuda")
        self.kv = S.sarathi_kv_alloc(self.cfg, n_slots, max_seq_len, self.kv_t.data_ptr(),
                                     self.kv_t.numel() * self.kv_t.element_size())
        self.n_slots, self.max_seq_len, self.max_tokens, self.max_chunks = n_slots, max_seq_len, max_tokens, max_chunks
        self.ws_bytes = S.sarathi_mixed_workspace_bytes(self.cfg, max_tokens, max_chunks, max_seq_len)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device="cuda")
        self.x = torch.empty((max_tokens, H), dtype=self.tdt, device="cuda").normal_(0.0, 1.0, generator=g)
        self.y = torch.empty_like(self.x)
        self.stream = torch.cuda.current_stream()

    def step(self, bb, x, y):
        """One model iteration over a sarathi_mixed_batch (any number of chunks)."""
        lib = S.lib()
        import ctypes as ct
        rc = lib.sarathi_mixed_model_step(ct.byref(self.cfg), self.wabi, self.kv.handle, ct.byref(bb),
                                          ct.c_void_p(x.data_ptr()), ct.c_void_p(y.data_ptr()),
                                          ct.c_void_p(self.ws.data_ptr()), self.ws_bytes,
                                          ct.c_void_p(self.stream.cuda_stream))
        S._check(rc)


def run_schedule(m: ServeModel, policy: int, requests: Sequence[Tuple[int, int]], max_batch: int, chunk: int,
                 inputs=None, outputs=None, max_chunks: int = 0, max_tokens: int = 0) -> dict:
    """Serve ``requests`` [(P, D)] under ``policy``; returns timing and
    scheduler counts.  ``inputs`` / ``outputs``: optional device tensors
    [n_requests, P + D, H]; row (r, pos) is the input / final hidden state of
    request r's token at position pos."""
    torch = m.torch
    if max_batch > m.n_slots:
        raise ValueError("max_batch exceeds the KV slots of the model")
    sched = S.Scheduler(policy, max_batch=max_batch, n_slots=m.n_slots, max_seq_len=m.max_seq_len, chunk=chunk,
                        max_chunks=max_chunks, max_tokens=max_tokens)
    for p, d in requests:
        sched.submit(p, d)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(m.stream)
    iters = 0
    while True:
        st = sched.next()
        if st.n_tokens == 0:
            break
        if st.n_tokens > m.max_tokens or st.n_chunks > m.max_chunks:
            raise ValueError(f"an iteration of {st.n_tokens} rows in {st.n_chunks} chunks exceeds the workspace "
                             f"({m.max_tokens} rows, {m.max_chunks} chunks)")
        bb, keep = st.mixed_batch()
        x, y = m.x[:st.n_tokens], m.y[:st.n_tokens]
        if inputs is not None:
            rows = _rows(st)
            x = inputs[rows[0], rows[1]]
        m.step(bb, x, y)
        if outputs is not None:
            rows = _rows(st)
            outputs[rows[0], rows[1]] = y
        sched.commit()
        iters += 1
    e1.record(m.stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1)
    stats = sched.stats()
    sched.close()
    tokens = stats["prefill_tokens"] + stats["decode_tokens"]
    return {"policy": POLICY_NAMES[policy], "iterations": iters, "ms": round(ms, 3), "host_wall_ms": round(wall * 1e3, 3),
            "tokens": tokens, "tokens_per_s": round(tokens / (ms * 1e-3), 1),
            "hybrid_iterations": stats["hybrid_iterations"],
            "prefill_only_iterations": stats["prefill_only_iterations"],
            "decode_only_iterations": stats["decode_only_iterations"]}


def _rows(st):
    """(request index, position) of every row of an iteration, as index lists."""
    req, pos = [], []
    for r, o, n in zip(st.chunk_request, st.chunk_offset, st.chunk_len):
        req += [r] * n
        pos += list(range(o, o + n))
    req += list(st.decode_request)
    pos += list(st.decode_ctx)
    return req, pos


def pd_split(seq_len: int, ratio: float) -> Tuple[int, int]:
    """(P, D) with P + D = seq_len and P / D as close to ``ratio`` as integers allow (D >= 1)."""
    d = max(1, round(seq_len / (ratio + 1.0)))
    return seq_len - d, d


def sweep(m: ServeModel, seq_len: int, ratios: Sequence[float], chunks: Sequence[int], max_batch: int,
          n_requests: int, log=lambda s: None, mixed: bool = False) -> List[dict]:
    """Decode-maximal (each chunk size) against the prefill/decode baseline
    for each P:D ratio; with ``mixed``, also Orca-style mixed batching (whole
    prompts of up to m.max_chunks requests plus every decode, within
    m.max_tokens rows)."""
    out = []
    for ratio in ratios:
        P, D = pd_split(seq_len, ratio)
        reqs = [(P, D)] * n_requests
        base = run_schedule(m, S.POLICY_PREFILL_DECODE, reqs, max_batch, 0)
        mix = None
        if mixed:
            mix = run_schedule(m, S.POLICY_MIXED, reqs, max_batch, 0, max_chunks=m.max_chunks,
                               max_tokens=m.max_tokens - max_batch)
        for C in chunks:
            dm = run_schedule(m, S.POLICY_DECODE_MAXIMAL, reqs, max_batch, C)
            out.append({"seq_len": seq_len, "P": P, "D": D, "pd": round(P / D, 2), "B": max_batch, "C": C,
                        "n_requests": n_requests, "peak_pd": round(C / max(1, max_batch - 1), 2),
                        "decode_maximal": dm, "baseline": base, "mixed": mix,
                        "speedup": round(dm["tokens_per_s"] / base["tokens_per_s"], 3),
                        "mixed_speedup": round(mix["tokens_per_s"] / base["tokens_per_s"], 3) if mix else None})
            log(f"seq {seq_len} P:D {P}:{D} C {C}: {dm['tokens_per_s']:.0f} vs {base['tokens_per_s']:.0f} tok/s "
                f"({out[-1]['speedup']}x)")
    return out


def to_markdown(res: dict) -> str:
    L = [f"# End-to-end throughput vs P:D: {res['workload']}", "", f"Command: `{res['command']}`", "",
         res["note"], ""]
    eq = res.get("batch_equation")
    if eq:
        L += [f"B from Sec. 4.3.1: floor((M_G - headroom - M_S) / (L m_kv)) = floor(({eq['mem_gpu'] / 1e9:.1f} - "
              f"{eq['headroom'] / 1e9:.1f} - {eq['mem_params'] / 1e9:.2f} GB) / ({eq['seq_len']} x "
              f"{eq['kv_bytes_per_token'] / 1e3:.1f} KB)) = {eq['B']}.", ""]
    L += [
         "| seq | P | D | P:D | B | C | C/(B-1) | decode-maximal tok/s | baseline tok/s | speedup | "
         "mixed tok/s (speedup) | hybrid / prefill-only / decode-only iterations |",
         "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for e in res["sweep"]:
        dm, b, mx = e["decode_maximal"], e["baseline"], e.get("mixed")
        mixed = f"{mx['tokens_per_s']:.0f} ({e['mixed_speedup']:.3f})" if mx else "-"
        L.append(f"| {e['seq_len']} | {e['P']} | {e['D']} | {e['pd']} | {e['B']} | {e['C']} | {e['peak_pd']} | "
                 f"{dm['tokens_per_s']:.0f} | {b['tokens_per_s']:.0f} | {e['speedup']:.3f} | {mixed} | "
                 f"{dm['hybrid_iterations']} / {dm['prefill_only_iterations']} / {dm['decode_only_iterations']} |")
    return "\n".join(L) + "\n"


def equation_batch(shape, n_layers: int, seq_len: int, mem_gpu: int, headroom: int = 0) -> dict:
    """The decode batch of Sec. 4.3.1, B = floor((M_G - M_S) / (L * m_kv)):
    M_G the device memory (less ``headroom`` for activations and the
    workspace), M_S the bytes of the model's weights, L the sequence length
    and m_kv the K and V bytes of one token over all layers."""
    es = 2 if shape.dtype == "bf16" else 4
    H, nh, d, F = shape.hidden, shape.n_heads, shape.head_dim, shape.ffn
    per_layer = (3 * nh * d * H + H * nh * d + shape.up_rows * H + H * F + 2 * H) * es
    m_s = n_layers * per_layer
    m_kv = n_layers * 2 * nh * d * es
    b = accounting.max_decode_batch(mem_gpu - headroom, m_s, seq_len, m_kv)
    return {"B": b, "mem_gpu": mem_gpu, "headroom": headroom, "mem_params": m_s, "kv_bytes_per_token": m_kv,
            "seq_len": seq_len}


def main(argv: Optional[Sequence[str]] = None) -> int:
    ap = argparse.ArgumentParser(description="decode-maximal batching vs prefill/decode batches, end to end")
    ap.add_argument("--layers", type=int, default=40)
    ap.add_argument("--batch", type=int, default=0,
                    help="decode batch B (default: the Sec. 4.3.1 equation over the device memory)")
    ap.add_argument("--mem-gb", type=float, default=0.0,
                    help="device memory M_G for the B equation, GB (default: the device's total)")
    ap.add_argument("--max-batch", type=int, default=0, help="cap on the equation's B (0: none)")
    ap.add_argument("--seq", type=int, nargs="+", default=[1024])
    ap.add_argument("--chunks", type=int, nargs="+", default=[128, 256, 512])
    ap.add_argument("--ratios", type=float, nargs="+", default=[1, 2, 4, 8, 14, 28, 50, 100])
    ap.add_argument("--requests", type=int, default=0, help="requests per run (default 2 x batch)")
    ap.add_argument("--mixed", action="store_true", help="also run Orca-style mixed batching")
    ap.add_argument("--mixed-chunks", type=int, default=4, help="prompts per mixed iteration")
    ap.add_argument("--json", default=None)
    ap.add_argument("--md", default=None)
    args = ap.parse_args(argv)

    import torch

    import workloads as wl

    assert torch.cuda.is_available(), "the serving study runs on a GPU"
    shape = wl.LLAMA13B_LAYER.shape
    eq = None
    if args.batch <= 0:
        mem = int(args.mem_gb * 1e9) if args.mem_gb > 0 else torch.cuda.get_device_properties(0).total_memory
        eq = equation_batch(shape, args.layers, max(args.seq), mem, headroom=8 << 30)
        args.batch = eq["B"] if args.max_batch <= 0 else min(eq["B"], args.max_batch)
        print(f"# B = {args.batch} from Sec. 4.3.1: floor(({eq['mem_gpu'] / 1e9:.1f} GB - {eq['headroom'] / 1e9:.1f} GB "
              f"headroom - {eq['mem_params'] / 1e9:.2f} GB weights) / ({eq['seq_len']} x "
              f"{eq['kv_bytes_per_token'] / 1e3:.1f} KB)) = {eq['B']}"
              + (f", capped at {args.max_batch}" if args.max_batch > 0 and args.max_batch < eq["B"] else ""),
              file=sys.stderr, flush=True)
    n_req = args.requests or 2 * args.batch
    max_seq = max(args.seq)
    max_tokens = max(max(args.seq), max(args.chunks) + args.batch)
    max_chunks = 1
    if args.mixed:
        max_chunks = args.mixed_chunks
        max_tokens = max(max_tokens, args.mixed_chunks * max(args.seq) + args.batch)
    t0 = time.time()
    log = lambda s: print(f"# {s} ({time.time() - t0:.1f}s)", file=sys.stderr, flush=True)
    m = ServeModel(shape, args.layers, args.batch, max_seq, max_tokens, max_chunks=max_chunks)
    log(f"{args.layers}-layer model on the device")
    run_schedule(m, S.POLICY_DECODE_MAXIMAL, [(64, 4)] * 2, 2, 32)     # warm-up
    res = {"workload": f"llama13b-{args.layers}layers-bf16", "command":
           "python -m paper_2308_16369_amd.serve " + " ".join(argv if argv is not None else sys.argv[1:]),
           "note": f"{n_req} requests of equal P and D per run, B = {args.batch} resident at once; baseline = "
                   f"whole-prompt prefill-only iterations then decode-only iterations (Sec. 5.1); synthetic "
                   f"hidden states stand in for tokens.",
           "batch_equation": eq, "sweep": []}
    for seq in args.seq:
        res["sweep"] += sweep(m, seq, args.ratios, args.chunks, args.batch, n_req, log, mixed=args.mixed)
    if args.json:
        with open(args.json, "w") as f:
            json.dump(res, f, indent=1)
    if args.md:
        with open(args.md, "w") as f:
            f.write(to_markdown(res))
    best = max(res["sweep"], key=lambda e: e["speedup"])
    print(json.dumps({"workload": res["workload"], "points": len(res["sweep"]), "best_speedup": best["speedup"],
                      "best_at": {k: best[k] for k in ("seq_len", "P", "D", "C", "B")}}))
    return 0


if __name__ == "__main__":
    sys.exit(main())
