"""Pipeline-parallel bubble study on a cost model measured on this GPU (Sec. 3.2,
Sec. 5.3).

With pipeline parallelism each stage runs a range of layers and micro-batches
flow through the stages; an iteration of one micro-batch cannot start before
its previous iteration has left the last stage (the next tokens depend on
it).  When consecutive micro-batches need different amounts of compute -- a
long prefill next to a few decodes -- later stages wait: pipeline bubbles.
Decode-maximal batching gives every iteration one chunk of C tokens plus
decodes, so micro-batches cost about the same and the bubbles shrink.

The paper measures this in a simulator driven by per-operation profiles.  Here:

* ``measure_cost_model`` times one decoder layer of the given shape through
  the C-ABI (stage events) over grids of row counts, chunk offsets and decode
  context lengths, and fits the per-layer time of any batch as
      linear(T) + sum over chunks of (a*pairs + b*keys + c) + (d*keys + e*B + f)
  with linear(T) interpolated from the measured table (so tile quantization
  is kept), and reports its error on random held-out batches;
* ``simulate`` replays iteration-level scheduling of M micro-batches, each
  with its own requests and scheduler (the library's host scheduler:
  decode-maximal, or Orca-style mixed batching of whole prompts), through S
  stages of L/S layers, and returns each request's bubble time (the idle
  time of every stage right before each of its micro-batch's iterations,
  summed) and the makespan.

Command line:
    python -m paper_2308_16369_amd.pipeline_sim measure --out cost.json   (GPU)
    python -m paper_2308_16369_amd.pipeline_sim simulate --cost cost.json --md out.md
"""
from __future__ import annotations

import argparse
import bisect
import json
import sys
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import sarathi as S

NON_ATTN = ("norm_1", "preproj", "rope_kv_append", "attention_combine", "postproj", "norm_2", "ffn_ln1", "ffn_ln2")


# ============================================================================ cost model

@dataclass
class CostModel:
    """Per-layer milliseconds of a batch (see the module docstring)."""
    rows: List[int]                 # T grid of the linear-op table (ascending)
    linear_ms: List[float]          # non-attention stages at each T
    pre: Tuple[float, float, float]   # chunk attention: a (per pair), b (per key read), c (per chunk)
    dec: Tuple[float, float, float]   # decode attention: d (per key), e (per decode), f (per batch with decodes)
    shape: str = ""
    check: Optional[dict] = None

    def linear(self, T: int) -> float:
        r, v = self.rows, self.linear_ms
        if T <= r[0]:
            return v[0] * T / r[0] if T < r[0] else v[0]
        if T >= r[-1]:
            return v[-1] * T / r[-1]
        i = bisect.bisect_right(r, T)
        t = (T - r[i - 1]) / (r[i] - r[i - 1])
        return v[i - 1] + t * (v[i] - v[i - 1])

    def chunk_attn(self, offset: int, length: int) -> float:
        a, b, c = self.pre
        pairs = length * offset + length * (length + 1) / 2
        return a * pairs + b * (offset + length) + c

    def decode_attn(self, ctx: Sequence[int]) -> float:
        if len(ctx) == 0:
            return 0.0
        d, e, f = self.dec
        return d * float(np.sum(np.asarray(ctx, np.float64) + 1)) + e * len(ctx) + f

    def layer_ms(self, chunks: Sequence[Tuple[int, int]], ctx: Sequence[int]) -> float:
        """chunks: [(offset, length)]; ctx: decode context lengths."""
        T = sum(n for _, n in chunks) + len(ctx)
        if T == 0:
            return 0.0
        return self.linear(T) + sum(self.chunk_attn(o, n) for o, n in chunks) + self.decode_attn(ctx)

    def to_json(self) -> dict:
        return {"shape": self.shape, "rows": self.rows, "linear_ms": self.linear_ms, "pre": list(self.pre),
                "dec": list(self.dec), "check": self.check}

    @staticmethod
    def from_json(d: dict) -> "CostModel":
        return CostModel(rows=list(d["rows"]), linear_ms=list(d["linear_ms"]), pre=tuple(d["pre"]),
                         dec=tuple(d["dec"]), shape=d.get("shape", ""), check=d.get("check"))


def fit_linear_terms(X: np.ndarray, y: np.ndarray) -> np.ndarray:
    """Least-squares coefficients of y ~ X, clipped at zero (times cannot
    fall as work grows)."""
    coef, *_ = np.linalg.lstsq(np.asarray(X, np.float64), np.asarray(y, np.float64), rcond=None)
    return np.maximum(coef, 0.0)


def measure_cost_model(shape, max_seq: int = 4096, max_decodes: int = 32, log=lambda s: None) -> CostModel:
    """Time one layer of ``shape`` on the current GPU and fit a CostModel."""
    from .ablation import LayerRunner, Batch

    n_slots = max_decodes + 4
    grid = [1, 2, 4, 8, 16, 24, 27, 32, 48, 64, 96, 128, 160, 192, 256, 283, 320, 384, 512, 768, 1024, 1536,
            2048, 3072, 4096]
    grid = [t for t in grid if t <= max_seq]
    r = LayerRunner(shape, n_slots, max_seq, max(grid) + max_decodes, max_decodes, max_chunks=4)

    def stages(calls, iters=4):
        return r.stages(calls, iters)

    for T in grid:   # one untimed pass first: the first launch of each kernel instance is not its cost
        r.call(Batch(0, 0, T, [], []))()
    lin = []
    for T in grid:   # prefill-only at offset 0: non-attention stages (median of three)
        reps = [sum(stages([r.call(Batch(0, 0, T, [], []))])[k] for k in NON_ATTN) for _ in range(3)]
        lin.append(float(np.median(reps)))
    log("linear table measured")
    Xp, yp = [], []
    for off in sorted({0, 256, 1024, 2048, max(0, max_seq - 512)}):
        for n in [16, 64, 256, 512]:
            if off + n > max_seq:
                continue
            st = stages([r.call(Batch(0, off, n, [], []))])
            Xp.append([n * off + n * (n + 1) / 2, off + n, 1.0])
            yp.append(st["chunk_attention"])
    pre = fit_linear_terms(np.array(Xp), np.array(yp))
    log("chunk attention fitted")
    Xd, yd = [], []
    rng = np.random.default_rng(0)
    for B in sorted({b for b in (1, 4, 8, 16, max_decodes) if b <= max_decodes}):
        for hi in sorted({h for h in (256, 1024, 2048, max_seq - 1) if h <= max_seq - 1}):
            ctx = rng.integers(max(0, hi // 4), hi, size=B)
            st = stages([r.call(Batch(-1, 0, 0, list(range(1, B + 1)), [int(c) for c in ctx]))])
            Xd.append([float(np.sum(ctx + 1)), B, 1.0])
            yd.append(st["decode_attention"])
    dec = fit_linear_terms(np.array(Xd), np.array(yd))
    log("decode attention fitted")
    cm = CostModel(rows=grid, linear_ms=[float(v) for v in lin], pre=tuple(float(v) for v in pre),
                   dec=tuple(float(v) for v in dec))
    # held-out check: random hybrid and mixed batches, whole-layer time (no stage events)
    errs = []
    for _ in range(12):
        k = int(rng.integers(0, 3))
        chunks, slot = [], 0
        for _c in range(k):
            n = int(rng.choice([v for v in (64, 128, 256, 300, 512) if v < max_seq // 2]))
            off = int(rng.integers(0, max_seq - n))
            chunks.append((slot, off, n))
            slot += 1
        B = int(rng.integers(0 if k else 1, max_decodes + 1))
        ctx = [int(c) for c in rng.integers(16, max_seq - 1, size=B)]
        slots = list(range(slot, slot + B))
        ms = r.time([r.call_mixed(chunks, slots, ctx)], iters=10)
        pred = cm.layer_ms([(o, n) for _, o, n in chunks], ctx)
        errs.append(abs(pred - ms) / ms)
    cm.check = {"held_out_batches": len(errs), "median_rel_err": float(np.median(errs)),
                "max_rel_err": float(np.max(errs))}
    log(f"cost model error on held-out batches: median {np.median(errs):.3f}, max {np.max(errs):.3f}")
    return cm


# ============================================================================ simulator

def zipf_lengths(n: int, lo: int, hi: int, theta: float, seed: int = 0) -> np.ndarray:
    """n sequence lengths in [lo, hi] with P(lo + k) proportional to (k + 1)^-theta."""
    k = np.arange(hi - lo + 1, dtype=np.float64)
    p = (k + 1.0) ** (-theta)
    p /= p.sum()
    rng = np.random.default_rng(seed)
    return lo + rng.choice(len(k), size=n, p=p)


def pd_requests(lengths: Sequence[int], pd: float) -> List[Tuple[int, int]]:
    """Split each sequence length into (P, D) with P / D = pd (D >= 1)."""
    out = []
    for L in lengths:
        d = max(1, int(round(L / (pd + 1.0))))
        out.append((int(L) - d, d))
    return out


@dataclass
class SimResult:
    policy: str
    makespan_ms: float
    bubble_ms_per_request: np.ndarray
    stage_busy_frac: float
    iterations: int

    def summary(self) -> dict:
        b = self.bubble_ms_per_request
        return {"policy": self.policy, "makespan_ms": round(self.makespan_ms, 3),
                "bubble_ms_median": round(float(np.median(b)), 3), "bubble_ms_p90": round(float(np.percentile(b, 90)), 3),
                "bubble_ms_mean": round(float(np.mean(b)), 3), "stage_busy_frac": round(self.stage_busy_frac, 4),
                "iterations": self.iterations}


def simulate(requests: Sequence[Tuple[int, int]], policy: int, n_stages: int, n_layers: int,
             micro_batches: int, batch_per_mb: int, cost: CostModel, chunk: int = 256,
             max_chunks: int = 0, max_tokens: int = 0, send_ms: float = 0.0) -> SimResult:
    """Iteration-level pipeline schedule of ``micro_batches`` micro-batches
    through ``n_stages`` stages of n_layers / n_stages layers.

    Requests are handed out in order to whichever micro-batch has a free
    place when it forms its next iteration; each micro-batch runs the
    library's scheduler with ``policy`` (B = batch_per_mb).  Stage s starts a
    task when the task has left stage s-1 (plus ``send_ms``) and the stage is
    free; stage 0 starts micro-batch m's next iteration only after its
    previous one has left the last stage.  Tasks are served in arrival order."""
    if n_layers % n_stages:
        raise ValueError("n_layers must be a multiple of n_stages")
    lps = n_layers // n_stages
    max_seq = max(p + d for p, d in requests)
    scheds = [S.Scheduler(policy, max_batch=batch_per_mb, n_slots=batch_per_mb, max_seq_len=max_seq, chunk=chunk,
                          max_chunks=max_chunks or batch_per_mb, max_tokens=max_tokens or 1 << 30)
              for _ in range(micro_batches)]
    owner = [[] for _ in range(micro_batches)]   # per micro-batch: local request id -> global id
    queue = list(range(len(requests)))
    qi = 0
    bubble = np.zeros(len(requests))
    stage_free = [0.0] * n_stages
    stage_busy = [0.0] * n_stages
    stage_started = [False] * n_stages
    mb_ready = [0.0] * micro_batches            # when the micro-batch's previous iteration left the pipeline
    done = [False] * micro_batches
    iterations = 0
    end_time = 0.0
    while not all(done):
        # next task on stage 0: the micro-batch that can start earliest (ties: lowest index)
        order = sorted((max(mb_ready[m], stage_free[0]), m) for m in range(micro_batches) if not done[m])
        _, m = order[0]
        sch = scheds[m]
        st = sch.stats()
        while qi < len(queue) and st["resident"] + (st["submitted"] - st["admitted"]) < batch_per_mb:
            p, d = requests[queue[qi]]
            sch.submit(p, d)
            owner[m].append(queue[qi])
            qi += 1
            st = sch.stats()
        step = sch.next()
        if step.n_tokens == 0:
            done[m] = True
            continue
        ms = lps * cost.layer_ms(list(zip(step.chunk_offset, step.chunk_len)), step.decode_ctx)
        members = [owner[m][r] for r in set(step.chunk_request) | set(step.decode_request)]
        t = mb_ready[m]
        for s in range(n_stages):
            start = max(t, stage_free[s])
            if stage_started[s]:
                gap = start - stage_free[s]
                for g in members:
                    bubble[g] += gap
            stage_started[s] = True
            stage_free[s] = start + ms
            stage_busy[s] += ms
            t = stage_free[s] + (send_ms if s + 1 < n_stages else 0.0)
        mb_ready[m] = t
        end_time = max(end_time, t)
        sch.commit()
        iterations += 1
    for sch in scheds:
        sch.close()
    busy = sum(stage_busy) / (n_stages * end_time) if end_time > 0 else 0.0
    name = {S.POLICY_DECODE_MAXIMAL: f"decode-maximal C={chunk}", S.POLICY_MIXED: "mixed (Orca-style)",
            S.POLICY_PREFILL_DECODE: "prefill/decode"}[policy]
    return SimResult(policy=name, makespan_ms=end_time, bubble_ms_per_request=bubble, stage_busy_frac=busy,
                     iterations=iterations)


# ============================================================================ CLI

def _md(res: dict) -> str:
    L = [f"# Pipeline bubbles on a measured cost model: {res['shape']}", "", f"Commands: `{res['command']}`", "",
         res["note"], "", "Cost model check (whole-layer time vs prediction on held-out batches): "
         f"median error {res['cost_check']['median_rel_err']:.3f}, max {res['cost_check']['max_rel_err']:.3f}.", "",
         "| stages | micro-batches | B per micro-batch | policy | makespan s | bubble ms / request (median) | p90 | "
         "stage busy |", "|---|---|---|---|---|---|---|---|"]
    for e in res["runs"]:
        L.append(f"| {e['stages']} | {e['micro_batches']} | {e['B']} | {e['policy']} | {e['makespan_ms'] / 1e3:.2f} | "
                 f"{e['bubble_ms_median']:.1f} | {e['bubble_ms_p90']:.1f} | {e['stage_busy_frac']:.3f} |")
    for k, v in res.get("ratios", {}).items():
        L.append(f"\n{k}: {v}")
    return "\n".join(L) + "\n"


def main(argv: Optional[Sequence[str]] = None) -> int:
    ap = argparse.ArgumentParser(description="pipeline bubbles of decode-maximal vs mixed batching")
    sub = ap.add_subparsers(dest="cmd", required=True)
    mp = sub.add_parser("measure")
    mp.add_argument("--shape", default="gpt3", choices=["gpt3", "llama13b"])
    mp.add_argument("--out", required=True)
    sp = sub.add_parser("simulate")
    sp.add_argument("--cost", required=True)
    sp.add_argument("--requests", type=int, default=2000)
    sp.add_argument("--layers", type=int, default=96)
    sp.add_argument("--stages", type=int, default=8)
    sp.add_argument("--batch", type=int, default=27)
    sp.add_argument("--chunk", type=int, default=256)
    sp.add_argument("--pd", type=float, default=10.0)
    sp.add_argument("--mixed-tokens", type=int, default=4096, help="prompt rows per mixed iteration")
    sp.add_argument("--json", default=None)
    sp.add_argument("--md", default=None)
    args = ap.parse_args(argv)
    cmdline = "python -m paper_2308_16369_amd.pipeline_sim " + " ".join(argv if argv is not None else sys.argv[1:])

    if args.cmd == "measure":
        import workloads as wl
        shape = wl.GPT3_LAYER.shape if args.shape == "gpt3" else wl.LLAMA13B_LAYER.shape
        cm = measure_cost_model(shape, log=lambda s: print(f"# {s}", file=sys.stderr, flush=True))
        cm.shape = args.shape
        d = cm.to_json()
        d["command"] = cmdline
        with open(args.out, "w") as f:
            json.dump(d, f, indent=1)
        print(json.dumps({"shape": args.shape, "check": cm.check}))
        return 0

    cm_json = json.load(open(args.cost))
    cm = CostModel.from_json(cm_json)
    lengths = zipf_lengths(args.requests, 1024, 4096, 0.4, seed=0)
    reqs = pd_requests(lengths, args.pd)
    runs = []
    for policy in (S.POLICY_MIXED, S.POLICY_DECODE_MAXIMAL):
        r = simulate(reqs, policy, args.stages, args.layers, args.stages, args.batch, cm, chunk=args.chunk,
                     max_chunks=args.batch, max_tokens=args.mixed_tokens)
        e = r.summary()
        e.update(stages=args.stages, micro_batches=args.stages, B=args.batch)
        runs.append(e)
        print(f"# {e}", file=sys.stderr, flush=True)
    res = {"shape": cm.shape, "command": cmdline + f"  (cost model: {cm_json.get('command', '')})",
           "note": f"{args.requests} requests, sequence length Zipf(theta 0.4) over [1024, 4096], P:D = {args.pd}, "
                   f"{args.layers} layers in {args.stages} stages, {args.stages} micro-batches of B = {args.batch}, "
                   f"chunk {args.chunk}; mixed batching takes whole prompts up to {args.mixed_tokens} prompt rows "
                   f"per iteration; per-layer times from the measured cost model (one layer, unsharded, on one "
                   f"MI355X); stage-to-stage sends not modelled.",
           "cost_check": cm.check or {"median_rel_err": float("nan"), "max_rel_err": float("nan")}, "runs": runs}
    mx, dm = runs[0], runs[1]
    res["ratios"] = {"median bubble time, mixed / decode-maximal":
                     round(mx["bubble_ms_median"] / max(dm["bubble_ms_median"], 1e-9), 2),
                     "makespan, mixed / decode-maximal": round(mx["makespan_ms"] / dm["makespan_ms"], 3)}
    if args.json:
        with open(args.json, "w") as f:
            json.dump(res, f, indent=1)
    if args.md:
        with open(args.md, "w") as f:
            f.write(_md(res))
    print(json.dumps(res["ratios"]))
    return 0


if __name__ == "__main__":
    sys.exit(main())
