"""Host-side checks of the benchmark's bookkeeping (no GPU): the algorithmic
work per stage against closed forms, the overhead accounting, the one-GPU
guard and the oracle timing helpers."""
import os
import subprocess
import sys

import numpy as np

import bench
import oracle
import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_stage_work_matches_closed_forms_for_the_llama13b_layer():
    w = wl.WORKLOADS["llama13b-layer-bf16-c256-b64"]
    b, s = wl.draw_batch(np.random.Generator(np.random.PCG64(w.seed)), w.batch), w.shape   # generate()'s first draw
    T, H, F, QD = b.n_tokens, s.hidden, s.ffn, s.n_heads * s.head_dim
    work = bench.stage_work(s, b)
    lin = ("preproj", "postproj", "ffn_ln1", "ffn_ln2")
    flops = sum(work[k][0] for k in lin)
    assert flops == 2 * T * H * (3 * QD + QD + 2 * F) + 2 * T * F * H
    assert abs(flops / 1e9 - 203.0) < 0.05                      # 320 rows of the LLaMA-13B layer
    weight_bytes = 2 * (3 * QD * H + H * QD + 2 * F * H + H * F)
    assert abs(weight_bytes / 1e6 - 634.4) < 0.05
    act = sum(work[k][1] for k in lin) - weight_bytes
    assert 0 < act < 0.1 * weight_bytes                          # activations are a small share at 320 rows
    keys = int(np.sum(b.decode_ctx.astype(np.int64) + 1))
    dec_flops, dec_bytes = work["decode_attention"]
    assert dec_flops == 4.0 * keys * QD
    assert dec_bytes >= keys * 2 * QD * 2                         # every cached K and V byte once
    pairs = b.chunk_len * b.chunk_offset + b.chunk_len * (b.chunk_len + 1) // 2
    assert work["chunk_attention"][0] == 4.0 * pairs * QD         # masked pairs not counted


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_oracle_cpu_baseline_fields():
    w = wl.TINY
    inst = wl.generate(w)
    b = inst.batch
    ob = oracle.OracleBatch(b.prefill_slot, b.chunk_offset, b.chunk_len, list(b.decode_slots), list(b.decode_ctx))
    cpu = bench.oracle_cpu_baseline(oracle, w.shape, inst.weights[0], inst.kv[0], ob, inst.x, b.n_tokens)
    assert cpu["kind"] == "oracle" and cpu["unit"] == "tokens/s"
    assert cpu["value"] > 0 and cpu["cores"] >= 1
    assert cpu["one_core_value"] is not None and cpu["one_core_value"] > 0
    assert "median of" in cpu["sample"]


def test_stage_overhead_is_separate_from_method_bytes():
    w = wl.WORKLOADS["llama13b-layer-bf16-c256-b64"]
    b, s = wl.draw_batch(np.random.Generator(np.random.PCG64(w.seed)), w.batch), w.shape
    T, H, QD = b.n_tokens, s.hidden, s.n_heads * s.head_dim
    work = bench.stage_work(s, b)
    assert work["attention_combine"] == (0.0, 0.0)             # the combine is not the method's work
    plan = {"chunk_items": 3, "decode_items": 100, "partial_rows_written": 100 + 512, "partial_rows_read": 612,
            "combine_rows": T}
    over = bench.stage_overhead(s, b, plan, {"postproj": 3, "ffn_ln2": 1})
    assert over["postproj"] == 2.0 * 3 * T * H * 4               # fp32 partials written and read back
    assert over["ffn_ln2"] == 0.0                                 # no split, no partials
    part_row = s.n_heads * (s.head_dim + 4) * 4
    assert over["decode_attention"] == 100 * part_row
    assert over["chunk_attention"] == 512 * part_row
    assert over["attention_combine"] == 612 * part_row + T * QD * 2
    for k in ("preproj", "ffn_ln1", "norm_1", "norm_2"):
        assert over[k] == 0.0


def test_stack_oracle_baseline_is_labelled_extrapolated():
    w = wl.TINY
    b = wl.draw_batch(np.random.Generator(np.random.PCG64(w.seed)), w.batch)
    r = bench.oracle_stack_baseline(oracle, w.shape, b, 40, budget_s=0.5)
    assert r["extrapolated"] is True and r["kind"] == "oracle"
    assert r["value"] > 0 and "times 40 layers" in r["sample"]
    assert abs(r["ms_per_step"] - b.n_tokens / r["value"] * 1e3) < 0.01 * r["ms_per_step"] + 1
