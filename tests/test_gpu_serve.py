"""End-to-end serving on the device: the host scheduler drives
sarathi_model_step over a small model, and the final hidden state of every
token is checked

  * against the oracle's one-shot causal forward of that request's whole
    sequence (prompt and decode inputs together, Sec. 4.2: chunking and
    piggybacking do not change the result), and
  * across policies: decode-maximal batching and the prefill-only /
    decode-only baseline give the same per-token outputs.
"""
import dataclasses

import numpy as np
import pytest

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

from gpu_harness import TOL, from_dev, log, rel_err  # noqa: E402
from paper_2308_16369_amd import sarathi as S  # noqa: E402
from paper_2308_16369_amd import serve  # noqa: E402

REQS = [(40, 5), (23, 7), (64, 0), (10, 12), (17, 3)]


def setup(dtype, n_layers, seed):
    shape = dataclasses.replace(wl.TINY.shape, dtype=dtype)
    rng = np.random.Generator(np.random.PCG64(seed))
    weights = [wl.draw_weights(rng, shape) for _ in range(n_layers)]
    maxlen = max(p + d for p, d in REQS)
    X = rng.standard_normal((len(REQS), maxlen, shape.hidden)).astype(np.float32)
    if dtype == "bf16":
        X = wl.round_to_bf16(X)
    m = serve.ServeModel(shape, n_layers, n_slots=3, max_seq_len=maxlen, max_tokens=256, weights=weights,
                         max_chunks=3)
    xin = torch.from_numpy(X).to(m.tdt).cuda()
    return shape, weights, X, m, xin


def oracle_outputs(shape, weights, X):
    outs = []
    for r, (p, d) in enumerate(REQS):
        n = p + d
        kv = np.zeros((len(weights), 1, 2, shape.n_heads, n, shape.head_dim))
        ob = oracle.OracleBatch(0, 0, n, [], [])
        outs.append(oracle.model_step(shape, weights, kv, ob, X[r, :n])[-1].y)
    return outs


def serve_outputs(m, xin, policy, B, C, **kw):
    out = torch.full_like(xin, float("nan"))
    res = serve.run_schedule(m, policy, REQS, B, C, inputs=xin, outputs=out, **kw)
    torch.cuda.synchronize()
    return from_dev(out), res


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_served_tokens_match_one_shot_oracle(dtype):
    shape, weights, X, m, xin = setup(dtype, n_layers=2, seed=3)
    ref = oracle_outputs(shape, weights, X)
    for policy, C, kw in [(S.POLICY_DECODE_MAXIMAL, 16, {}), (S.POLICY_PREFILL_DECODE, 0, {}),
                          (S.POLICY_MIXED, 0, dict(max_chunks=3, max_tokens=200))]:
        got, res = serve_outputs(m, xin, policy, B=3, C=C, **kw)
        log(f"{serve.POLICY_NAMES[policy]} {dtype}: {res['iterations']} iterations "
            f"({res['hybrid_iterations']} hybrid)")
        for r, (p, d) in enumerate(REQS):
            e = rel_err(got[r, :p + d], ref[r])
            assert e <= TOL[dtype], (policy, r, e)
        if policy in (S.POLICY_DECODE_MAXIMAL, S.POLICY_MIXED):
            assert res["hybrid_iterations"] > 0


def test_policies_agree_token_by_token_bf16():
    shape, weights, X, m, xin = setup("bf16", n_layers=3, seed=5)
    a, _ = serve_outputs(m, xin, S.POLICY_DECODE_MAXIMAL, B=3, C=8)
    b, _ = serve_outputs(m, xin, S.POLICY_PREFILL_DECODE, B=3, C=0)
    c, _ = serve_outputs(m, xin, S.POLICY_DECODE_MAXIMAL, B=2, C=32)
    for r, (p, d) in enumerate(REQS):
        assert np.all(np.isfinite(a[r, :p + d]))
        assert rel_err(a[r, :p + d], b[r, :p + d]) <= TOL["bf16"]
        assert rel_err(c[r, :p + d], b[r, :p + d]) <= TOL["bf16"]


def test_sweep_runs_tiny():
    shape = wl.with_dtype(wl.TINY, "bf16").shape
    m = serve.ServeModel(shape, 2, n_slots=4, max_seq_len=128, max_tokens=128)
    rows = serve.sweep(m, 128, [1, 7], [32], max_batch=4, n_requests=6)
    assert len(rows) == 2
    for e in rows:
        assert e["P"] + e["D"] == 128
        assert e["decode_maximal"]["tokens"] == e["baseline"]["tokens"] == 6 * 128
        assert e["speedup"] > 0
