"""Pipeline-bubble simulator (host only): hand-worked schedules, the uniform
case, the cost model's interpolation, and the bubble ordering of the two
batching policies on a prefill-heavy cost model."""
import numpy as np
import pytest

from paper_2308_16369_amd import pipeline_sim as P
from paper_2308_16369_amd import sarathi as S


def flat_cost(ms=1.0):
    return P.CostModel(rows=[1, 100000], linear_ms=[ms, ms], pre=(0.0, 0.0, 0.0), dec=(0.0, 0.0, 0.0))


def rows_cost():
    """layer time = rows (ms), no attention terms."""
    return P.CostModel(rows=[1, 1000], linear_ms=[1.0, 1000.0], pre=(0.0, 0.0, 0.0), dec=(0.0, 0.0, 0.0))


def test_hand_worked_two_stage_schedule():
    """Stages 2, micro-batches 2, one request each: r0 = 10-token prompt, r1 =
    2-token prompt then 3 decodes; a layer costs its row count (ms), one layer
    per stage.  Worked by hand: r1's iterations wait 10 + 1 ms, then 1 + 1 ms
    twice on the two stages; makespan 28 ms."""
    res = P.simulate([(10, 0), (2, 3)], S.POLICY_DECODE_MAXIMAL, n_stages=2, n_layers=2, micro_batches=2,
                     batch_per_mb=1, cost=rows_cost(), chunk=16)
    assert res.makespan_ms == pytest.approx(28.0)
    np.testing.assert_allclose(res.bubble_ms_per_request, [0.0, 15.0])
    assert res.iterations == 5


def test_uniform_work_has_no_bubbles():
    """Equal work per micro-batch iteration and as many micro-batches as
    stages: the pipeline stays full, makespan = (iterations + S - 1) * t."""
    S_, L = 4, 8
    reqs = [(8, 5)] * 8
    res = P.simulate(reqs, S.POLICY_DECODE_MAXIMAL, n_stages=S_, n_layers=L, micro_batches=S_, batch_per_mb=1,
                     cost=flat_cost(0.5), chunk=8)
    t = (L // S_) * 0.5
    assert np.all(res.bubble_ms_per_request == 0.0)
    assert res.makespan_ms == pytest.approx((res.iterations + S_ - 1) * t)
    assert res.iterations == 8 * (1 + 5)


def test_cost_model_interpolates_and_adds_attention():
    cm = P.CostModel(rows=[16, 32, 64], linear_ms=[1.0, 1.5, 3.0], pre=(1e-6, 1e-4, 0.01), dec=(2e-5, 1e-3, 0.02))
    assert cm.linear(16) == 1.0 and cm.linear(48) == pytest.approx(2.25) and cm.linear(128) == pytest.approx(6.0)
    assert cm.linear(8) == pytest.approx(0.5)
    pairs = 10 * 100 + 10 * 11 / 2
    assert cm.chunk_attn(100, 10) == pytest.approx(1e-6 * pairs + 1e-4 * 110 + 0.01)
    assert cm.decode_attn([]) == 0.0
    assert cm.decode_attn([9, 19]) == pytest.approx(2e-5 * 30 + 2e-3 + 0.02)
    assert cm.layer_ms([(100, 10)], [9, 19]) == pytest.approx(cm.linear(12) + cm.chunk_attn(100, 10)
                                                            + cm.decode_attn([9, 19]))
    back = P.CostModel.from_json(cm.to_json())
    assert back.layer_ms([(0, 20)], [5]) == cm.layer_ms([(0, 20)], [5])


def test_fit_recovers_coefficients():
    rng = np.random.default_rng(0)
    X = np.column_stack([rng.uniform(0, 1e6, 30), rng.uniform(0, 4096, 30), np.ones(30)])
    y = X @ np.array([3e-9, 2e-6, 0.01])
    np.testing.assert_allclose(P.fit_linear_terms(X, y), [3e-9, 2e-6, 0.01], rtol=1e-6)


def test_zipf_lengths_and_pd_split():
    L = P.zipf_lengths(5000, 1024, 4096, 0.4, seed=1)
    assert L.min() >= 1024 and L.max() <= 4096
    assert np.mean(L < 2048) > np.mean(L >= 3072)          # decreasing density
    for p, d in P.pd_requests([1100, 4096, 2000], 10.0):
        assert d >= 1 and abs(p / d - 10.0) < 0.6


def test_decode_maximal_shrinks_bubbles_on_prefill_heavy_costs():
    """Sec. 3.2: with iteration costs dominated by prefill rows, mixed batches
    of whole prompts vary a lot between micro-batches, chunked ones do not."""
    cm = P.CostModel(rows=[1, 8192], linear_ms=[0.01, 8192 * 0.01], pre=(0.0, 0.0, 0.0), dec=(1e-6, 1e-4, 0.0))
    reqs = P.pd_requests(P.zipf_lengths(200, 1024, 4096, 0.4, seed=3), 10.0)
    mix = P.simulate(reqs, S.POLICY_MIXED, 4, 8, 4, 8, cm, max_chunks=8, max_tokens=4096)
    dm = P.simulate(reqs, S.POLICY_DECODE_MAXIMAL, 4, 8, 4, 8, cm, chunk=256)
    assert np.median(dm.bubble_ms_per_request) < np.median(mix.bubble_ms_per_request)
    assert dm.stage_busy_frac > mix.stage_busy_frac
