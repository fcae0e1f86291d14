"""Host scheduler (include/sarathi_sched.h): worked schedules under each
policy, invariants of random request sets, and argument errors.  Pure host
code -- no GPU."""
import random

import pytest

from paper_2308_16369_amd import sarathi as S

REQS = [(6, 2), (4, 1), (3, 0), (2, 1)]     # (prompt, decodes)


def run_all(sched, limit=100000):
    steps = []
    for _ in range(limit):
        st = sched.next()
        if st.n_tokens == 0:
            return steps
        steps.append(st)
        sched.commit()
    raise AssertionError("scheduler did not drain")


def summary(st):
    return ([(r, s, o, n) for r, s, o, n in zip(st.chunk_request, st.chunk_slot, st.chunk_offset, st.chunk_len)],
            [(r, s, c) for r, s, c in zip(st.decode_request, st.decode_slot, st.decode_ctx)])


def make(policy, reqs=REQS, B=3, C=4, **kw):
    s = S.Scheduler(policy, max_batch=B, n_slots=kw.pop("n_slots", B), max_seq_len=kw.pop("S", 64), chunk=C, **kw)
    for p, d in reqs:
        s.submit(p, d)
    return s


def test_decode_maximal_worked_schedule():
    """One chunk of at most C per iteration (oldest request in prefill) plus
    the decodes of the other resident requests (Sec. 4.3); worked by hand."""
    s = make(S.POLICY_DECODE_MAXIMAL)
    got = [summary(st) for st in run_all(s)]
    assert got == [
        ([(0, 0, 0, 4)], []),
        ([(0, 0, 4, 2)], []),
        ([(1, 1, 0, 4)], [(0, 0, 6)]),
        ([(2, 2, 0, 3)], [(0, 0, 7), (1, 1, 4)]),   # r2 (D=0), r0 and r1 finish here
        ([(3, 0, 0, 2)], []),                        # r3 admitted into the lowest free slot
        ([], [(3, 0, 2)]),
    ]
    st = s.stats()
    assert (st["iterations"], st["prefill_tokens"], st["decode_tokens"]) == (6, 15, 4)
    assert (st["hybrid_iterations"], st["prefill_only_iterations"], st["decode_only_iterations"]) == (2, 3, 1)
    assert (st["submitted"], st["admitted"], st["finished"], st["resident"]) == (4, 4, 4, 0)


def test_prefill_decode_baseline_worked_schedule():
    """Baseline of Sec. 5.1: whole prompts in prefill-only iterations, then
    decode-only iterations."""
    s = make(S.POLICY_PREFILL_DECODE)
    got = [summary(st) for st in run_all(s)]
    assert got == [
        ([(0, 0, 0, 6)], []),
        ([(1, 1, 0, 4)], []),
        ([(2, 2, 0, 3)], []),
        ([(3, 2, 0, 2)], []),
        ([], [(0, 0, 6), (1, 1, 4), (3, 2, 2)]),
        ([], [(0, 0, 7)]),
    ]
    st = s.stats()
    assert (st["hybrid_iterations"], st["prefill_only_iterations"], st["decode_only_iterations"]) == (0, 4, 2)


def test_mixed_worked_schedule():
    """Orca-style mixed batching: whole prompts (max_chunks, max_tokens)
    beside every decode."""
    s = make(S.POLICY_MIXED, C=0, max_chunks=2, max_tokens=8)
    got = [summary(st) for st in run_all(s)]
    assert got == [
        ([(0, 0, 0, 6)], []),
        ([(1, 1, 0, 4), (2, 2, 0, 3)], [(0, 0, 6)]),
        ([(3, 2, 0, 2)], [(0, 0, 7), (1, 1, 4)]),
        ([], [(3, 2, 2)]),
    ]


def test_next_is_stable_until_commit_and_sees_late_arrivals():
    s = S.Scheduler(S.POLICY_DECODE_MAXIMAL, max_batch=2, n_slots=2, max_seq_len=32, chunk=8)
    assert s.next().n_tokens == 0            # nothing submitted
    s.submit(5, 1)                           # seen although the last description was empty
    a, b = s.next(), s.next()
    assert summary(a) == summary(b) == ([(0, 0, 0, 5)], [])
    s.commit()
    assert summary(s.next()) == ([], [(0, 0, 5)])


@pytest.mark.parametrize("policy", [S.POLICY_DECODE_MAXIMAL, S.POLICY_PREFILL_DECODE, S.POLICY_MIXED])
@pytest.mark.parametrize("seed", range(6))
def test_random_request_sets_keep_the_invariants(policy, seed):
    rng = random.Random(seed * 7 + policy)
    B = rng.randint(1, 6)
    C = rng.choice([1, 3, 8, 16])
    n_slots = B + rng.randint(0, 2)
    Smax = 80
    reqs = []
    for _ in range(rng.randint(1, 14)):
        p = rng.randint(1, 50)
        reqs.append((p, rng.randint(0, Smax - p)))
    s = S.Scheduler(policy, max_batch=B, n_slots=n_slots, max_seq_len=Smax, chunk=C, max_chunks=3, max_tokens=60)
    for p, d in reqs:
        s.submit(p, d)
    prompt_done = [0] * len(reqs)
    dec_done = [0] * len(reqs)
    slot_of = {}
    for _ in range(100000):
        st = s.next()
        if st.n_tokens == 0:
            break
        ids = st.chunk_request + st.decode_request
        assert len(ids) == len(set(ids)), "a request twice in one iteration"
        assert st.n_tokens == sum(st.chunk_len) + st.n_decodes
        if policy != S.POLICY_MIXED:
            assert st.n_chunks <= 1
        if policy == S.POLICY_DECODE_MAXIMAL:
            assert all(n <= C for n in st.chunk_len)
            assert st.n_decodes <= (B - 1 if st.n_chunks else B)
        if policy == S.POLICY_PREFILL_DECODE:
            assert not (st.n_chunks and st.n_decodes)
        if policy == S.POLICY_MIXED:
            assert st.n_chunks <= 3
            assert st.n_chunks <= 1 or sum(st.chunk_len) <= 60
        # slots: one per resident request, exclusive, in range
        for r, sl in list(zip(st.chunk_request, st.chunk_slot)) + list(zip(st.decode_request, st.decode_slot)):
            assert 0 <= sl < n_slots
            assert slot_of.setdefault(r, sl) == sl, "a request changed slot"
        live = {r for r in slot_of if dec_done[r] < reqs[r][1] or prompt_done[r] < reqs[r][0]}
        assert len({slot_of[r] for r in live}) == len(live), "two live requests share a slot"
        assert len(live) <= B
        for r, o, n in zip(st.chunk_request, st.chunk_offset, st.chunk_len):
            assert o == prompt_done[r] and n >= 1 and o + n <= reqs[r][0]
            prompt_done[r] += n
        for r, c in zip(st.decode_request, st.decode_ctx):
            assert prompt_done[r] == reqs[r][0], "decode before the prompt is done"
            assert c == reqs[r][0] + dec_done[r] and c + 1 <= Smax
            dec_done[r] += 1
        s.commit()
        for r in list(slot_of):   # finished requests release their slots
            if prompt_done[r] == reqs[r][0] and dec_done[r] == reqs[r][1]:
                del slot_of[r]
                prompt_done[r] = dec_done[r] = 10 ** 9   # mark finished
    st = s.stats()
    assert st["finished"] == len(reqs)
    assert st["prefill_tokens"] == sum(p for p, _ in reqs)
    assert st["decode_tokens"] == sum(d for _, d in reqs)


def test_balanced_pd_piggybacks_every_decode():
    """When P:D = C/(B-1) with all requests arriving together in waves of B,
    decodes ride along the chunks of later requests (Sec. 5.1.3): the
    iterations are at most the chunks plus one drain of D decodes."""
    B, C, k = 5, 8, 4
    P, D = k * C, k * (B - 1)
    N = 4 * B
    s = S.Scheduler(S.POLICY_DECODE_MAXIMAL, max_batch=B, n_slots=B, max_seq_len=P + D, chunk=C)
    for _ in range(N):
        s.submit(P, D)
    run_all(s)
    st = s.stats()
    assert st["prefill_tokens"] == N * P and st["decode_tokens"] == N * D
    assert st["iterations"] <= N * P // C + D
    assert st["hybrid_iterations"] >= st["iterations"] - (P // C) - D


def test_argument_errors():
    cfg = dict(max_batch=2, n_slots=2, max_seq_len=16, chunk=4)
    for bad in [dict(cfg, max_batch=0), dict(cfg, chunk=0), dict(cfg, n_slots=1), dict(cfg, max_seq_len=0)]:
        with pytest.raises(S.SarathiError) as ei:
            S.Scheduler(S.POLICY_DECODE_MAXIMAL, **bad)
        assert ei.value.code == S.EINVAL
    with pytest.raises(S.SarathiError):
        S.Scheduler(7, **cfg)
    with pytest.raises(S.SarathiError):
        S.Scheduler(S.POLICY_MIXED, **cfg)            # max_chunks / max_tokens missing
    s = S.Scheduler(S.POLICY_DECODE_MAXIMAL, **cfg)
    for p, d in [(0, 1), (4, -1), (10, 7)]:
        with pytest.raises(S.SarathiError) as ei:
            s.submit(p, d)
        assert ei.value.code == S.ERANGE
    with pytest.raises(S.SarathiError) as ei:
        s.commit()
    assert ei.value.code == S.ENOSPC
    s.submit(10, 6)                                   # P + D == max_seq_len is allowed


def test_serving_batch_from_the_memory_equation():
    """Sec. 4.3.1: B = floor((M_G - M_S) / (L m_kv)) for the LLaMA-13B shape
    (40 layers, 634 MB of weights per layer, 0.8 MB of K/V per token)."""
    import workloads as wl
    from paper_2308_16369_amd.serve import equation_batch
    shape = wl.LLAMA13B_LAYER.shape
    eq = equation_batch(shape, 40, 1024, 288 * 10**9, headroom=8 << 30)
    m_s = 40 * 2 * (3 * 5120 * 5120 + 5120 * 5120 + 2 * 13824 * 5120 + 5120 * 13824 + 2 * 5120)
    m_kv = 40 * 2 * 5120 * 2
    assert eq["mem_params"] == m_s and eq["kv_bytes_per_token"] == m_kv
    assert eq["B"] == (288 * 10**9 - (8 << 30) - m_s) // (1024 * m_kv)
    # an A6000-sized device (48 GB, no headroom) gives the paper's order of magnitude
    assert 20 <= equation_batch(shape, 40, 1024, 48 * 10**9)["B"] <= 30
