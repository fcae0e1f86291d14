"""Pins of the float64 oracle against closed forms, invariants, library
routines, brute force and the paper's own printed values.

Each test names what would fail it: a dropped term, a wrong sign or index, a
transposed operand, an off-by-one in the mask, a misplaced cache write.
"""
import copy
import json
import math
import os

import numpy as np
import pytest
import scipy.special

import oracle
from oracle import OracleBatch
import workloads as wl
from paper_2308_16369_amd import accounting

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
RNG = np.random.default_rng(1234)


def tiny_shape(**kw):
    base = dict(hidden=32, n_heads=2, head_dim=16, ffn=24, norm="rms", act="swiglu",
                rope=True, rope_base=10000.0, eps=1e-6, dtype="f32")
    base.update(kw)
    return wl.LayerShape(**base)


def rand_weights(shape, rng, scale=0.2):
    H, nh, d, F = shape.hidden, shape.n_heads, shape.head_dim, shape.ffn
    w = {
        "w_qkv": rng.standard_normal((3 * nh * d, H)) * scale,
        "w_o": rng.standard_normal((H, nh * d)) * scale,
        "w_up": rng.standard_normal((shape.up_rows, H)) * scale,
        "w_down": rng.standard_normal((H, F)) * scale,
        "norm1_g": 1 + 0.1 * rng.standard_normal(H),
        "norm2_g": 1 + 0.1 * rng.standard_normal(H),
    }
    if shape.norm == "layer":
        w["norm1_b"] = 0.1 * rng.standard_normal(H)
        w["norm2_b"] = 0.1 * rng.standard_normal(H)
    return w


def empty_cache(shape, n_slots, S):
    return np.full((n_slots, 2, shape.n_heads, S, shape.head_dim), np.nan)


def fill_prefix(cache, slot, n, rng):
    cache[slot, :, :, :n, :] = rng.standard_normal(cache[slot, :, :, :n, :].shape)


# ============================================================================ linear

def test_linear_matches_triple_loop_on_nonsquare():
    x = RNG.standard_normal((3, 5))
    w = RNG.standard_normal((4, 5))
    y = oracle.linear(x, w)
    assert y.shape == (3, 4)
    for i in range(3):
        for j in range(4):
            acc = 0.0
            for k in range(5):
                acc += x[i, k] * w[j, k]
            assert abs(y[i, j] - acc) < 1e-12


# ============================================================================ norms

def test_rms_norm_unit_gain_rms_closed_form():
    x = RNG.standard_normal((6, 40)) * 3.0
    eps = 1e-2
    out = oracle.rms_norm(x, np.ones(40), eps)
    ms = np.mean(x * x, axis=1)
    np.testing.assert_allclose(np.sqrt(np.mean(out * out, axis=1)), np.sqrt(ms / (ms + eps)), rtol=1e-12)
    # direction is preserved: out is a positive multiple of x
    cos = np.sum(out * x, axis=1) / np.linalg.norm(out, axis=1) / np.linalg.norm(x, axis=1)
    np.testing.assert_allclose(cos, 1.0, rtol=1e-12)


def test_rms_norm_gain_is_elementwise_and_constant_row():
    g = 1 + RNG.standard_normal(16)
    x = RNG.standard_normal((3, 16))
    out = oracle.rms_norm(x, g, 1e-6)
    ref_dir = oracle.rms_norm(x, np.ones(16), 1e-6)
    np.testing.assert_allclose(out / g, ref_dir, rtol=1e-12)
    c = 2.5
    row = oracle.rms_norm(np.full((1, 16), c), g, 0.25)
    np.testing.assert_allclose(row[0], c / math.sqrt(c * c + 0.25) * g, rtol=1e-13)


def test_layer_norm_moments_and_affine():
    x = RNG.standard_normal((5, 64)) * 2 + 0.7
    eps = 1e-2
    out = oracle.layer_norm(x, np.ones(64), np.zeros(64), eps)
    var = np.var(x, axis=1)
    np.testing.assert_allclose(np.mean(out, axis=1), 0.0, atol=1e-13)
    np.testing.assert_allclose(np.var(out, axis=1), var / (var + eps), rtol=1e-12)
    g, b = 1 + RNG.standard_normal(64), RNG.standard_normal(64)
    out2 = oracle.layer_norm(x, g, b, eps)
    np.testing.assert_allclose((out2 - b) / g, out, rtol=1e-11, atol=1e-12)
    # a constant row normalises to the bias exactly
    np.testing.assert_allclose(oracle.layer_norm(np.full((1, 64), 3.0), g, b, eps)[0], b, atol=1e-15)


# ============================================================================ activations

def test_silu_and_gelu_against_library_routines():
    z = np.linspace(-9, 9, 301)
    np.testing.assert_allclose(oracle.silu(z), z * scipy.special.expit(z), rtol=1e-13, atol=1e-300)
    np.testing.assert_allclose(oracle.gelu(z), z * scipy.special.ndtr(z), rtol=1e-12, atol=1e-15)
    # odd-part identity: gelu(z) - gelu(-z) = z and silu(z) - silu(-z) = z
    np.testing.assert_allclose(oracle.gelu(z) - oracle.gelu(-z), z, atol=1e-13)
    np.testing.assert_allclose(oracle.silu(z) - oracle.silu(-z), z, atol=1e-13)


# ============================================================================ rotary embedding

def test_rope_d2_is_a_rotation_by_position():
    for p in [0, 1, 3, 17, 1000]:
        e0 = oracle.rope_rotate(np.array([[1.0, 0.0]]), np.array([p]), 10000.0)[0]
        e1 = oracle.rope_rotate(np.array([[0.0, 1.0]]), np.array([p]), 10000.0)[0]
        np.testing.assert_allclose(e0, [math.cos(p), math.sin(p)], atol=1e-12)
        np.testing.assert_allclose(e1, [-math.sin(p), math.cos(p)], atol=1e-12)


def test_rope_pairs_first_half_with_second_half():
    base, p = 100.0, 5
    th1 = base ** (-0.5)
    u = np.eye(4)
    r = oracle.rope_rotate(u, np.full(4, p), base)
    np.testing.assert_allclose(r[0], [math.cos(p), 0, math.sin(p), 0], atol=1e-12)
    np.testing.assert_allclose(r[1], [0, math.cos(p * th1), 0, math.sin(p * th1)], atol=1e-12)
    np.testing.assert_allclose(r[2], [-math.sin(p), 0, math.cos(p), 0], atol=1e-12)


def test_rope_identity_norm_and_relative_position():
    d = 64
    q = RNG.standard_normal((1, d))
    k = RNG.standard_normal((1, d))
    np.testing.assert_allclose(oracle.rope_rotate(q, np.array([0]), 1e4), q, atol=1e-15)
    r = oracle.rope_rotate(q, np.array([123]), 1e4)
    np.testing.assert_allclose(np.linalg.norm(r), np.linalg.norm(q), rtol=1e-13)
    for (m, n, s) in [(10, 3, 7), (0, 50, 200), (900, 899, 31)]:
        a = oracle.rope_rotate(q, np.array([m]), 1e4) @ oracle.rope_rotate(k, np.array([n]), 1e4).T
        b = oracle.rope_rotate(q, np.array([m + s]), 1e4) @ oracle.rope_rotate(k, np.array([n + s]), 1e4).T
        np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-9)


# ============================================================================ attention

def test_attend_special_cases():
    nh, d = 2, 8
    v1 = RNG.standard_normal((nh, 1, d))
    k1 = RNG.standard_normal((nh, 1, d))
    q = RNG.standard_normal((nh, d))
    np.testing.assert_array_equal(oracle.attend(q, k1, v1), v1[:, 0, :])       # one key
    n = 7
    vals = RNG.standard_normal((nh, n, d))
    same = np.repeat(RNG.standard_normal((nh, 1, d)), n, axis=1)
    np.testing.assert_allclose(oracle.attend(q, same, vals), vals.mean(axis=1), rtol=1e-12)  # equal keys
    keys = RNG.standard_normal((nh, n, d))
    np.testing.assert_allclose(oracle.attend(np.zeros((nh, d)), keys, vals), vals.mean(axis=1), rtol=1e-12)


def test_attend_two_keys_closed_form_and_scale():
    d = 4
    q = np.array([[1.0, 2.0, 0.0, -1.0]])
    keys = np.array([[[0.5, 0.0, 1.0, 0.0], [0.0, 1.0, 0.0, 1.0]]])
    vals = np.array([[[1.0, 0.0, 0.0, 0.0], [0.0, 1.0, 0.0, 0.0]]])
    s1, s2 = 0.5 / 2.0, 1.0 / 2.0          # q.k / sqrt(4)
    w1 = 1.0 / (1.0 + math.exp(s2 - s1))
    np.testing.assert_allclose(oracle.attend(q, keys, vals)[0], [w1, 1 - w1, 0, 0], rtol=1e-14)


def test_attend_weights_form_a_distribution():
    n = 9
    q = RNG.standard_normal((1, n)) * 3
    keys = RNG.standard_normal((1, n, n))
    wts = oracle.attend(q, keys, np.eye(n)[None])[0]      # values = identity -> weights
    assert np.all(wts >= 0)
    np.testing.assert_allclose(wts.sum(), 1.0, rtol=1e-14)
    # peaked scores pick the matching value
    k = np.eye(n)[None] * 1.0
    qp = np.zeros((1, n)); qp[0, 4] = 400.0
    vals = RNG.standard_normal((1, n, 3))
    np.testing.assert_allclose(oracle.attend(qp, k, vals)[0], vals[0, 4], atol=1e-12)


def test_attend_matches_pure_python_loops():
    nh, n, d = 3, 6, 5
    q = RNG.standard_normal((nh, d))
    keys = RNG.standard_normal((nh, n, d))
    vals = RNG.standard_normal((nh, n, d))
    got = oracle.attend(q, keys, vals)
    for h in range(nh):
        sc = [sum(q[h, i] * keys[h, j, i] for i in range(d)) / math.sqrt(d) for j in range(n)]
        mx = max(sc)
        ex = [math.exp(s - mx) for s in sc]
        tot = sum(ex)
        for i in range(d):
            ref = sum(ex[j] / tot * vals[h, j, i] for j in range(n))
            assert abs(got[h, i] - ref) < 1e-12


# ============================================================================ layer-level mask pins

def _run(shape, w, cache, batch, x):
    return oracle.layer_forward(shape, w, cache, batch, x)


def test_decode_with_empty_context_returns_its_own_value():
    shape = tiny_shape()
    w = rand_weights(shape, RNG)
    cache = empty_cache(shape, 3, 16)
    batch = OracleBatch(prefill_slot=-1, chunk_offset=0, chunk_len=0, decode_slots=[1], decode_ctx=[0])
    x = RNG.standard_normal((1, shape.hidden))
    out = _run(shape, w, cache, batch, x)
    np.testing.assert_allclose(out.o[0], out.v_new[0].reshape(-1), rtol=1e-14)


def test_no_read_past_position_nan_poison():
    shape = tiny_shape()
    w = rand_weights(shape, RNG)
    cache = empty_cache(shape, 4, 32)          # everything NaN ...
    fill_prefix(cache, 0, 5, RNG)              # ... except the valid prefixes
    fill_prefix(cache, 2, 11, RNG)
    fill_prefix(cache, 3, 3, RNG)
    batch = OracleBatch(prefill_slot=0, chunk_offset=5, chunk_len=6, decode_slots=[2, 3], decode_ctx=[11, 3])
    out = _run(shape, w, cache, batch, RNG.standard_normal((8, shape.hidden)))
    assert np.all(np.isfinite(out.y))
    # writes landed exactly at (slot, position) and nowhere else
    assert not np.isnan(cache[0, :, :, 5:11]).any() and np.isnan(cache[0, :, :, 11:]).all()
    assert not np.isnan(cache[2, :, :, 11]).any() and np.isnan(cache[2, :, :, 12:]).all()
    assert not np.isnan(cache[3, :, :, 3]).any() and np.isnan(cache[3, :, :, 4:]).all()
    assert np.isnan(cache[1]).all()


def _read_mask_fixture():
    blocks, cur = [], None
    with open(os.path.join(GOLDEN, "chunk_mask_c4_p12.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("iteration"):
                cur = []
                blocks.append((int(line.split()[3]), cur))
            else:
                cur.append([c == "1" for c in line])
    return [(off, np.array(rows, dtype=bool)) for off, rows in blocks]


def test_chunk_visibility_matches_paper_figure():
    fixture = _read_mask_fixture()
    vis = oracle.chunk_visibility(12, 4)
    assert len(vis) == len(fixture) == 3
    for (off, ref), got in zip(fixture, vis):
        np.testing.assert_array_equal(got, ref)


def test_layer_attention_dependence_matches_paper_figure():
    """Perturb one key (a cached token or a chunk token) and see which chunk
    queries' attention outputs move: exactly the visible ones."""
    shape = tiny_shape(rope=False)
    w = rand_weights(shape, RNG)
    fixture = _read_mask_fixture()
    for off, ref in fixture:
        C = 4
        cache = empty_cache(shape, 1, 12)
        fill_prefix(cache, 0, off, RNG)
        x = RNG.standard_normal((C, shape.hidden))
        batch = OracleBatch(prefill_slot=0, chunk_offset=off, chunk_len=C, decode_slots=[], decode_ctx=[])
        base = _run(shape, w, cache.copy(), batch, x).o
        for j in range(off + C):
            c2, x2 = cache.copy(), x.copy()
            if j < off:
                c2[0, :, :, j, :] += 1.0
            else:
                x2[j - off] += 1.0
            o2 = _run(shape, w, c2, batch, x2).o
            changed = np.any(np.abs(o2 - base) > 1e-12, axis=1)
            np.testing.assert_array_equal(changed, ref[:, j], err_msg=f"offset {off} key {j}")


# ============================================================================ method invariants

def _prompt_setup(shape, P, S, rng, n_slots=2):
    w = rand_weights(shape, rng)
    cache = empty_cache(shape, n_slots, S)
    x = rng.standard_normal((P, shape.hidden))
    return w, cache, x


def test_chunked_prefill_equals_one_shot_prefill():
    """Sec. 4.2: chunked prefill is mathematically equivalent to the full prefill."""
    shape = tiny_shape()
    P, C = 16, 4
    w, cache, x = _prompt_setup(shape, P, 20, RNG)
    full_cache = cache.copy()
    full = _run(shape, w, full_cache,
                OracleBatch(prefill_slot=1, chunk_offset=0, chunk_len=P, decode_slots=[], decode_ctx=[]), x)
    ch_cache = cache.copy()
    ys = []
    for off in range(0, P, C):
        out = _run(shape, w, ch_cache,
                   OracleBatch(prefill_slot=1, chunk_offset=off, chunk_len=C, decode_slots=[], decode_ctx=[]),
                   x[off:off + C])
        ys.append(out.y)
    np.testing.assert_allclose(np.concatenate(ys), full.y, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(ch_cache[1, :, :, :P], full_cache[1, :, :, :P], rtol=1e-11, atol=1e-12)
    assert np.isnan(ch_cache[1, :, :, P:]).all()


def test_decode_equals_chunk_of_length_one():
    shape = tiny_shape()
    w, cache, _ = _prompt_setup(shape, 1, 16, RNG, n_slots=3)
    fill_prefix(cache, 2, 9, RNG)
    x = RNG.standard_normal((1, shape.hidden))
    c1, c2 = cache.copy(), cache.copy()
    a = _run(shape, w, c1, OracleBatch(-1, 0, 0, [2], [9]), x)
    b = _run(shape, w, c2, OracleBatch(2, 9, 1, [], []), x)
    np.testing.assert_allclose(a.y, b.y, rtol=1e-13)
    np.testing.assert_array_equal(np.isnan(c1), np.isnan(c2))
    np.testing.assert_allclose(np.nan_to_num(c1), np.nan_to_num(c2), rtol=1e-13)


def _hybrid_setup(shape, rng):
    n_slots, S = 5, 24
    w = rand_weights(shape, rng)
    cache = empty_cache(shape, n_slots, S)
    fill_prefix(cache, 3, 6, rng)             # chunk slot, 6 tokens cached
    ctx = {0: 4, 1: 13, 4: 0}
    for s, n in ctx.items():
        fill_prefix(cache, s, n, rng)
    C = 5
    xc = rng.standard_normal((C, shape.hidden))
    xd = rng.standard_normal((3, shape.hidden))
    return w, cache, xc, xd, [0, 1, 4], [ctx[0], ctx[1], ctx[4]]


@pytest.mark.parametrize("kind", ["llama", "gpt"])
def test_concatenation_and_batch_invariance(kind):
    """Sec. 4.3: the hybrid batch is prefill-only rows + decode-only rows, and a
    piggybacked decode equals the same decode run alone."""
    shape = tiny_shape() if kind == "llama" else tiny_shape(norm="layer", act="gelu", rope=False, eps=1e-5)
    w, cache, xc, xd, ds, dc = _hybrid_setup(shape, RNG)
    hyb_cache = cache.copy()
    hyb = _run(shape, w, hyb_cache, OracleBatch(3, 6, 5, ds, dc), np.concatenate([xc, xd]))
    pc = cache.copy()
    pre = _run(shape, w, pc, OracleBatch(3, 6, 5, [], []), xc)
    dec = _run(shape, w, pc, OracleBatch(-1, 0, 0, ds, dc), xd)
    np.testing.assert_allclose(hyb.y, np.concatenate([pre.y, dec.y]), rtol=1e-12, atol=1e-13)
    np.testing.assert_array_equal(np.isnan(hyb_cache), np.isnan(pc))
    np.testing.assert_allclose(np.nan_to_num(hyb_cache), np.nan_to_num(pc), rtol=1e-12, atol=1e-13)
    for b in range(3):
        alone = _run(shape, w, cache.copy(), OracleBatch(-1, 0, 0, [ds[b]], [dc[b]]), xd[b:b + 1])
        np.testing.assert_allclose(hyb.y[5 + b], alone.y[0], rtol=1e-12, atol=1e-13)


def test_mixed_batch_equals_its_chunks_run_one_by_one():
    """Mixed batching (several prompt chunks in one iteration, the baseline
    mechanism of Sec. 5.2): every chunk's rows equal the same chunk run alone
    as a prefill-only hybrid batch, the decodes equal a decode-only batch,
    and a one-chunk mixed batch is the hybrid batch itself."""
    shape = tiny_shape()
    rng = np.random.default_rng(77)
    w = rand_weights(shape, rng)
    S = 32
    cache = empty_cache(shape, 6, S)
    chunks = [(2, 5, 4), (0, 0, 3), (5, 11, 6)]     # (slot, offset, length)
    for slot, off, _ in chunks:
        fill_prefix(cache, slot, off, rng)
    ds, dc = [1, 4], [9, 0]
    for slot, ctx in zip(ds, dc):
        fill_prefix(cache, slot, ctx, rng)
    x = rng.standard_normal((4 + 3 + 6 + 2, shape.hidden))
    mix_cache = cache.copy()
    mix = _run(shape, w, mix_cache, oracle.OracleMixedBatch(chunks, ds, dc), x)
    ref_cache = cache.copy()
    r0 = 0
    for slot, off, n in chunks:
        one = _run(shape, w, ref_cache, OracleBatch(slot, off, n, [], []), x[r0:r0 + n])
        np.testing.assert_allclose(mix.y[r0:r0 + n], one.y, rtol=1e-12, atol=1e-13)
        np.testing.assert_array_equal(mix.slots[r0:r0 + n], slot)
        np.testing.assert_array_equal(mix.positions[r0:r0 + n], np.arange(off, off + n))
        r0 += n
    dec = _run(shape, w, ref_cache, OracleBatch(-1, 0, 0, ds, dc), x[r0:])
    np.testing.assert_allclose(mix.y[r0:], dec.y, rtol=1e-12, atol=1e-13)
    np.testing.assert_array_equal(np.isnan(mix_cache), np.isnan(ref_cache))
    np.testing.assert_allclose(np.nan_to_num(mix_cache), np.nan_to_num(ref_cache), rtol=1e-12, atol=1e-13)
    single = _run(shape, w, cache.copy(), oracle.OracleMixedBatch([chunks[0]], ds, dc),
                  np.concatenate([x[:4], x[r0:]]))
    hyb = _run(shape, w, cache.copy(), OracleBatch(2, 5, 4, ds, dc), np.concatenate([x[:4], x[r0:]]))
    np.testing.assert_array_equal(single.y, hyb.y)


def test_permuting_decodes_permutes_rows():
    shape = tiny_shape()
    w, cache, xc, xd, ds, dc = _hybrid_setup(shape, RNG)
    a = _run(shape, w, cache.copy(), OracleBatch(3, 6, 5, ds, dc), np.concatenate([xc, xd]))
    p = [2, 0, 1]
    b = _run(shape, w, cache.copy(), OracleBatch(3, 6, 5, [ds[i] for i in p], [dc[i] for i in p]),
             np.concatenate([xc, xd[p]]))
    np.testing.assert_allclose(b.y[5:], a.y[5:][p], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(b.y[:5], a.y[:5], rtol=1e-12, atol=1e-13)


def test_prefill_then_teacher_forced_decodes_equals_longer_prefill():
    shape = tiny_shape()
    n, k = 7, 4
    w, cache, x = _prompt_setup(shape, n + k, 16, RNG)
    c_full = cache.copy()
    full = _run(shape, w, c_full, OracleBatch(0, 0, n + k, [], []), x)
    c_inc = cache.copy()
    ys = [_run(shape, w, c_inc, OracleBatch(0, 0, n, [], []), x[:n]).y]
    for t in range(k):
        ys.append(_run(shape, w, c_inc, OracleBatch(-1, 0, 0, [0], [n + t]), x[n + t:n + t + 1]).y)
    np.testing.assert_allclose(np.concatenate(ys), full.y, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(np.nan_to_num(c_inc), np.nan_to_num(c_full), rtol=1e-11, atol=1e-12)


def test_zero_output_projections_give_identity_layer():
    shape = tiny_shape()
    w, cache, xc, xd, ds, dc = _hybrid_setup(shape, RNG)
    w = dict(w, w_o=np.zeros_like(w["w_o"]), w_down=np.zeros_like(w["w_down"]))
    x = np.concatenate([xc, xd])
    c = cache.copy()
    out = _run(shape, w, c, OracleBatch(3, 6, 5, ds, dc), x)
    np.testing.assert_array_equal(out.y, x)
    # the K/V of every new token are still appended
    assert not np.isnan(c[3, :, :, 6:11]).any()
    for s, n in zip(ds, dc):
        assert not np.isnan(c[s, :, :, n]).any()


def test_model_step_chains_layers():
    shape = tiny_shape()
    L = 3
    ws = [rand_weights(shape, RNG) for _ in range(L)]
    kv = np.stack([empty_cache(shape, 5, 24) for _ in range(L)])
    for layer in range(L):
        fill_prefix(kv[layer], 3, 6, RNG)
        fill_prefix(kv[layer], 0, 4, RNG)
    batch = OracleBatch(3, 6, 5, [0], [4])
    x = RNG.standard_normal((6, shape.hidden))
    kv1 = kv.copy()
    outs = oracle.model_step(shape, ws, kv1, batch, x)
    h = x
    kv2 = kv.copy()
    for layer in range(L):
        h = oracle.layer_forward(shape, ws[layer], kv2[layer], batch, h).y
    np.testing.assert_array_equal(outs[-1].y, h)
    zero = [dict(w, w_o=np.zeros_like(w["w_o"]), w_down=np.zeros_like(w["w_down"])) for w in ws]
    outs0 = oracle.model_step(shape, zero, kv.copy(), batch, x)
    np.testing.assert_array_equal(outs0[-1].y, x)


# ============================================================================ full-layer brute force

def _brute_layer(shape, w, cache, slots, pos, x):
    """Pure-Python loops over one layer (lists and the math module only)."""
    H, nh, d, F = shape.hidden, shape.n_heads, shape.head_dim, shape.ffn
    T = len(x)

    def norm(row, g, b):
        if shape.norm == "rms":
            ms = sum(v * v for v in row) / H
            return [row[i] / math.sqrt(ms + shape.eps) * g[i] for i in range(H)]
        mu = sum(row) / H
        var = sum((v - mu) ** 2 for v in row) / H
        return [(row[i] - mu) / math.sqrt(var + shape.eps) * g[i] + b[i] for i in range(H)]

    def matvec(W, row):
        return [sum(W[j][i] * row[i] for i in range(len(row))) for j in range(len(W))]

    def rot(vec, p):
        if not shape.rope:
            return list(vec)
        out = list(vec)
        for i in range(d // 2):
            th = shape.rope_base ** (-2.0 * i / d)
            c, s = math.cos(p * th), math.sin(p * th)
            out[i] = vec[i] * c - vec[i + d // 2] * s
            out[i + d // 2] = vec[i] * s + vec[i + d // 2] * c
        return out

    g1, g2 = list(w["norm1_g"]), list(w["norm2_g"])
    b1 = list(w.get("norm1_b", np.zeros(H)))
    b2 = list(w.get("norm2_b", np.zeros(H)))
    Wqkv, Wo, Wup, Wd = (w[k].tolist() for k in ("w_qkv", "w_o", "w_up", "w_down"))
    qs, ks, vs = [], [], []
    for t in range(T):
        a = norm(list(x[t]), g1, b1)
        qkv = matvec(Wqkv, a)
        qs.append([rot(qkv[h * d:(h + 1) * d], pos[t]) for h in range(nh)])
        ks.append([rot(qkv[nh * d + h * d: nh * d + (h + 1) * d], pos[t]) for h in range(nh)])
        vs.append([qkv[2 * nh * d + h * d: 2 * nh * d + (h + 1) * d] for h in range(nh)])
    ys = []
    for t in range(T):
        o = []
        for h in range(nh):
            keys, vals = [], []
            for j in range(pos[t] + 1):
                src = [u for u in range(T) if slots[u] == slots[t] and pos[u] == j]
                if src:
                    keys.append(ks[src[0]][h]); vals.append(vs[src[0]][h])
                else:
                    keys.append(list(cache[slots[t], 0, h, j])); vals.append(list(cache[slots[t], 1, h, j]))
            sc = [sum(qs[t][h][i] * kk[i] for i in range(d)) / math.sqrt(d) for kk in keys]
            mx = max(sc)
            ex = [math.exp(s - mx) for s in sc]
            tot = sum(ex)
            o += [sum(ex[j] / tot * vals[j][i] for j in range(len(vals))) for i in range(d)]
        hres = [x[t][i] + v for i, v in enumerate(matvec(Wo, o))]
        bn = norm(hres, g2, b2)
        up = matvec(Wup, bn)
        if shape.act == "swiglu":
            m = [up[i] / (1 + math.exp(-up[i])) * up[F + i] for i in range(F)]
        else:
            m = [0.5 * u * (1 + math.erf(u / math.sqrt(2))) for u in up]
        ys.append([hres[i] + v for i, v in enumerate(matvec(Wd, m))])
    return np.array(ys)


@pytest.mark.parametrize("kind", ["llama", "gpt"])
def test_full_layer_matches_pure_python_brute_force(kind):
    if kind == "llama":
        shape = tiny_shape(hidden=8, n_heads=2, head_dim=4, ffn=6)
    else:
        shape = tiny_shape(hidden=8, n_heads=2, head_dim=4, ffn=6, norm="layer", act="gelu", rope=False, eps=1e-5)
    rng = np.random.default_rng(7)
    w = rand_weights(shape, rng, scale=0.5)
    cache = empty_cache(shape, 3, 8)
    fill_prefix(cache, 0, 2, rng)
    fill_prefix(cache, 1, 3, rng)
    fill_prefix(cache, 2, 0, rng)
    batch = OracleBatch(0, 2, 2, [1, 2], [3, 0])
    x = rng.standard_normal((4, shape.hidden))
    slots, pos = oracle.token_positions(batch)
    ref = _brute_layer(shape, w, cache, list(slots), [int(p) for p in pos], x)
    got = _run(shape, w, cache.copy(), batch, x).y
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)


# ============================================================================ paper's printed numbers

def test_decode_accounting_reproduces_table2():
    with open(os.path.join(GOLDEN, "table2_decode_accounting.json")) as f:
        g = json.load(f)
    base = accounting.decode_time_per_token_baseline(g["decode_only_total_ms"], g["decode_only_batch"])
    hyb = accounting.decode_time_per_token_hybrid(g["decode_maximal_total_ms"], g["prefill_only_total_ms"],
                                                  g["decode_maximal_decodes"])
    assert round(base, 2) == g["expected_decode_ms_per_token_baseline"]
    assert round(hyb, 2) == g["expected_decode_ms_per_token_hybrid"]


def test_max_decode_batch_formula():
    # (M_G - M_S) / (L * m_kv) floored; one chunk takes one of the B slots
    assert accounting.max_decode_batch(48e9, 26e9, 1024, 819200) == 26
    assert accounting.max_decode_batch(48e9, 26e9, 4096, 819200) == 6


# ============================================================================ input generator (host logic)

def test_bf16_rounding_is_nearest_even():
    one = np.float32(1.0)
    vals = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -7, -(1 + 2 ** -8 + 2 ** -20), np.nan],
                    dtype=np.float32)
    r = wl.round_to_bf16(vals)
    np.testing.assert_array_equal(r[:4], np.array([1.0, 1 + 2 ** -6, 1 + 2 ** -7, -(1 + 2 ** -7)], np.float32))
    assert np.isnan(r[4])
    bits = wl.bf16_bits(r)
    assert bits[0] == 0x3F80 and bits[4] == 0x7FC0
    np.testing.assert_array_equal(wl.bits_to_f32(bits[:4]), r[:4])
    assert one == wl.round_to_bf16(np.array([one]))[0]


def test_generator_is_deterministic_and_nan_fills_empty_positions():
    a = wl.generate(wl.TINY)
    b = wl.generate(wl.TINY)
    np.testing.assert_array_equal(a.x, b.x)
    np.testing.assert_array_equal(a.batch.decode_ctx, b.batch.decode_ctx)
    np.testing.assert_array_equal(a.weights[0]["w_up"], b.weights[0]["w_up"])
    spec = wl.TINY.batch
    assert sorted([a.batch.prefill_slot] + list(a.batch.decode_slots)) == list(range(spec.n_slots))
    assert np.all((a.batch.decode_ctx >= spec.ctx_lo) & (a.batch.decode_ctx <= spec.ctx_hi))
    valid = wl.valid_lengths(a.batch, spec.n_slots)
    for s in range(spec.n_slots):
        assert not np.isnan(a.kv[0, s, :, :, :valid[s]]).any()
        assert np.isnan(a.kv[0, s, :, :, valid[s]:]).all()
