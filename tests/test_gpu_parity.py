"""GPU parity: the HIP library (through its C-ABI) against the float64 oracle.

Tolerances (per tensor, max |gpu - oracle| / max |oracle|): 2e-2 for bf16
runs, 1e-4 for fp32 runs.  KV indexing is checked bit-exactly: exactly the
oracle's (layer, slot, position) entries change, every other element keeps
its bit pattern (including the NaN sentinel of empty positions, so an
over-read would also poison the outputs)."""
import dataclasses

import numpy as np
import pytest

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from gpu_harness import (TOL, DeviceModel, assert_checks, bits_of, compare_layer, delta_err, from_dev,  # noqa: E402
                         log, oracle_batch, rel_err, to_dev)
from paper_2308_16369_amd import sarathi as S  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _lib():
    # On a GPU machine the library must be there: no fallback exists.
    S.lib()


def run_and_check(inst: wl.HostInstance, label: str, layer: int = 0):
    log(f"{label}: T={inst.batch.n_tokens} C={inst.batch.chunk_len}@{inst.batch.chunk_offset} "
        f"B={inst.batch.n_decodes} dtype={inst.shape.dtype}")
    dm = DeviceModel(inst)
    x = to_dev(inst.x, inst.shape.dtype)
    before = bits_of(dm.kv_dev)
    y = dm.layer(layer, inst.batch, x)
    torch.cuda.synchronize()
    ref = oracle.layer_forward(inst.shape, inst.weights[layer], inst.kv[layer].copy(), oracle_batch(inst.batch),
                               inst.x)
    checks = compare_layer(dm, layer, inst.batch, inst.x.astype(np.float64), y, before, inst.kv[layer], ref)
    assert_checks(checks, label)
    assert np.all(np.isfinite(from_dev(y)))


# ============================================================================ linear ops

LIN_SHAPES = [(72, 200, 264), (320, 640, 512), (283, 1000, 1032), (5, 17, 8), (544, 384, 256), (160, 128, 64),
              (300, 5120, 2048)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kind", [S.LINEAR_PLAIN, S.LINEAR_RESID, S.LINEAR_RESID_F32IN, S.LINEAR_SWIGLU,
                                  S.LINEAR_GELU])
@pytest.mark.parametrize("mnk", LIN_SHAPES)
def test_linear_matches_oracle(dtype, kind, mnk):
    M, N, K = mnk
    rng = np.random.default_rng(M * 7 + N * 3 + K + kind)
    st = (lambda a: wl.round_to_bf16(a)) if dtype == "bf16" else (lambda a: a.astype(np.float32))
    x = st(rng.standard_normal((M, K)).astype(np.float32))
    wrows = 2 * N if kind == S.LINEAR_SWIGLU else N
    w = st((rng.standard_normal((wrows, K)) * 0.05).astype(np.float32))
    resid = rng.standard_normal((M, N)).astype(np.float32)
    if kind == S.LINEAR_RESID:
        resid = st(resid)
    z = oracle.linear(x, w)
    if kind == S.LINEAR_PLAIN:
        ref = z
    elif kind in (S.LINEAR_RESID, S.LINEAR_RESID_F32IN):
        ref = resid.astype(np.float64) + z
    elif kind == S.LINEAR_SWIGLU:
        ref = oracle.silu(z[:, :N]) * z[:, N:]
    else:
        ref = oracle.gelu(z)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    rd = to_dev(resid, dtype) if kind == S.LINEAR_RESID else torch.from_numpy(resid).cuda()
    out = torch.empty((M, N), dtype=torch.float32 if kind == S.LINEAR_RESID else tdt, device="cuda")
    scratch = torch.empty(S.sarathi_linear_scratch_bytes(M, N), dtype=torch.uint8, device="cuda")
    S.sarathi_linear(S.BF16 if dtype == "bf16" else S.F32, kind, M, N, K, xd.data_ptr(), wd.data_ptr(),
                     rd.data_ptr() if kind in (S.LINEAR_RESID, S.LINEAR_RESID_F32IN) else 0, out.data_ptr(),
                     scratch.data_ptr(), scratch.numel(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    got = from_dev(out)
    err = rel_err(got, ref)
    if kind in (S.LINEAR_RESID, S.LINEAR_RESID_F32IN):
        out_dt = "f32" if kind == S.LINEAR_RESID else dtype
        err = max(err, delta_err(got, ref, z, out_dt))
    log(f"linear {dtype} kind {kind} {mnk}: err {err:.3e}")
    assert err <= TOL[dtype]


TILE_SHAPES = [(37, 456, 1024), (200, 456, 1024)]


@pytest.mark.parametrize("mnk", TILE_SHAPES)
def test_linear_every_tile_shape(mnk):
    """Every tile shape of the bf16 matmul kernel, with every epilogue (and
    3 K-splits for the residual kinds), against the oracle on ragged shapes."""
    M, N, K = mnk
    n_tiles = S.sarathi_linear_tile_count()
    rng = np.random.default_rng(M + N + K)
    x = wl.round_to_bf16(rng.standard_normal((M, K)).astype(np.float32))
    w = wl.round_to_bf16((rng.standard_normal((2 * N, K)) * 0.05).astype(np.float32))
    resid = rng.standard_normal((M, N)).astype(np.float32)
    resid_bf = wl.round_to_bf16(resid)
    z2 = oracle.linear(x, w)
    z = z2[:, :N]
    xd, wd = to_dev(x, "bf16"), to_dev(w, "bf16")
    rd_bf, rd_f32 = to_dev(resid_bf, "bf16"), torch.from_numpy(resid).cuda()
    scratch = torch.empty(S.sarathi_linear_scratch_bytes(M, N), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    refs = {S.LINEAR_PLAIN: z, S.LINEAR_RESID: resid_bf.astype(np.float64) + z,
            S.LINEAR_RESID_F32IN: resid.astype(np.float64) + z,
            S.LINEAR_SWIGLU: oracle.silu(z2[:, :N]) * z2[:, N:], S.LINEAR_GELU: oracle.gelu(z)}
    for tile in range(n_tiles):
        for kind, ref in refs.items():
            for n_split in ((1, 3) if kind in (S.LINEAR_RESID, S.LINEAR_RESID_F32IN) else (1,)):
                out = torch.full((M, N), float("nan"), device="cuda",
                                 dtype=torch.float32 if kind == S.LINEAR_RESID else torch.bfloat16)
                rd = rd_bf if kind == S.LINEAR_RESID else rd_f32
                S.sarathi_linear_tiled(kind, M, N, K, xd.data_ptr(), wd.data_ptr(),
                                       rd.data_ptr() if kind in (S.LINEAR_RESID, S.LINEAR_RESID_F32IN) else 0,
                                       out.data_ptr(), scratch.data_ptr(), scratch.numel(), tile, n_split, stream)
                torch.cuda.synchronize()
                got = from_dev(out)
                err = rel_err(got, ref)
                if kind in (S.LINEAR_RESID, S.LINEAR_RESID_F32IN):
                    err = max(err, delta_err(got, ref, z, "f32" if kind == S.LINEAR_RESID else "bf16"))
                label = f"tile {S.sarathi_linear_tile_shape(tile)} kind {kind} split {n_split} {mnk}"
                log(f"{label}: err {err:.3e}")
                assert np.all(np.isfinite(got)), label
                assert err <= TOL["bf16"], label


@pytest.mark.parametrize("kind", [S.LINEAR_RESID, S.LINEAR_RESID_F32IN])
def test_linear_split_k_deterministic(kind):
    """Split-K (small M, large K) gives bit-identical results run to run, and
    agrees with the unsplit op (no scratch) to fp32 summation order."""
    M, N, K = 48, 5120, 13824
    rng = np.random.default_rng(11 + kind)
    x = wl.round_to_bf16(rng.standard_normal((M, K)).astype(np.float32))
    w = wl.round_to_bf16((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
    resid = rng.standard_normal((M, N)).astype(np.float32)
    if kind == S.LINEAR_RESID:
        resid = wl.round_to_bf16(resid)
    xd, wd = to_dev(x, "bf16"), to_dev(w, "bf16")
    rd = to_dev(resid, "bf16") if kind == S.LINEAR_RESID else torch.from_numpy(resid).cuda()
    odt = torch.float32 if kind == S.LINEAR_RESID else torch.bfloat16
    scratch = torch.empty(S.sarathi_linear_scratch_bytes(M, N), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    outs = []
    for use_scratch in (True, True, False):
        out = torch.full((M, N), float("nan"), dtype=odt, device="cuda")
        S.sarathi_linear(S.BF16, kind, M, N, K, xd.data_ptr(), wd.data_ptr(), rd.data_ptr(), out.data_ptr(),
                         scratch.data_ptr() if use_scratch else 0, scratch.numel() if use_scratch else 0, stream)
        outs.append(out)
    torch.cuda.synchronize()
    assert np.array_equal(bits_of(outs[0]), bits_of(outs[1])), "split-K result differs between runs"
    ref = resid.astype(np.float64) + oracle.linear(x, w)
    for o in outs[0], outs[2]:
        err = rel_err(from_dev(o), ref)
        log(f"split-K kind {kind}: err {err:.3e}")
        assert err <= TOL["bf16"]


@pytest.mark.parametrize("kind", [S.LINEAR_RESID, S.LINEAR_RESID_F32IN])
@pytest.mark.parametrize("mnk", [(72, 256, 688), (5, 17, 1000), (130, 200, 4104)])
def test_linear_split_k_fp32(kind, mnk):
    """fp32 residual ops split over K when their 64x64 tiles leave most CUs
    idle (ragged last split included): bit-identical run to run, and both
    the split and the unsplit op (no scratch) within the fp32 tolerance."""
    M, N, K = mnk
    rng = np.random.default_rng(M + N + K + kind)
    x = rng.standard_normal((M, K)).astype(np.float32)
    w = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    resid = rng.standard_normal((M, N)).astype(np.float32)
    xd, wd, rd = (torch.from_numpy(a).cuda() for a in (x, w, resid))
    scratch = torch.empty(S.sarathi_linear_scratch_bytes(M, N), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    outs = []
    for use_scratch in (True, True, False):
        out = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        S.sarathi_linear(S.F32, kind, M, N, K, xd.data_ptr(), wd.data_ptr(), rd.data_ptr(), out.data_ptr(),
                         scratch.data_ptr() if use_scratch else 0, scratch.numel() if use_scratch else 0, stream)
        outs.append(out)
    torch.cuda.synchronize()
    assert np.array_equal(bits_of(outs[0]), bits_of(outs[1])), "split-K result differs between runs"
    ref = resid.astype(np.float64) + oracle.linear(x, w)
    for o in outs[0], outs[2]:
        err = rel_err(from_dev(o), ref)
        log(f"fp32 split-K kind {kind} {mnk}: err {err:.3e}")
        assert err <= TOL["f32"]


# ============================================================================ whole layer

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_layer_tiny_workload(dtype):
    w = wl.TINY if dtype == "f32" else wl.with_dtype(wl.TINY, "bf16")
    run_and_check(wl.generate(w), f"tiny layer {dtype}")


def _tiny_shape(dtype, **kw):
    return dataclasses.replace(wl.TINY.shape, dtype=dtype, **kw)


EDGE = {
    # name: (prefill_slot, offset, C, decode_slots, decode_ctx, S, n_slots)
    "decode_only": (-1, 0, 0, [3, 0, 7, 5, 1, 2, 8, 6], [32, 77, 128, 0, 5, 250, 64, 100], 256, 9),
    "prefill_only": (4, 128, 64, [], [], 256, 9),
    "prefill_from_zero": (2, 0, 64, [0, 5, 8], [10, 1, 63], 256, 9),
    "ragged_chunk": (6, 100, 37, [1, 2, 3, 4, 5], [7, 99, 128, 200, 33], 256, 9),
    "single_token_chunk": (0, 200, 1, [1, 2], [31, 64], 256, 9),
    "full_cache": (1, 192, 64, [0, 2, 3], [255, 254, 0], 256, 9),
    "multi_split_decodes": (3, 700, 200, list(range(4, 20)),
                            [256, 257, 511, 512, 513, 1000, 1087, 300, 640, 768, 900, 1023, 1024, 1050, 600, 700],
                            1088, 20),
    "many_decodes_bf16_tail": (-1, 0, 0, list(range(1, 70)), [(37 * i) % 300 for i in range(1, 70)], 320, 71),
}


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", list(EDGE))
def test_layer_edge_cases(dtype, case):
    ps, off, C, ds, dc, S_, ns = EDGE[case]
    b = wl.Batch(prefill_slot=ps, chunk_offset=off, chunk_len=C, decode_slots=np.array(ds, np.int32),
                 decode_ctx=np.array(dc, np.int32))
    inst = wl.make_instance(_tiny_shape(dtype), b, max_seq_len=S_, n_slots=ns, seed=11)
    run_and_check(inst, f"edge {case} {dtype}")


def test_layer_gpt_style_tiny_bf16():
    shape = _tiny_shape("bf16", norm="layer", act="gelu", rope=False, eps=1e-5)
    b = wl.Batch(prefill_slot=0, chunk_offset=64, chunk_len=100, decode_slots=np.array([1, 2, 3], np.int32),
                 decode_ctx=np.array([5, 150, 255], np.int32))
    run_and_check(wl.make_instance(shape, b, max_seq_len=256, n_slots=4, seed=3), "gpt-style tiny bf16")


def test_layer_head_dim_128_tiny_bf16():
    shape = _tiny_shape("bf16", hidden=512, n_heads=4, head_dim=128, ffn=1376)
    b = wl.Batch(prefill_slot=2, chunk_offset=300, chunk_len=130, decode_slots=np.array([0, 1, 3], np.int32),
                 decode_ctx=np.array([0, 511, 258], np.int32))
    run_and_check(wl.make_instance(shape, b, max_seq_len=512, n_slots=4, seed=5), "hd128 tiny bf16")


# (heads, head_dim, chunk rows, decodes, preproj tile the planner picks): the
# fused RoPE + KV-append epilogue on every producer/consumer tile width,
# including tiles that cut heads (BN 192 and 224 against 128-wide heads) and
# a ragged last column tile
ROPE_TILES = [(40, 128, 4, 4, (64, 64)), (52, 128, 5, 3, (64, 128)), (52, 128, 66, 4, (96, 128)),
              (52, 128, 96, 4, (96, 192)), (52, 128, 190, 10, (160, 192)), (52, 128, 330, 10, (160, 256)),
              (52, 128, 790, 10, (160, 224)), (104, 64, 790, 10, (160, 224))]


@pytest.mark.parametrize("nh,hd,C,B,tile", ROPE_TILES)
def test_layer_rope_epilogue_every_tile(nh, hd, C, B, tile):
    """q, k_new and v_new from preproj's fused rotary + KV-append epilogue
    against the oracle, on wide-QKV layers whose row counts make the planner
    pick each tile shape."""
    # the FFN about as wide as the attention output, so that y - hres (the FFN
    # output) is not small beside the error that postproj's long sum puts on h
    shape = _tiny_shape("bf16", hidden=512, n_heads=nh, head_dim=hd, ffn=4096)
    T = C + B
    assert tuple(S.sarathi_linear_plan(S.BF16, S.LINEAR_PLAIN, T, 3 * nh * hd, 512, 0)[:2]) == tile
    b = wl.Batch(prefill_slot=0, chunk_offset=17, chunk_len=C, decode_slots=np.arange(1, B + 1, dtype=np.int32),
                 decode_ctx=np.array([(53 * i) % 1000 for i in range(1, B + 1)], np.int32))
    run_and_check(wl.make_instance(shape, b, max_seq_len=1024, n_slots=B + 1, seed=23),
                  f"rope epilogue nh={nh} hd={hd} T={T} tile={tile}")


@pytest.mark.parametrize("dtype,hidden,norm", [("bf16", 24576, "rms"), ("bf16", 12296, "layer"), ("bf16", 4104, "rms"),
                                               ("f32", 12288, "layer"), ("f32", 1032, "rms")])
def test_layer_wide_hidden(dtype, hidden, norm):
    """Rows as wide as the configuration accepts (the norms keep a row in
    registers; the register footprint is picked from the row width), plus
    widths just past a size step, for RMSNorm and LayerNorm."""
    shape = _tiny_shape(dtype, hidden=hidden, n_heads=2, head_dim=64, ffn=256, norm=norm,
                        act="gelu" if norm == "layer" else "swiglu", rope=norm == "rms",
                        eps=1e-5 if norm == "layer" else 1e-6)
    b = wl.Batch(prefill_slot=0, chunk_offset=9, chunk_len=5, decode_slots=np.array([1, 2], np.int32),
                 decode_ctx=np.array([3, 40], np.int32))
    run_and_check(wl.make_instance(shape, b, max_seq_len=64, n_slots=3, seed=17), f"wide hidden {hidden} {norm}")


@pytest.mark.parametrize("C,off,decodes", [(2048, 0, []), (1000, 2048, [(0, 3047), (2, 17)])])
def test_layer_long_chunk_bf16(C, off, decodes):
    """Chunks as long as the full prefills of the chunk-size ablation (a
    2048-token prompt in one call; a 1000-row chunk after 2048 cached
    positions with decodes beside it), head_dim 128."""
    shape = _tiny_shape("bf16", hidden=512, n_heads=4, head_dim=128, ffn=1376)
    b = wl.Batch(prefill_slot=1, chunk_offset=off, chunk_len=C,
                 decode_slots=np.array([d[0] for d in decodes], np.int32),
                 decode_ctx=np.array([d[1] for d in decodes], np.int32))
    run_and_check(wl.make_instance(shape, b, max_seq_len=3072, n_slots=3, seed=41), f"long chunk {C}@{off}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_layer_long_contexts(dtype):
    """Contexts of tens of thousands of keys: decodes of 65 and 137 512-key
    splits (the combine pass reads a row's partials 64 splits at a time, so
    this crosses one and two of its chunk boundaries) and a 100-row chunk
    after 50000 cached positions (its query blocks cut ~780 key tiles into
    ranges)."""
    S_ = 70016
    shape = _tiny_shape(dtype, hidden=128, n_heads=2, head_dim=64, ffn=256)
    b = wl.Batch(prefill_slot=1, chunk_offset=50000, chunk_len=100, decode_slots=np.array([3, 0], np.int32),
                 decode_ctx=np.array([69999, 33000], np.int32))
    run_and_check(wl.make_instance(shape, b, max_seq_len=S_, n_slots=4, seed=29), f"long contexts {dtype}")


def test_layer_max_cache_length_bf16():
    """The longest cache the library accepts (2^20 positions): a decode at
    the last position (2048 key splits) and an 8-row chunk ending there
    (16384 key tiles for its query block)."""
    S_ = 1 << 20
    shape = _tiny_shape("bf16", hidden=64, n_heads=1, head_dim=64, ffn=128)
    b = wl.Batch(prefill_slot=1, chunk_offset=S_ - 8, chunk_len=8, decode_slots=np.array([0], np.int32),
                 decode_ctx=np.array([S_ - 1], np.int32))
    run_and_check(wl.make_instance(shape, b, max_seq_len=S_, n_slots=2, seed=31), "max cache length bf16")


MIXED = {
    # name: (chunks [(slot, offset, len)], decodes [(slot, ctx)], max_seq_len, n_slots)
    "three_chunks_and_decodes": ([(2, 100, 37), (0, 0, 64), (5, 190, 65)], [(1, 77), (3, 0), (7, 250)], 256, 9),
    "chunks_only": ([(4, 0, 1), (6, 255, 1), (8, 128, 100)], [], 256, 9),
    "many_small_chunks": ([(i, 3 * i, 5 + i) for i in range(6)], [(7, 10), (8, 200)], 256, 9),
    "long_and_split": ([(0, 300, 200), (1, 0, 129)], [(2, 511), (3, 256)], 512, 4),
}


def run_mixed_and_check(inst, label, layer=0):
    b = inst.batch
    log(f"{label}: T={b.n_tokens} chunks={b.chunks} B={b.n_decodes} dtype={inst.shape.dtype}")
    dm = DeviceModel(inst, max_chunks=max(1, len(b.chunks)))
    x = to_dev(inst.x, inst.shape.dtype)
    before = bits_of(dm.kv_dev)
    y = dm.mixed_layer(layer, b, x)
    torch.cuda.synchronize()
    ref = oracle.layer_forward(inst.shape, inst.weights[layer], inst.kv[layer].copy(), oracle_batch(b), inst.x)
    checks = compare_layer(dm, layer, b, inst.x.astype(np.float64), y, before, inst.kv[layer], ref)
    assert_checks(checks, label)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", list(MIXED))
def test_mixed_batch_layer(dtype, case):
    """Several prompt chunks in one layer call (Sec. 5.2's mixed batching):
    each chunk attends over its own slot, decodes over theirs."""
    chunks, decs, S_, ns = MIXED[case]
    shape = _tiny_shape(dtype, hidden=512, n_heads=4, head_dim=128, ffn=1376) if case == "long_and_split" \
        else _tiny_shape(dtype)
    b = wl.MixedBatch(chunks=chunks, decode_slots=np.array([d[0] for d in decs], np.int32),
                      decode_ctx=np.array([d[1] for d in decs], np.int32))
    run_mixed_and_check(wl.make_instance(shape, b, max_seq_len=S_, n_slots=ns, seed=17), f"mixed {case} {dtype}")


def _random_batch(rng, S_, n_slots, mixed):
    """A random batch over distinct slots: 0-3 prompt chunks (at most one for
    the hybrid entry point) at random offsets and lengths, 0-79 decodes at
    random context lengths, at least one row."""
    slots = rng.permutation(n_slots)
    k = int(rng.integers(0, 4)) if mixed else int(rng.integers(0, 2))
    chunks = []
    for i in range(k):
        n = int(rng.choice([1, int(rng.integers(2, 130)), int(rng.integers(130, 400))]))
        off = int(rng.integers(0, S_ - n + 1))
        chunks.append((int(slots[i]), off, n))
    B = int(rng.integers(0 if k else 1, 80))
    ctx = rng.integers(0, S_, size=B)
    ctx[: B // 4] = rng.choice([0, 511, 512, 1023, S_ - 1], size=B // 4)   # split boundaries and the ends
    ds = np.array(slots[k:k + B], np.int32)
    if mixed:
        return wl.MixedBatch(chunks=chunks, decode_slots=ds, decode_ctx=np.array(ctx, np.int32))
    ps, off, C = chunks[0] if chunks else (-1, 0, 0)
    return wl.Batch(prefill_slot=ps, chunk_offset=off, chunk_len=C, decode_slots=ds,
                    decode_ctx=np.array(ctx, np.int32))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seed", range(8))
def test_random_batches(dtype, seed):
    """Seeded random batches through both entry points (hybrid: one chunk or
    none; mixed: up to three), head_dim 64 and 128, a cache of 1100
    positions so decodes cross 512-key splits and chunks span many key
    tiles; every output, intermediate and KV entry against the oracle."""
    rng = np.random.default_rng(1000 + seed)
    mixed = seed % 2 == 1
    hd128 = seed % 3 != 0
    shape = _tiny_shape(dtype, hidden=512, n_heads=4, head_dim=128, ffn=1376) if hd128 else _tiny_shape(dtype)
    S_, ns = 1100, 84
    b = _random_batch(rng, S_, ns, mixed)
    inst = wl.make_instance(shape, b, max_seq_len=S_, n_slots=ns, seed=2000 + seed)
    label = f"random {'mixed' if mixed else 'hybrid'} seed {seed} hd {shape.head_dim} {dtype}"
    if mixed:
        run_mixed_and_check(inst, label)
    else:
        run_and_check(inst, label)


def test_mixed_model_step_three_layers_bf16():
    shape = dataclasses.replace(_tiny_shape("bf16"), n_layers=3)
    chunks, decs, S_, ns = MIXED["three_chunks_and_decodes"]
    b = wl.MixedBatch(chunks=chunks, decode_slots=np.array([d[0] for d in decs], np.int32),
                      decode_ctx=np.array([d[1] for d in decs], np.int32))
    inst = wl.make_instance(shape, b, max_seq_len=S_, n_slots=ns, seed=23, n_layers=3)
    dm = DeviceModel(inst, max_chunks=3)
    y = dm.mixed_step(b, to_dev(inst.x, "bf16"))
    torch.cuda.synchronize()
    okv = inst.kv.astype(np.float64)
    outs = oracle.model_step(shape, inst.weights, okv, oracle_batch(b), inst.x)
    err = rel_err(from_dev(y), outs[-1].y)
    log(f"mixed model step bf16: y {err:.3e}")
    assert err <= TOL["bf16"]


# ============================================================================ method invariants on the GPU

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_chunked_prefill_on_gpu_matches_one_shot_oracle(dtype):
    """Chunks of a prompt through the library (KV grown in place between
    calls) against the oracle's one-shot causal prefill (Sec. 4.2)."""
    shape = _tiny_shape(dtype)
    P, C = 256, 64
    b_full = wl.Batch(prefill_slot=1, chunk_offset=0, chunk_len=P, decode_slots=np.zeros(0, np.int32),
                      decode_ctx=np.zeros(0, np.int32))
    inst = wl.make_instance(shape, b_full, max_seq_len=P, n_slots=2, seed=21)
    ref = oracle.layer_forward(shape, inst.weights[0], inst.kv[0].copy(), oracle_batch(b_full), inst.x)
    dm = DeviceModel(inst, max_tokens=C)
    ys = []
    for off in range(0, P, C):
        b = wl.Batch(prefill_slot=1, chunk_offset=off, chunk_len=C, decode_slots=np.zeros(0, np.int32),
                     decode_ctx=np.zeros(0, np.int32))
        ys.append(from_dev(dm.layer(0, b, to_dev(inst.x[off:off + C], dtype))))
    torch.cuda.synchronize()
    err = rel_err(np.concatenate(ys), ref.y)
    kv = from_dev(dm.kv_dev)[0, 1, :, :, :P]
    kerr = rel_err(kv[0], ref.k_new.transpose(1, 0, 2))
    verr = rel_err(kv[1], ref.v_new.transpose(1, 0, 2))
    log(f"chunked prefill {dtype}: y {err:.3e} k {kerr:.3e} v {verr:.3e}")
    assert max(err, kerr, verr) <= TOL[dtype]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_model_step_consecutive_steps(dtype):
    """Three consecutive decode-maximal steps through a 3-layer stack: chunks
    at offsets 0, 64, 128 of a prompt, decodes advancing one position per
    step, the KV grown in place by the library; compared with the oracle run
    the same way on its own cache."""
    shape = dataclasses.replace(_tiny_shape(dtype), n_layers=3)
    L, Sx, n_slots = 3, 256, 6
    b0 = wl.Batch(prefill_slot=2, chunk_offset=0, chunk_len=64, decode_slots=np.array([0, 4, 5, 1], np.int32),
                  decode_ctx=np.array([10, 100, 0, 191], np.int32))
    inst = wl.make_instance(shape, b0, max_seq_len=Sx, n_slots=n_slots, seed=31, n_layers=L)
    dm = DeviceModel(inst)
    okv = inst.kv.astype(np.float64)
    rng = np.random.default_rng(5)
    for step in range(3):
        b = wl.Batch(prefill_slot=2, chunk_offset=64 * step, chunk_len=64, decode_slots=b0.decode_slots,
                     decode_ctx=b0.decode_ctx + step)
        xs = inst.x if step == 0 else (wl.round_to_bf16 if dtype == "bf16" else np.float32)(
            rng.standard_normal(inst.x.shape).astype(np.float32))
        xs = np.asarray(xs, np.float32)
        before = bits_of(dm.kv_dev)
        y = dm.step(b, to_dev(xs, dtype))
        torch.cuda.synchronize()
        outs = oracle.model_step(shape, inst.weights, okv, oracle_batch(b), xs)
        after = bits_of(dm.kv_dev)
        written = np.zeros(after.shape, bool)
        for layer in range(L):
            for s, p in zip(outs[layer].slots, outs[layer].positions):
                written[layer, s, :, :, p, :] = True
        assert np.array_equal(after[~written], before[~written]), "KV changed outside the new positions"
        kvf = from_dev(dm.kv_dev)
        err_kv = rel_err(kvf[written], okv[written])
        err_y = rel_err(from_dev(y), outs[-1].y)
        log(f"model_step {dtype} step {step}: y {err_y:.3e} kv {err_kv:.3e}")
        assert err_y <= TOL[dtype] and err_kv <= TOL[dtype]


def test_model_step_forty_layers_f32_chained():
    """A 40-layer fp32 stack (tiny layer shapes) over two consecutive steps
    through sarathi_model_step: every layer's output, run layer by layer on
    the same batch, against the oracle chained through all 40 layers on its
    own outputs (one iteration of the model, Sec. 4.5), at the fp32
    tolerance; the model step equals the layer-by-layer run bit for bit; the
    K/V written at every layer matches the oracle's."""
    L, Sx, n_slots = 40, 256, 6
    shape = dataclasses.replace(_tiny_shape("f32"), n_layers=L)
    b0 = wl.Batch(prefill_slot=3, chunk_offset=0, chunk_len=48, decode_slots=np.array([0, 5, 1], np.int32),
                  decode_ctx=np.array([7, 130, 64], np.int32))
    inst = wl.make_instance(shape, b0, max_seq_len=Sx, n_slots=n_slots, seed=41, n_layers=L)
    dm = DeviceModel(inst)
    okv = inst.kv.astype(np.float64)
    rng = np.random.default_rng(9)
    for step in range(2):
        b = wl.Batch(prefill_slot=3, chunk_offset=48 * step, chunk_len=48, decode_slots=b0.decode_slots,
                     decode_ctx=b0.decode_ctx + step)
        xs = inst.x if step == 0 else rng.standard_normal(inst.x.shape).astype(np.float32)
        x_dev = to_dev(xs, "f32")
        y_ms = dm.step(b, x_dev)
        hs = [x_dev]
        for layer in range(L):
            hs.append(dm.layer(layer, b, hs[-1]))
        torch.cuda.synchronize()
        assert torch.equal(y_ms, hs[-1]), "model step differs from the layer-by-layer run"
        outs = oracle.model_step(shape, inst.weights, okv, oracle_batch(b), xs)
        errs = [rel_err(from_dev(hs[layer + 1]), outs[layer].y) for layer in range(L)]
        kvf = from_dev(dm.kv_dev)
        kv_errs = []
        for layer in range(L):
            got = np.stack([kvf[layer, s, :, :, p, :] for s, p in zip(outs[layer].slots, outs[layer].positions)])
            kv_errs.append(rel_err(got[:, 0], outs[layer].k_new))
            kv_errs.append(rel_err(got[:, 1], outs[layer].v_new))
        log(f"40-layer f32 step {step}: y error by layer (first, 20th, last) {errs[0]:.2e} {errs[19]:.2e} "
            f"{errs[-1]:.2e}; max over layers {max(errs):.2e}; K/V max {max(kv_errs):.2e}")
        assert max(errs) <= TOL["f32"] and max(kv_errs) <= TOL["f32"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_piggybacked_decode_equals_decode_alone(dtype):
    """Sec. 4.3: a decode piggybacked on a chunk gives the same row as the same
    decode run alone (both against the oracle and against each other)."""
    shape = _tiny_shape(dtype)
    b = wl.Batch(prefill_slot=0, chunk_offset=64, chunk_len=64, decode_slots=np.array([1, 2, 3], np.int32),
                 decode_ctx=np.array([40, 200, 3], np.int32))
    inst = wl.make_instance(shape, b, max_seq_len=256, n_slots=4, seed=41)
    dm = DeviceModel(inst)
    y_h = from_dev(dm.layer(0, b, to_dev(inst.x, dtype)))
    for i in range(3):
        dm.kv_dev.copy_(to_dev(inst.kv, dtype))
        bi = wl.Batch(prefill_slot=-1, chunk_offset=0, chunk_len=0, decode_slots=b.decode_slots[i:i + 1],
                      decode_ctx=b.decode_ctx[i:i + 1])
        y_a = from_dev(dm.layer(0, bi, to_dev(inst.x[64 + i:65 + i], dtype)))
        err = rel_err(y_h[64 + i:65 + i], y_a)
        log(f"piggyback {dtype} decode {i}: {err:.3e}")
        assert err <= TOL[dtype]


# ============================================================================ paper-shaped workloads

def test_layer_llama13b_workload():
    run_and_check(wl.generate(wl.LLAMA13B_LAYER), "llama13b layer c256 b64")


@pytest.mark.parametrize("chunk", [128, 256, 512])
def test_layer_llama33b_workloads(chunk):
    run_and_check(wl.generate(wl.llama33b_layer(chunk)), f"llama33b layer c{chunk} b32")


def test_layer_gpt3_workload():
    run_and_check(wl.generate(wl.GPT3_LAYER), "gpt3 layer c256 b27")
