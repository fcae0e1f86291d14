"""Host-side tests of the C-ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments on the host before any launch
(no GPU needed: every call here fails validation before touching HIP)."""
import ctypes as ct
import glob
import os
import re

import pytest

from paper_2308_16369_amd import sarathi as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))

FAKE_DEV = 0x10000          # never dereferenced: validation fails first


def header_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(sarathi_[a-z_0-9]+)\s*\(", text))
    return sorted(names)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(S.LIB_PATH):
        pytest.fail("libsarathi.so is not built (python -m paper_2308_16369_amd.build)")
    return S.lib()


def test_exports_every_declared_symbol(lib):
    names = header_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), f"{n} declared in include/*.h but not exported"
        assert n in S.EXPORTS, f"{n} has no binding"
    assert S.sarathi_version() == 1


def tiny_cfg(**kw):
    base = dict(hidden=256, n_heads=4, head_dim=64, ffn=688, n_layers=2, dtype=S.F32)
    base.update(kw)
    return S.make_cfg(**base)


def test_kv_bytes_and_strides(lib):
    cfg = tiny_cfg()
    n = S.sarathi_kv_bytes(cfg, 9, 256)
    assert n == 2 * 9 * 2 * 4 * 256 * 64 * 4
    kv = S.sarathi_kv_alloc(cfg, 9, 256, FAKE_DEV, n)
    st = kv.strides()
    assert (st.pos, st.head, st.kv, st.slot, st.layer) == (64, 256 * 64, 4 * 256 * 64, 2 * 4 * 256 * 64,
                                                            9 * 2 * 4 * 256 * 64)
    kv.free()
    assert S.sarathi_kv_bytes(tiny_cfg(head_dim=96), 9, 256) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=96), S.EUNSUPPORTED), (dict(dtype=7), S.EUNSUPPORTED), (dict(hidden=250), S.EUNSUPPORTED),
    (dict(ffn=690), S.EUNSUPPORTED), (dict(n_layers=0), S.EINVAL), (dict(eps=0.0), S.EINVAL),
    (dict(norm=3), S.EUNSUPPORTED), (dict(act=5), S.EUNSUPPORTED), (dict(rope_base=0.5), S.EINVAL),
])
def test_kv_alloc_rejects_bad_cfg(lib, kw, code):
    cfg = tiny_cfg(**kw)
    h = ct.c_void_p()
    rc = lib.sarathi_kv_alloc(ct.byref(cfg), 9, 256, ct.c_void_p(FAKE_DEV), 1 << 30, ct.byref(h))
    assert rc == code, S.sarathi_last_error()
    assert S.sarathi_last_error()


def test_kv_alloc_rejects_small_memory_and_nulls(lib):
    cfg = tiny_cfg()
    h = ct.c_void_p()
    need = S.sarathi_kv_bytes(cfg, 9, 256)
    assert lib.sarathi_kv_alloc(ct.byref(cfg), 9, 256, ct.c_void_p(FAKE_DEV), need - 1, ct.byref(h)) == S.ENOSPC
    assert lib.sarathi_kv_alloc(ct.byref(cfg), 9, 256, None, need, ct.byref(h)) == S.EINVAL
    assert lib.sarathi_kv_alloc(ct.byref(cfg), 0, 256, ct.c_void_p(FAKE_DEV), need, ct.byref(h)) == S.EINVAL
    assert lib.sarathi_kv_alloc(None, 9, 256, ct.c_void_p(FAKE_DEV), need, ct.byref(h)) == S.EINVAL
    assert lib.sarathi_kv_alloc(ct.byref(cfg), 9, 256, ct.c_void_p(FAKE_DEV + 2), need, ct.byref(h)) == S.EINVAL
    # the largest accepted cache length (positions < 2^20) and the first rejected one
    top = S.sarathi_kv_bytes(cfg, 1, 1 << 20)
    assert lib.sarathi_kv_alloc(ct.byref(cfg), 1, 1 << 20, ct.c_void_p(FAKE_DEV), top, ct.byref(h)) == S.OK
    lib.sarathi_kv_free(h)
    assert lib.sarathi_kv_alloc(ct.byref(cfg), 1, (1 << 20) + 1, ct.c_void_p(FAKE_DEV), 2 * top,
                                ct.byref(h)) == S.EINVAL
    assert lib.sarathi_kv_alloc(ct.byref(cfg), (1 << 20) + 1, 1, ct.c_void_p(FAKE_DEV), 1 << 40, ct.byref(h)) == S.EINVAL


def test_workspace_layout_is_consistent(lib):
    cfg = tiny_cfg(dtype=S.BF16)
    L = S.sarathi_workspace_layout(cfg, 72, 8, 256)
    assert L.total == S.sarathi_workspace_bytes(cfg, 72, 8, 256) > 0
    offs = [L.a, L.qkv, L.o, L.hres, L.m]
    assert offs == sorted(offs) and all(o % 256 == 0 for o in offs)
    assert L.qkv - L.a >= 72 * 256 * 2 and L.o - L.qkv >= 72 * 3 * 256 * 2
    with pytest.raises(S.SarathiError):
        S.sarathi_workspace_layout(cfg, 0, 0, 256)


# --------------------------------------------------------------------------- forward validation

class Setup:
    def __init__(self, lib, n_slots=9, S_=256, dtype=S.F32):
        self.cfg = tiny_cfg(dtype=dtype)
        self.kv = S.sarathi_kv_alloc(self.cfg, n_slots, S_, FAKE_DEV, S.sarathi_kv_bytes(self.cfg, n_slots, S_))
        self.w = S.make_weights({k: FAKE_DEV for k in ("norm1_g", "norm1_b", "w_qkv", "w_o", "norm2_g", "norm2_b",
                                                       "w_up", "w_down")})
        self.ws_bytes = S.sarathi_workspace_bytes(self.cfg, 128, 64, S_)

    def call(self, batch, layer=0, x_in=0x200000, x_out=0x300000, ws=0x40000000, ws_bytes=None, w=None, cfg=None):
        b, keep = batch
        return S.sarathi_hybrid_layer_forward(cfg or self.cfg, w or self.w, self.kv, layer, b, x_in, x_out, ws,
                                              self.ws_bytes if ws_bytes is None else ws_bytes, check=False)


@pytest.mark.parametrize("batch,code", [
    ((0, 0, 0, [], []), S.EINVAL),                       # empty batch
    ((9, 0, 4, [], []), S.EINVAL),                       # prefill slot out of range
    ((-1, 0, 4, [], []), S.EINVAL),
    ((1, -1, 4, [], []), S.ERANGE),                      # negative offset
    ((1, 250, 7, [], []), S.ERANGE),                     # offset + C > max_seq_len
    ((1, 0, -2, [], []), S.ERANGE),                      # negative chunk
    ((1, 0, 4, [2, 2], [3, 4]), S.EINVAL),               # duplicate decode slot
    ((1, 0, 4, [1], [3]), S.EINVAL),                     # decode slot == prefill slot
    ((1, 0, 4, [9], [3]), S.EINVAL),                     # decode slot out of range
    ((1, 0, 4, [3], [-1]), S.ERANGE),                    # negative context
    ((1, 0, 4, [3], [256]), S.ERANGE),                   # ctx + 1 > max_seq_len
])
def test_forward_rejects_bad_batches(lib, batch, code):
    s = Setup(lib)
    rc = s.call(S.make_batch(*batch))
    assert rc == code, S.sarathi_last_error()


@pytest.mark.parametrize("chunks,decodes,code", [
    ([], ([], []), S.EINVAL),                                  # empty batch
    ([(1, 0, 4), (1, 8, 4)], ([], []), S.EINVAL),             # one slot in two chunks
    ([(1, 0, 4), (2, 0, 0)], ([], []), S.ERANGE),             # empty chunk
    ([(1, 0, 4), (9, 0, 4)], ([], []), S.EINVAL),             # slot out of range
    ([(1, 0, 4), (2, 250, 7)], ([], []), S.ERANGE),           # offset + len > max_seq_len
    ([(1, 0, 4), (2, -3, 7)], ([], []), S.ERANGE),            # negative offset
    ([(1, 0, 4), (2, 0, 7)], ([2], [5]), S.EINVAL),           # decode slot == a chunk's slot
    ([(1, 0, 4), (2, 0, 7)], ([3], [256]), S.ERANGE),         # ctx + 1 > max_seq_len
])
def test_mixed_forward_rejects_bad_batches(lib, chunks, decodes, code):
    s = Setup(lib)
    b, keep = S.make_mixed_batch(chunks, *decodes)
    ws = S.sarathi_mixed_workspace_bytes(s.cfg, 128, 4, 256)
    rc = S.sarathi_mixed_layer_forward(s.cfg, s.w, s.kv, 0, b, 0x200000, 0x300000, 0x40000000, ws, check=False)
    assert rc == code, S.sarathi_last_error()
    rc = S.sarathi_mixed_model_step(s.cfg, [s.w, s.w], s.kv, b, 0x200000, 0x300000, 0x40000000, ws, check=False)
    assert rc == code, S.sarathi_last_error()


def test_mixed_batch_bad_header_fields(lib):
    s = Setup(lib)
    b, keep = S.make_mixed_batch([(1, 0, 4)], [], [])
    b.n_chunks = -1
    ws = S.sarathi_mixed_workspace_bytes(s.cfg, 128, 4, 256)
    assert S.sarathi_mixed_layer_forward(s.cfg, s.w, s.kv, 0, b, 0x200000, 0x300000, 0x40000000, ws,
                                         check=False) == S.EINVAL
    b.n_chunks = 2
    b.chunk_lens = ct.cast(None, ct.POINTER(ct.c_int))
    assert S.sarathi_mixed_layer_forward(s.cfg, s.w, s.kv, 0, b, 0x200000, 0x300000, 0x40000000, ws,
                                         check=False) == S.EINVAL


def test_mixed_workspace_grows_with_chunks_and_matches_hybrid(lib):
    cfg = tiny_cfg(dtype=S.BF16)
    one = S.sarathi_mixed_workspace_bytes(cfg, 300, 1, 512)
    assert one == S.sarathi_workspace_bytes(cfg, 300, 8, 512)
    assert S.sarathi_mixed_workspace_bytes(cfg, 300, 5, 512) > one
    L1, L5 = S.sarathi_mixed_workspace_layout(cfg, 300, 1, 512), S.sarathi_mixed_workspace_layout(cfg, 300, 5, 512)
    assert (L1.a, L1.qkv, L1.o, L1.hres, L1.m) == (L5.a, L5.qkv, L5.o, L5.hres, L5.m)
    s = Setup(lib)
    b, keep = S.make_mixed_batch([(1, 0, 40), (2, 0, 40), (3, 0, 40)], [], [])
    small = S.sarathi_mixed_workspace_bytes(s.cfg, 120, 1, 256)
    assert S.sarathi_mixed_layer_forward(s.cfg, s.w, s.kv, 0, b, 0x200000, 0x300000, 0x40000000, small,
                                         check=False) == S.ENOSPC      # sized for one chunk, three given


def test_forward_accepts_edge_positions_up_to_validation(lib):
    # offset + C == max_seq_len and ctx + 1 == max_seq_len are legal: only the
    # workspace is too small here, so validation gets all the way to ENOSPC.
    s = Setup(lib)
    assert s.call(S.make_batch(1, 252, 4, [3], [255]), ws_bytes=16) == S.ENOSPC


def test_forward_rejects_other_misuse(lib):
    s = Setup(lib)
    good = S.make_batch(1, 0, 4, [3, 5], [10, 20])
    assert s.call(good, layer=2) == S.EINVAL                      # layer out of range
    assert s.call(good, layer=-1) == S.EINVAL
    assert s.call(good, ws_bytes=1024) == S.ENOSPC                # workspace too small
    assert s.call(good, x_out=0x200000) == S.EINVAL               # x_in == x_out
    assert s.call(good, x_in=0) == S.EINVAL                       # null input
    assert s.call(good, ws=0) == S.EINVAL
    assert s.call(good, x_in=0x200002) == S.EINVAL                # misaligned
    assert s.call(good, ws=0x200000 + 64) == S.EINVAL             # ws overlaps x_in
    other = tiny_cfg(ffn=696)
    assert s.call(good, cfg=other) == S.EINVAL                    # cfg differs from the KV's
    w = S.make_weights({k: FAKE_DEV for k in ("norm1_g", "w_qkv", "w_o", "norm2_g", "w_up")})
    assert s.call(good, w=w) == S.EINVAL                          # missing w_down
    b, keep = S.make_batch(1, 0, 4, [3], [10])
    b.decode_slots = ct.POINTER(ct.c_int)()
    assert S.sarathi_hybrid_layer_forward(s.cfg, s.w, s.kv, 0, b, 0x200000, 0x300000, 0x40000000, s.ws_bytes,
                                          check=False) == S.EINVAL
    assert "NULL" in S.sarathi_last_error()


def test_layernorm_needs_biases(lib):
    cfg = tiny_cfg(norm=S.NORM_LAYER, act=S.ACT_GELU, rope=0)
    kv = S.sarathi_kv_alloc(cfg, 9, 256, FAKE_DEV, S.sarathi_kv_bytes(cfg, 9, 256))
    w = S.make_weights({k: FAKE_DEV for k in ("norm1_g", "w_qkv", "w_o", "norm2_g", "w_up", "w_down")})
    b, keep = S.make_batch(1, 0, 4, [], [])
    rc = S.sarathi_hybrid_layer_forward(cfg, w, kv, 0, b, 0x200000, 0x300000, 0x40000000, 1 << 30, check=False)
    assert rc == S.EINVAL and "bias" in S.sarathi_last_error()


def test_model_step_validates_every_layer(lib):
    s = Setup(lib)
    good_w = s.w
    bad_w = S.make_weights({k: FAKE_DEV for k in ("norm1_g", "w_qkv", "w_o", "norm2_g", "w_up")})
    b, keep = S.make_batch(1, 0, 4, [3], [10])
    rc = S.sarathi_model_step(s.cfg, [good_w, bad_w], s.kv, b, 0x200000, 0x300000, 0x40000000, s.ws_bytes,
                              check=False)
    assert rc == S.EINVAL and "layer 1" in S.sarathi_last_error()


def test_linear_validation(lib):
    assert S.sarathi_linear(S.BF16, S.LINEAR_PLAIN, 4, 4, 12, FAKE_DEV, FAKE_DEV, 0, FAKE_DEV,
                            check=False) == S.EUNSUPPORTED                 # K % 8
    assert S.sarathi_linear(S.BF16, 9, 4, 4, 16, FAKE_DEV, FAKE_DEV, 0, FAKE_DEV, check=False) == S.EINVAL
    assert S.sarathi_linear(S.BF16, S.LINEAR_RESID, 4, 4, 16, FAKE_DEV, FAKE_DEV, 0, FAKE_DEV,
                            check=False) == S.EINVAL                        # resid missing
    assert S.sarathi_linear(S.BF16, S.LINEAR_PLAIN, 0, 4, 16, FAKE_DEV, FAKE_DEV, 0, FAKE_DEV,
                            check=False) == S.EINVAL
    assert S.sarathi_linear_scratch_bytes(320, 5120) == 6 * 320 * 5120 * 4


def test_linear_tile_queries_and_validation(lib):
    n = S.sarathi_linear_tile_count()
    assert n >= 4
    shapes = [S.sarathi_linear_tile_shape(t) for t in range(n)]
    assert len(set(shapes)) == n
    for bm, bn in shapes:
        assert bm % 16 == 0 and bn % 32 == 0
    bm, bn = ct.c_int(), ct.c_int()
    assert lib.sarathi_linear_tile_shape(n, ct.byref(bm), ct.byref(bn)) == S.EINVAL
    assert lib.sarathi_linear_tile_shape(-1, ct.byref(bm), ct.byref(bn)) == S.EINVAL
    assert lib.sarathi_linear_tile_shape(0, None, ct.byref(bn)) == S.EINVAL
    call = lambda **kw: S.sarathi_linear_tiled(kw.get("kind", S.LINEAR_PLAIN), 4, 4, kw.get("K", 64), FAKE_DEV,
                                               FAKE_DEV, 0, FAKE_DEV, 0, 0, kw.get("tile", 0),
                                               kw.get("n_split", 1), check=False)
    assert call(tile=n) == S.EINVAL
    assert call(tile=-1) == S.EINVAL
    assert call(n_split=0) == S.EINVAL
    assert call(K=96) == S.EUNSUPPORTED                  # not a multiple of 64
    assert call(kind=9) == S.EINVAL
    assert call(kind=S.LINEAR_RESID) == S.EINVAL         # resid is NULL


def test_noalloc_validates_and_rejects_batches_beyond_its_scratch(lib):
    s = Setup(lib)
    b, keep = S.make_batch(1, 0, 4, [2, 2], [3, 4])                # duplicate decode slot
    assert S.sarathi_hybrid_layer_forward_noalloc(s.cfg, s.w, s.kv, 0, b, 0x200000, 0x300000,
                                                  check=False) == S.EINVAL
    b, keep = S.make_batch(1, 0, 4, [3], [10])
    assert S.sarathi_hybrid_layer_forward_noalloc(s.cfg, s.w, s.kv, 5, b, 0x200000, 0x300000,
                                                  check=False) == S.EINVAL      # layer out of range
    assert S.sarathi_hybrid_layer_forward_noalloc(s.cfg, s.w, s.kv, 0, b, 0x200000, 0x200000,
                                                  check=False) == S.EINVAL      # x_in == x_out
    # a batch whose workspace exceeds the static scratch
    n_slots, S_ = 2, 1 << 20
    cfg = tiny_cfg(dtype=S.BF16)
    kv = S.sarathi_kv_alloc(cfg, n_slots, S_, FAKE_DEV, S.sarathi_kv_bytes(cfg, n_slots, S_))
    w = S.make_weights({k: FAKE_DEV for k in ("norm1_g", "w_qkv", "w_o", "norm2_g", "w_up", "w_down")})
    big = S.make_batch(0, 0, 100000, [1], [5])
    assert S.sarathi_workspace_bytes(cfg, 100001, 1, S_) > S.NOALLOC_SCRATCH_BYTES
    rc = S.sarathi_hybrid_layer_forward_noalloc(cfg, w, kv, 0, big[0], 0x200000, 0x40000000, check=False)
    assert rc == S.ENOSPC and "static scratch" in S.sarathi_last_error()


def test_linear_plan_reports_split_choice():
    from paper_2308_16369_amd import sarathi as S
    # residual op of the LLaMA-13B layer at 320 rows: split over K when the scratch allows it
    cfg = S.make_cfg(hidden=5120, n_heads=40, head_dim=128, ffn=13824, n_layers=1, dtype=S.BF16)
    scratch = S.sarathi_layer_split_scratch_bytes(cfg, 320)
    assert scratch == 6 * 320 * 5120 * 4
    bm, bn, ns = S.sarathi_linear_plan(S.BF16, S.LINEAR_RESID, 320, 5120, 5120, scratch)
    assert bm > 0 and bn > 0 and 1 <= ns <= 6
    assert S.sarathi_linear_plan(S.BF16, S.LINEAR_RESID, 320, 5120, 5120, 0)[2] == 1     # no scratch: no split
    assert S.sarathi_linear_plan(S.BF16, S.LINEAR_PLAIN, 320, 15360, 5120, scratch)[2] == 1
    with pytest.raises(S.SarathiError):
        S.sarathi_linear_plan(S.BF16, 9, 320, 5120, 5120, 0)


def test_attention_plan_counts_partials():
    from paper_2308_16369_amd import sarathi as S
    cfg = S.make_cfg(hidden=5120, n_heads=40, head_dim=128, ffn=13824, n_layers=1, dtype=S.BF16)
    # decodes only: one partial row per 512-key split, every row combined
    bb, keep = S.make_batch(-1, 0, 0, [1, 2, 3], [10, 600, 1500])
    p = S.sarathi_attention_plan(cfg, bb)
    assert p["chunk_items"] == 0 and p["decode_items"] == 1 + 2 + 3
    assert p["partial_rows_written"] == 6 and p["partial_rows_read"] == 6 and p["combine_rows"] == 3
    # a short chunk at offset 0 (two key tiles) is one item that writes its rows directly
    bb, keep = S.make_batch(0, 0, 100, [], [])
    p = S.sarathi_attention_plan(cfg, bb)
    assert p == {"chunk_items": 1, "decode_items": 0, "partial_rows_written": 0, "partial_rows_read": 0,
                 "combine_rows": 0}
    # a long prefix is split over keys: every split writes the block's rows, the combine reads them all
    bb, keep = S.make_batch(0, 4096, 100, [7], [5])
    p = S.sarathi_attention_plan(cfg, bb)
    assert p["chunk_items"] > 1 and p["decode_items"] == 1
    assert p["partial_rows_written"] == 100 * p["chunk_items"] + 1
    assert p["partial_rows_read"] == p["partial_rows_written"] and p["combine_rows"] == 101
    with pytest.raises(S.SarathiError):
        S.sarathi_attention_plan(cfg, S.make_batch(-1, 0, 0, [], [])[0])


def test_attention_plan_invariants_random():
    """On random single-chunk batches (several head counts, chunk lengths,
    prefixes and decode contexts) the plan's counts are consistent: one
    decode item per 512-key split; every partial row written is read back
    once; the combine pass covers the decodes plus exactly the chunk rows
    whose query block was split; a prefix-plus-chunk of at most four key
    tiles is never split; the chunk items cover every query block."""
    import random
    from paper_2308_16369_amd import sarathi as S
    rng = random.Random(2308)
    for nh in (8, 40, 52, 96):
        cfg = S.make_cfg(hidden=nh * 128, n_heads=nh, head_dim=128, ffn=4 * nh * 128, n_layers=1, dtype=S.BF16)
        for _ in range(60):
            C = rng.choice([0, 1, rng.randint(2, 127), 128, rng.randint(129, 600), rng.randint(600, 2048)])
            off = rng.choice([0, rng.randint(1, 300), rng.randint(300, 20000)]) if C else 0
            B = rng.randint(0 if C else 1, 40)
            ctx = [rng.randint(0, 5000) for _ in range(B)]
            bb, keep = S.make_batch(0 if C else -1, off, C, list(range(1, B + 1)), ctx)
            p = S.sarathi_attention_plan(cfg, bb)
            assert p["decode_items"] == sum((c + 1 + 511) // 512 for c in ctx)
            assert p["partial_rows_written"] == p["partial_rows_read"]
            chunk_partials = p["partial_rows_written"] - p["decode_items"]
            split_rows = p["combine_rows"] - B
            assert 0 <= split_rows <= C and chunk_partials >= 2 * split_rows
            if off + C <= 256:
                assert chunk_partials == 0 and split_rows == 0
            if C:
                assert -(-C // 256) <= p["chunk_items"] <= -(-C // 128) * -(-(off + C) // 256)
            else:
                assert p["chunk_items"] == 0


def test_attention_plan_block_size():
    """The plan prices 256-query blocks (8 waves) and 128-query blocks (4
    waves, 0.82 of the time per key tile) with the same model -- rounds of
    256 blocks x (largest key range + 4 tiles) -- and takes the cheaper."""
    from paper_2308_16369_amd import sarathi as S
    # LLaMA-13B, chunk 256 @ 512: 256-query blocks: 12 tiles in ranges of 4
    # (120 blocks, cost 8); 128-query blocks: 10 and 12 tiles in ranges of at
    # most 4 (240 blocks, cost 8 x 0.82) -> 2 blocks x 3 ranges per head
    cfg = S.make_cfg(hidden=5120, n_heads=40, head_dim=128, ffn=13824, n_layers=1, dtype=S.BF16)
    bb, keep = S.make_batch(0, 512, 256, [1], [700])
    p = S.sarathi_attention_plan(cfg, bb)
    assert p["chunk_items"] == 6
    assert p["partial_rows_written"] == 3 * 256 + 2
    # LLaMA-33B, chunk 512 @ 2048: 256-query blocks of 36 and 40 tiles in two
    # ranges each fit one round (208 blocks, cost 24); 128-query blocks do no
    # better than 44 x 0.82 -> 2 blocks x 2 ranges per head
    cfg = S.make_cfg(hidden=6656, n_heads=52, head_dim=128, ffn=17920, n_layers=1, dtype=S.BF16)
    bb, keep = S.make_batch(0, 2048, 512, [], [])
    p = S.sarathi_attention_plan(cfg, bb)
    assert p["chunk_items"] == 4
    assert p["partial_rows_written"] == 2 * 512 and p["combine_rows"] == 512
