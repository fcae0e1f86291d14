"""The chunk-size ablation runs end to end on the device (tiny bf16 layer).
Its kernels' numerics are covered by the parity tests; this checks the
measurement driver: every sweep point is timed and the full-prefill rows of
the chunking table report an overhead of one."""
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

from paper_2308_16369_amd import ablation  # noqa: E402
import workloads as wl  # noqa: E402


def test_ablation_tiny(tmp_path):
    shape = wl.with_dtype(wl.TINY, "bf16").shape
    r = ablation.LayerRunner(shape, n_slots=5, max_seq_len=256, max_tokens=256, max_decodes=4)
    tq = ablation.tile_quantization(r, [63, 64, 65], iters=3)
    assert [e["rows"] for e in tq] == [63, 64, 65]
    assert all(e["ms"] > 0 and e["linear_ms"] > 0 for e in tq)
    co = ablation.chunking_overhead(r, [256], [64, 128], iters=2)
    assert sorted(e["chunk"] for e in co) == [64, 128, 256]
    assert [e["n_chunks"] for e in co if e["chunk"] == 64] == [4]
    full = [e for e in co if e["chunk"] == 256][0]
    assert 0.5 < full["overhead"] < 2.0
    pg = ablation.piggyback(r, [64], [4], ctx=100, offset=64, iters=3)
    assert pg[0]["rows"] == 68 and pg[0]["hybrid_ms"] > 0
    md = ablation.to_markdown({"workload": "tiny", "command": "test", "tile_quantization": tq,
                               "chunking_overhead": co, "piggyback_ctx": 100, "piggyback_offset": 64,
                               "piggyback": pg})
    assert md.count("\n|") > 8


def test_tile_sweep_tiny():
    """Every tile of the four linear ops of a small bf16 layer is timed and the
    planner's pick is among them exactly once per op and K-split."""
    shape = wl.with_dtype(wl.TINY, "bf16").shape
    rows = ablation.tile_sweep(shape, 72, iters=2)
    ops = {e["op"] for e in rows}
    assert ops == {"preproj", "postproj", "ffn_ln1", "ffn_ln2"}
    assert all(e["us"] > 0 and e["tflops"] > 0 for e in rows)
    for op in ops:
        assert sum(e["picked"] for e in rows if e["op"] == op) == 1
    # ffn_ln2's K (the FFN width 688) is off the 64-wide k-tiles: one row, the planner's kernel
    assert [e["picked"] for e in rows if e["op"] == "ffn_ln2"] == [True]
    md = ablation.tile_sweep_markdown("tiny", rows)
    assert md.count("\n|") == len(rows) + 2
