"""Host-side logic of the chunk-size ablation (no GPU)."""
import pytest

from paper_2308_16369_amd.ablation import chunk_plan, tile_lengths


@pytest.mark.parametrize("P,c", [(1, 1), (1024, 64), (1000, 256), (3072, 512), (100, 512), (7, 3)])
def test_chunk_plan_tiles_the_prompt(P, c):
    plan = chunk_plan(P, c)
    assert plan[0][0] == 0
    for (o, n), (o2, _) in zip(plan, plan[1:]):
        assert o2 == o + n and n == c            # contiguous, every chunk but the last full
    o, n = plan[-1]
    assert o + n == P and 1 <= n <= c
    assert len(plan) == -(-P // c)


def test_chunk_plan_rejects_bad_sizes():
    with pytest.raises(ValueError):
        chunk_plan(0, 64)
    with pytest.raises(ValueError):
        chunk_plan(64, 0)


def test_tile_lengths_brackets_every_multiple():
    pts = tile_lengths(32, 512, 32, [128])
    for m in (128, 256, 384, 512):
        assert m in pts and m - 1 in pts
        if m + 1 <= 512:
            assert m + 1 in pts
    assert pts == sorted(set(pts)) and pts[0] >= 32 and pts[-1] <= 512
