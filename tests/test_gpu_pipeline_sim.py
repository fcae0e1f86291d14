"""The cost-model measurement behind the pipeline-bubble simulator runs on
the device (tiny bf16 layer) and predicts held-out whole-layer times."""
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

import workloads as wl  # noqa: E402
from paper_2308_16369_amd import pipeline_sim as P  # noqa: E402


def test_measure_cost_model_tiny():
    shape = wl.with_dtype(wl.TINY, "bf16").shape
    cm = P.measure_cost_model(shape, max_seq=512, max_decodes=8)
    assert cm.rows == sorted(cm.rows) and all(v > 0 for v in cm.linear_ms)
    assert cm.check["held_out_batches"] == 12
    assert cm.layer_ms([(0, 64)], [100, 200]) > cm.layer_ms([], [100])
    back = P.CostModel.from_json(cm.to_json())
    assert back.layer_ms([(10, 30)], [5]) == cm.layer_ms([(10, 30)], [5])
