"""The layer forward and the model step captured in a HIP graph (through
torch.cuda.graph) and replayed: the library enqueues only kernels on the
caller's stream (no allocation, no memset, no host synchronisation, batch
metadata carried in kernel arguments), so a captured call replays the same
work.  Each replay follows eager work on the same buffers and a
synchronisation, and its output must equal the eager call's bit for bit
(the replay rewrites the same KV positions with the same values)."""
import numpy as np
import pytest

import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from gpu_harness import DeviceModel, log  # noqa: E402
from paper_2308_16369_amd import sarathi as S  # noqa: E402


def bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def to_dev(a, dtype):
    if dtype == "bf16":
        return torch.from_numpy(wl.bf16_bits(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("entry", ["layer", "noalloc", "model_step"])
def test_captured_call_replays_bit_identical(dtype, entry):
    inst = wl.generate(wl.with_dtype(wl.TINY, dtype), n_layers=3 if entry == "model_step" else 1)
    dm = DeviceModel(inst)
    b = inst.batch
    x = to_dev(inst.x, dtype)
    y = torch.empty_like(x)
    bb, keep = dm.batch_abi(b)

    def call(stream):
        if entry == "layer":
            S.sarathi_hybrid_layer_forward(dm.cfg, dm.w_abi[0], dm.kv, 0, bb, x.data_ptr(), y.data_ptr(),
                                           dm.ws.data_ptr(), dm.ws_bytes, stream)
        elif entry == "noalloc":
            S.sarathi_hybrid_layer_forward_noalloc(dm.cfg, dm.w_abi[0], dm.kv, 0, bb, x.data_ptr(), y.data_ptr(),
                                                   stream)
        else:
            S.sarathi_model_step(dm.cfg, dm.w_abi, dm.kv, bb, x.data_ptr(), y.data_ptr(), dm.ws.data_ptr(),
                                 dm.ws_bytes, stream)

    # eager reference (also the warm-up: one-time set-up happens outside the capture)
    call(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    y_eager = y.clone()
    kv_eager = dm.kv_dev.clone()

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=side):
        call(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()

    for rep in range(3):
        # eager work on the same buffers between replays
        y.fill_(float("nan"))
        junk = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        same_y = torch.equal(bits(y), bits(y_eager))
        same_kv = torch.equal(bits(dm.kv_dev), bits(kv_eager))
        log(f"graph {entry} {dtype} replay {rep}: y {same_y}, KV {same_kv} ({float(junk):.1f})")
        assert same_y and same_kv, f"replay {rep}"
