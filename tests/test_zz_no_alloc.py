"""The entry point without allocation (sarathi_hybrid_layer_forward_noalloc)
against sarathi_hybrid_layer_forward, through the C-ABI: two calls in a row
on one GPU, the second with a smaller batch (so the static scratch still
holds the first call's contents), each compared bit for bit with the
existing entry point run on its own copy of the inputs and the KV cache
(same kernels, same plan: identical results).  A batch larger than the
static scratch is rejected on the host (tests/test_abi_host.py)."""
import numpy as np
import pytest

import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from gpu_harness import TOL, DeviceModel, log, rel_err, from_dev  # noqa: E402
from paper_2308_16369_amd import sarathi as S  # noqa: E402


def run_pair(inst, label):
    """Layer 0 of `inst` through both entry points, each on its own KV copy."""
    ref = DeviceModel(inst)
    new = DeviceModel(inst)
    b = inst.batch
    x = torch.from_numpy(wl.bf16_bits(inst.x).view(np.int16)).view(torch.bfloat16).cuda() \
        if inst.shape.dtype == "bf16" else torch.from_numpy(inst.x).cuda()
    y_ref = ref.layer(0, b, x)
    y_new = torch.empty_like(x)
    bb, keep = new.batch_abi(b)
    S.sarathi_hybrid_layer_forward_noalloc(new.cfg, new.w_abi[0], new.kv, 0, bb, x.data_ptr(), y_new.data_ptr(),
                                           torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    same_y = torch.equal(y_new.view(torch.int16) if y_new.dtype == torch.bfloat16 else y_new.view(torch.int32),
                         y_ref.view(torch.int16) if y_ref.dtype == torch.bfloat16 else y_ref.view(torch.int32))
    same_kv = torch.equal(new.kv_dev.view(torch.int16) if new.kv_dev.dtype == torch.bfloat16
                          else new.kv_dev.view(torch.int32),
                          ref.kv_dev.view(torch.int16) if ref.kv_dev.dtype == torch.bfloat16
                          else ref.kv_dev.view(torch.int32))
    err = rel_err(from_dev(y_new), from_dev(y_ref))
    log(f"{label}: T={b.n_tokens}: y bit-identical {same_y}, KV bit-identical {same_kv}, rel err {err:.3e}")
    assert err <= TOL[inst.shape.dtype]
    assert same_y and same_kv, label


def test_noalloc_matches_hybrid_layer_forward_twice():
    shp = wl.with_dtype(wl.TINY, "bf16").shape
    # call 1: the tiny workload (chunk 64 at offset 128 + 8 decodes)
    run_pair(wl.generate(wl.with_dtype(wl.TINY, "bf16")), "call 1")
    # call 2: a smaller batch on the same static scratch (chunk 16 at 40 + 3 decodes)
    b = wl.Batch(prefill_slot=2, chunk_offset=40, chunk_len=16, decode_slots=np.array([5, 0, 7], np.int32),
                 decode_ctx=np.array([100, 3, 57], np.int32))
    run_pair(wl.make_instance(shp, b, max_seq_len=256, n_slots=9, seed=3), "call 2 (smaller)")
