"""GPU parity of the 40-layer model step (LLaMA-13B-shaped stack, bf16):
four consecutive decode-maximal steps, each one 256-token chunk of a
1024-token prompt plus 48 decodes, the KV cache (85 GB) grown in place.

Checks:
  * step 0 run layer by layer: layers 0, 19 and 39 against the oracle on the
    GPU's own input of that layer (layer-local parity);
  * step 0 through sarathi_model_step equals the layer-by-layer result;
  * every step: the last layer of the model step against the oracle on its
    input (read from the model step's ping-pong buffer); cache positions
    beyond each slot's valid length keep their NaN sentinel, positions below
    it are finite, and the pre-filled positions of layers 0 and 39 keep their
    contents (checksums);
  * the decode-only batch of the same decodes (the paper's comparison) runs.
"""
import numpy as np
import pytest

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from gpu_harness import TOL, cfg_of, delta_err, from_dev, log, oracle_batch, rel_err  # noqa: E402
from paper_2308_16369_amd import sarathi as S  # noqa: E402


def host_layer(st, layer):
    """fp32 host copies of one layer's weights and KV (exact bf16 values)."""
    w = {k: from_dev(t) for k, t in st.weights[layer].items()}
    kv = from_dev(st.kv[layer])
    return w, kv


def check_layer(st, layer, b, x_dev, y_dev, label):
    w, kv = host_layer(st, layer)
    x = from_dev(x_dev)
    ref = oracle.layer_forward(st.workload.shape, w, kv, oracle_batch(b), x)
    y = from_dev(y_dev)
    e_y = rel_err(y, ref.y)
    e_d = delta_err(y, ref.y, ref.y - ref.hres, "bf16")
    log(f"{label}: layer {layer}: y {e_y:.3e}, y-hres beyond rounding {e_d:.3e}")
    assert e_y <= TOL["bf16"] and e_d <= TOL["bf16"], label


def test_llama13b_stack_four_steps():
    w = wl.LLAMA13B_STACK
    from workloads.stack import generate_stack_on_device

    log("generating the 40-layer stack on the device")
    st = generate_stack_on_device(w)
    shp, L = w.shape, w.shape.n_layers
    cfg = cfg_of(shp, L)
    kvb = st.kv.numel() * 2
    kv = S.sarathi_kv_alloc(cfg, st.kv.shape[1], st.kv.shape[4], st.kv.data_ptr(), kvb)
    wabi = [S.make_weights({k: t.data_ptr() for k, t in lw.items()}) for lw in st.weights]
    T = st.batch.n_tokens
    Sx = st.kv.shape[4]
    ws_bytes = S.sarathi_workspace_bytes(cfg, T, st.batch.n_decodes, Sx)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream

    def batch_abi(b):
        return S.make_batch(b.prefill_slot, b.chunk_offset, b.chunk_len, list(b.decode_slots), list(b.decode_ctx))

    # checksums of the pre-filled cache of layers 0 and L-1
    valid0 = wl.valid_lengths(st.batch, st.kv.shape[1])

    def prefilled_sum(layer):
        tot = 0.0
        for s in range(st.kv.shape[1]):
            n = int(valid0[s])
            if n:
                tot += st.kv[layer, s, :, :, :n, :].float().double().sum().item()
        return tot

    sums0 = {layer: prefilled_sum(layer) for layer in (0, L - 1)}

    # ---- step 0 layer by layer, layer-local parity at 0, 19, 39
    b0 = st.step_batch(0)
    bb, keep = batch_abi(b0)
    xs = [st.x]
    for layer in range(L):
        y = torch.empty_like(st.x)
        S.sarathi_hybrid_layer_forward(cfg, wabi[layer], kv, layer, bb, xs[-1].data_ptr(), y.data_ptr(),
                                       ws.data_ptr(), ws_bytes, stream)
        xs.append(y)
    torch.cuda.synchronize()
    log("step 0 layer by layer done")
    for layer in (0, L // 2 - 1, L - 1):
        check_layer(st, layer, b0, xs[layer], xs[layer + 1], "step 0 layer-by-layer")

    # ---- step 0 through the model step: same result as layer by layer
    y_ms = torch.empty_like(st.x)
    S.sarathi_model_step(cfg, wabi, kv, bb, st.x.data_ptr(), y_ms.data_ptr(), ws.data_ptr(), ws_bytes, stream)
    torch.cuda.synchronize()
    e = rel_err(from_dev(y_ms), from_dev(xs[-1]))
    log(f"step 0 model_step vs layer-by-layer: {e:.3e}")
    assert e <= TOL["bf16"]

    lay = S.sarathi_workspace_layout(cfg, T, st.batch.n_decodes, Sx)
    ping = lay.ping[(L - 1) % 2]

    def last_input():
        return ws[ping:ping + T * shp.hidden * 2].view(torch.bfloat16).view(T, shp.hidden).clone()

    rng = torch.Generator(device="cuda")
    rng.manual_seed(1)
    for step in range(4):
        b = st.step_batch(step)
        bb, keep = batch_abi(b)
        x = st.x if step == 0 else torch.empty_like(st.x).normal_(0.0, 1.0, generator=rng)
        y = torch.empty_like(x)
        S.sarathi_model_step(cfg, wabi, kv, bb, x.data_ptr(), y.data_ptr(), ws.data_ptr(), ws_bytes, stream)
        torch.cuda.synchronize()
        log(f"step {step}: model_step done (chunk @ {b.chunk_offset}, ctx + {step})")
        assert torch.isfinite(y.float()).all()
        check_layer(st, L - 1, b, last_input(), y, f"step {step} model_step last layer")
        # valid prefixes finite, everything after them still the NaN sentinel
        valid = wl.valid_lengths(b, st.kv.shape[1])
        if b.chunk_len:
            valid[b.prefill_slot] += b.chunk_len
        for s in b.decode_slots:
            valid[int(s)] += 1
        for layer in (0, L - 1):
            for s in range(st.kv.shape[1]):
                n = int(valid[s])
                blk = st.kv[layer, s]
                assert torch.isfinite(blk[:, :, :n, :].float()).all(), (step, layer, s)
                assert torch.isnan(blk[:, :, n:, :].float()).all(), (step, layer, s)
    for layer in (0, L - 1):
        assert prefilled_sum(layer) == sums0[layer], f"pre-filled cache of layer {layer} changed"

    # ---- the decode-only comparison batch (same decodes, next positions)
    bd = st.step_batch(4)
    bd = wl.Batch(prefill_slot=-1, chunk_offset=0, chunk_len=0, decode_slots=bd.decode_slots,
                  decode_ctx=bd.decode_ctx)
    bb, keep = batch_abi(bd)
    xd = st.x[st.batch.chunk_len:].clone()
    yd = torch.empty_like(xd)
    S.sarathi_model_step(cfg, wabi, kv, bb, xd.data_ptr(), yd.data_ptr(), ws.data_ptr(), ws_bytes, stream)
    torch.cuda.synchronize()
    lay_d = S.sarathi_workspace_layout(cfg, bd.n_tokens, bd.n_decodes, Sx)
    pd = lay_d.ping[(L - 1) % 2]
    xl = ws[pd:pd + bd.n_tokens * shp.hidden * 2].view(torch.bfloat16).view(bd.n_tokens, shp.hidden).clone()
    check_layer(st, L - 1, bd, xl, yd, "decode-only model_step last layer")
