"""GPU parity of the 40-layer model step (LLaMA-13B-shaped stack, bf16):
four consecutive decode-maximal steps, each one 256-token chunk of a
1024-token prompt plus 48 decodes, the KV cache (85 GB) grown in place, then
the decode-only batch (C = 0) of the same 48 decodes -- one iteration of the
model per step (Sec. 4.5).

All GPU work runs first (module fixture): every batch is run layer by layer
through sarathi_hybrid_layer_forward, keeping each layer's input, output and
fp32 residual h, and then again through sarathi_model_step, whose output must
equal the layer-by-layer one bit for bit (same kernels, same plan, same
inputs).  The oracle checks then read the final cache: a batch reads, per
slot, only positions up to its own rows' positions, which no later batch
writes, and the oracle replaces the batch's own new positions with its own
K/V before attending, so the cache after all batches serves every batch.

Checks:
  * step 0, every one of the 40 layers against the oracle on the GPU's input
    of that layer: y, the FFN contribution y - h, the attention contribution
    h - x, and the K/V written at exactly the rows' (slot, position);
  * steps 1-3 and the decode-only batch: the same at layers 0, 19 and 39;
  * step 0 chained: the oracle fed its own output from x through all 40
    layers; the drift of the GPU's bf16 activations from it is logged layer
    by layer and bounded by tol * sqrt(layer + 1) (independent per-layer
    errors, each within tol, accumulating);
  * after every batch: positions beyond each slot's valid length keep their
    NaN sentinel, positions below it are finite; the pre-filled positions of
    layers 0 and 39 keep their contents (checksums).
(The 40-layer chain at the fp32 tolerance, where the drift stays far below
it, is tests/test_gpu_parity.py::test_model_step_forty_layers_f32_chained.)
"""
import numpy as np
import pytest

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from gpu_harness import TOL, cfg_of, half_ulp_bf16, log, oracle_batch, rel_err  # noqa: E402
from paper_2308_16369_amd import sarathi as S  # noqa: E402

LOCAL_LAYERS = (0, 19, 39)
N_STEPS = 4


def f32_host(t):
    """Device tensor -> fp32 numpy; bf16 is widened on the device (exact)."""
    return t.float().cpu().numpy()


def need_positions(b: wl.Batch, n_slots: int) -> dict:
    """Positions [0, n) of each slot that the batch's rows read (own key included)."""
    need = {}
    if b.chunk_len:
        need[b.prefill_slot] = b.chunk_offset + b.chunk_len
    for s, c in zip(b.decode_slots, b.decode_ctx):
        need[int(s)] = int(c) + 1
    return need


class HostKV:
    """One layer's cache as the oracle reads it: per slot, an fp32 copy of
    positions [0, n) only (a whole layer is 2 GB)."""

    def __init__(self, kv_dev_layer, need: dict):
        self.blk = {s: f32_host(kv_dev_layer[s, :, :, :n, :]) for s, n in need.items()}

    def __getitem__(self, idx):
        return self.blk[int(idx[0])][tuple(idx[1:])]

    def __setitem__(self, idx, val):
        self.blk[int(idx[0])][tuple(idx[1:])] = val


def ffn_err(y_gpu, h_gpu, ref) -> float:
    """Error of the FFN contribution y - h: the GPU's own y - h against the
    oracle's, beyond half a bf16 ulp of y (y's unavoidable rounding), on the
    scale of the oracle's y - h."""
    d_gpu = np.asarray(y_gpu, np.float64) - np.asarray(h_gpu, np.float64)
    d_ref = ref.y - ref.hres
    diff = np.maximum(np.abs(d_gpu - d_ref) - half_ulp_bf16(np.maximum(np.abs(y_gpu), np.abs(ref.y))), 0.0)
    return float(np.max(diff) / np.max(np.abs(d_ref)))


class StackRun:
    """The stack, its cache and everything the GPU produced."""

    def __init__(self):
        w = wl.LLAMA13B_STACK
        from workloads.stack import generate_stack_on_device

        log("generating the 40-layer stack on the device")
        self.st = st = generate_stack_on_device(w)
        self.shp, self.L = w.shape, w.shape.n_layers
        self.cfg = cfg_of(self.shp, self.L)
        self.n_slots, self.Sx = st.kv.shape[1], st.kv.shape[4]
        self.kv = S.sarathi_kv_alloc(self.cfg, self.n_slots, self.Sx, st.kv.data_ptr(), st.kv.numel() * 2)
        self.wabi = [S.make_weights({k: t.data_ptr() for k, t in lw.items()}) for lw in st.weights]
        T = st.batch.n_tokens
        self.ws_bytes = S.sarathi_workspace_bytes(self.cfg, T, st.batch.n_decodes, self.Sx)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device="cuda")
        self.stream = torch.cuda.current_stream().cuda_stream
        self._host_w = {}

        valid0 = wl.valid_lengths(st.batch, self.n_slots)
        self.valid = valid0.copy()       # cached positions per slot, advanced after every batch
        self.sums0 = {layer: self.prefilled_sum(layer, valid0) for layer in (0, self.L - 1)}

        # the four decode-maximal steps, then the decode-only batch (C = 0) of
        # the same decodes at their next positions
        self.batches = [st.step_batch(i) for i in range(N_STEPS)]
        bd = st.step_batch(N_STEPS)
        self.batches.append(wl.Batch(prefill_slot=-1, chunk_offset=0, chunk_len=0, decode_slots=bd.decode_slots,
                                     decode_ctx=bd.decode_ctx))
        rng = torch.Generator(device="cuda")
        rng.manual_seed(1)
        self.runs = []
        self.model_step_equal = []
        self.cache_ok = []
        for i, b in enumerate(self.batches):
            if i == 0:
                x = st.x
            elif b.chunk_len == 0:
                x = st.x[st.batch.chunk_len:].clone()
            else:
                x = torch.empty_like(st.x).normal_(0.0, 1.0, generator=rng)
            keep_all = i == 0
            self.runs.append(self.run_layers(b, x, keep_all))
            y_ms = torch.empty_like(x)
            bb, keep = self.batch_abi(b)
            S.sarathi_model_step(self.cfg, self.wabi, self.kv, bb, x.data_ptr(), y_ms.data_ptr(), self.ws.data_ptr(),
                                 self.ws_bytes, self.stream)
            torch.cuda.synchronize()
            self.model_step_equal.append(bool(torch.equal(y_ms, self.runs[-1]["x"][self.L])))
            self.cache_ok.append(self.check_cache(b))
            log(f"batch {i}: C={b.chunk_len} @ {b.chunk_offset}, {b.n_decodes} decodes: layer by layer and model "
                f"step done; model step bit-identical {self.model_step_equal[-1]}, cache ok {self.cache_ok[-1]}")
        self.prefill_kept = {layer: self.prefilled_sum(layer, valid0) == self.sums0[layer]
                             for layer in (0, self.L - 1)}
        self.chain_h = np.asarray(f32_host(st.x), np.float64)   # the chained oracle's input to layer 0
        self.local_rms = {}

    def batch_abi(self, b):
        return S.make_batch(b.prefill_slot, b.chunk_offset, b.chunk_len, list(b.decode_slots), list(b.decode_ctx))

    def prefilled_sum(self, layer, valid):
        tot = 0.0
        for s in range(self.n_slots):
            n = int(valid[s])
            if n:
                tot += self.st.kv[layer, s, :, :, :n, :].double().sum().item()
        return tot

    def run_layers(self, b, x, keep_all):
        """The batch layer by layer; every layer's input/output on the device,
        h (fp32) of every layer (step 0) or of the locally checked layers."""
        T = b.n_tokens
        H = self.shp.hidden
        lay = S.sarathi_workspace_layout(self.cfg, T, b.n_decodes, self.Sx)
        bb, keep = self.batch_abi(b)
        xs, hs = [x], {}
        for layer in range(self.L):
            y = torch.empty_like(x)
            S.sarathi_hybrid_layer_forward(self.cfg, self.wabi[layer], self.kv, layer, bb, xs[-1].data_ptr(),
                                           y.data_ptr(), self.ws.data_ptr(), self.ws_bytes, self.stream)
            if keep_all or layer in LOCAL_LAYERS:
                hs[layer] = self.ws[lay.hres:lay.hres + T * H * 4].view(torch.float32).view(T, H).clone()
            xs.append(y)
        torch.cuda.synchronize()
        return {"x": xs, "h": hs}

    def check_cache(self, b):
        """Valid prefixes finite and everything after them the NaN sentinel,
        at layers 0 and L-1, after the batch."""
        for s, n in need_positions(b, self.n_slots).items():
            self.valid[s] = max(int(self.valid[s]), n)
        valid = self.valid
        for layer in (0, self.L - 1):
            for s in range(self.n_slots):
                n = int(valid[s])
                blk = self.st.kv[layer, s]
                if not torch.isfinite(blk[:, :, :n, :].float()).all():
                    return False
                if not torch.isnan(blk[:, :, n:, :].float()).all():
                    return False
        return True

    def host_weights(self, layer):
        if layer not in self._host_w:
            self._host_w = {layer: {k: f32_host(t) for k, t in self.st.weights[layer].items()}}
        return self._host_w[layer]

    def oracle_layer(self, layer, b, x_host):
        """The oracle layer on the given input, plus the K/V the GPU wrote at
        the rows' (slot, position) (read before the oracle overwrites them in
        its copy)."""
        hkv = HostKV(self.st.kv[layer], need_positions(b, self.n_slots))
        slots, pos = oracle.token_positions(oracle_batch(b))
        k_gpu = np.stack([hkv.blk[int(s)][0, :, int(p), :] for s, p in zip(slots, pos)])
        v_gpu = np.stack([hkv.blk[int(s)][1, :, int(p), :] for s, p in zip(slots, pos)])
        ref = oracle.layer_forward(self.shp, self.host_weights(layer), hkv, oracle_batch(b), x_host)
        return ref, k_gpu, v_gpu


@pytest.fixture(scope="module")
def stack():
    run = StackRun()
    yield run
    torch.cuda.synchronize()


def check(label, errs):
    for name, e in errs.items():
        log(f"  {label}: {name:34s} {e:.3e}")
    bad = {n: e for n, e in errs.items() if not e <= TOL["bf16"]}
    assert not bad, f"{label}: {bad}"


def test_model_step_equals_layer_by_layer(stack):
    assert all(stack.model_step_equal), stack.model_step_equal


def test_cache_sentinels_and_prefill_kept(stack):
    assert all(stack.cache_ok), stack.cache_ok
    assert all(stack.prefill_kept.values()), stack.prefill_kept


def rms_rel(got, ref) -> float:
    ref = np.asarray(ref, np.float64)
    return float(np.sqrt(np.mean((np.asarray(got, np.float64) - ref) ** 2) / np.mean(ref ** 2)))


def layer_errs(stack, layer, b, run, x_ref, ref, k_gpu, v_gpu):
    y = f32_host(run["x"][layer + 1])
    h = f32_host(run["h"][layer])
    x_gpu = f32_host(run["x"][layer])
    return {
        "y": rel_err(y, ref.y),
        "y - h (beyond y rounding)": ffn_err(y, h, ref),
        "h - x": rel_err(h.astype(np.float64) - x_gpu, ref.hres - x_ref),
        "k_new": rel_err(k_gpu, ref.k_new),
        "v_new": rel_err(v_gpu, ref.v_new),
        "y rms": rms_rel(y, ref.y),
    }


def local_layers(stack, lo, hi):
    """Step 0, layers lo..hi-1, each against the oracle on the GPU's own input."""
    b, run = stack.batches[0], stack.runs[0]
    for layer in range(lo, hi):
        x = f32_host(run["x"][layer])
        ref, k_gpu, v_gpu = stack.oracle_layer(layer, b, x)
        errs = layer_errs(stack, layer, b, run, x, ref, k_gpu, v_gpu)
        stack.local_rms[layer] = errs["y rms"]
        check(f"step 0 layer {layer} (own input)", errs)


def test_step0_every_layer_local_0_to_19(stack):
    local_layers(stack, 0, 20)


def test_step0_every_layer_local_20_to_39(stack):
    local_layers(stack, 20, stack.L)


def test_step0_chained_through_40_layers(stack):
    """The oracle fed its own output from x through all 40 layers.  Each
    GPU layer stores its output in bf16 (the interface type), so the GPU's
    input to layer l drifts from the oracle's by the errors of the layers
    before it; every layer's own error is held to the tolerance by the
    layer-local tests.  Here the drift is logged layer by layer and bounded
    by the accumulation of independent per-layer errors: y within
    tol * sqrt(l + 1) of the chained oracle at layer l.  The KV written at
    every layer is checked the same way."""
    b, run = stack.batches[0], stack.runs[0]
    h_ref = stack.chain_h
    worst = []
    for layer in range(stack.L):
        ref, k_gpu, v_gpu = stack.oracle_layer(layer, b, h_ref)
        errs = layer_errs(stack, layer, b, run, h_ref, ref, k_gpu, v_gpu)
        errs["x in rms (drift)"] = rms_rel(f32_host(run["x"][layer]), h_ref)
        for name, e in errs.items():
            log(f"  step 0 chained layer {layer}: {name:30s} {e:.3e}")
        bound = TOL["bf16"] * np.sqrt(layer + 1)
        worst.append((layer, max(errs["y"], errs["k_new"], errs["v_new"]), bound))
        h_ref = ref.y
    bad = [(l, e, bnd) for l, e, bnd in worst if not e <= bnd]
    log("  chained y/k/v error by layer: " + ", ".join(f"{l}:{e:.2e}" for l, e, _ in worst))
    assert not bad, f"chained drift beyond tol * sqrt(l + 1): {bad}"


@pytest.mark.parametrize("batch", range(1, N_STEPS + 1), ids=["step1", "step2", "step3", "decode_only"])
def test_layer_local(stack, batch):
    b = stack.batches[batch]
    run = stack.runs[batch]
    for layer in LOCAL_LAYERS:
        x = f32_host(run["x"][layer])
        ref, k_gpu, v_gpu = stack.oracle_layer(layer, b, x)
        y = f32_host(run["x"][layer + 1])
        h = f32_host(run["h"][layer])
        check(f"batch {batch} layer {layer} (own input)", {
            "y": rel_err(y, ref.y),
            "y - h (beyond y rounding)": ffn_err(y, h, ref),
            "h - x": rel_err(h.astype(np.float64) - x, ref.hres - x),
            "k_new": rel_err(k_gpu, ref.k_new),
            "v_new": rel_err(v_gpu, ref.v_new),
        })
