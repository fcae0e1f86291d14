/*
 * sarathi.h -- C-ABI of libsarathi.so: one decoder layer (and a stack of
 * layers) over a decode-maximal hybrid batch on an AMD MI355X (gfx950).
 *
 * The method (Sarathi, arXiv 2308.16369):
 *   - chunked prefills: a prompt is split into equal chunks, one chunk per
 *     iteration; a chunk's queries see the cached keys/values of the earlier
 *     chunks plus, causally, those of the chunk itself (Sec. 4.2 and its
 *     attention-mask figure);
 *   - decode-maximal batching: one prefill chunk plus decodes in the other
 *     slots; the linear ops (preproj, postproj, ffn_ln1, ffn_ln2) run as one
 *     matmul over all rows while the attention of the chunk and of the
 *     decodes runs separately (Sec. 4.3);
 *   - the KV cache is pre-allocated per request for the maximum sequence
 *     length and updated in place (Sec. 4.5).
 *
 * Conventions for every entry point:
 *   - Every pointer is borrowed.  Device pointers (weights, activations, KV
 *     memory, workspace) come from the caller; the library never allocates or
 *     frees device memory.  Host pointers (cfg, batch arrays) are read during
 *     the call only and may be reused as soon as it returns.
 *   - Work is enqueued asynchronously on the caller's HIP stream (`hip_stream`
 *     is a hipStream_t; NULL means the default stream).  Nothing is enqueued
 *     when a call returns an error found on the host.
 *   - Return value: SARATHI_OK or a negative error code; the thread-local
 *     message of the last error is returned by sarathi_last_error().
 *   - Calls that overlap on one stream are ordered by it; calls on different
 *     streams that share a workspace or KV region race.
 */
#ifndef SARATHI_H
#define SARATHI_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------------ status */
#define SARATHI_OK             0
#define SARATHI_EINVAL        -1  /* null pointer, empty batch, bad slot/layer, cfg mismatch, aliasing */
#define SARATHI_ERANGE        -2  /* offset/length/context outside [0, max_seq_len) */
#define SARATHI_ENOSPC        -3  /* workspace or KV memory too small */
#define SARATHI_EUNSUPPORTED  -4  /* shape or dtype outside what the kernels implement */
#define SARATHI_EHIP          -5  /* a HIP launch failed (message in sarathi_last_error) */

/* ------------------------------------------------------------------ model config */
#define SARATHI_F32   0
#define SARATHI_BF16  1

#define SARATHI_NORM_RMS    0   /* x / sqrt(mean(x^2) + eps) * g */
#define SARATHI_NORM_LAYER  1   /* (x - mean) / sqrt(var + eps) * g + b, biased var */

#define SARATHI_ACT_SWIGLU  0   /* ffn_ln1 -> silu(gate) * up, w_up rows: gate [0,F) then up [F,2F) */
#define SARATHI_ACT_GELU    1   /* ffn_ln1 -> gelu(z), exact erf form, w_up rows [0,F) */

/*
 * Shape of a pre-norm decoder layer (Sec. 2.1, Table 1: preproj, attn,
 * postproj, ffn_ln1, ffn_ln2 and the "others").  Multi-head attention with
 * n_heads heads of head_dim; rope != 0 rotates q and k by absolute position
 * (pairs (i, i + head_dim/2), angle pos * rope_base^(-2i/head_dim)).
 * Activations, weights and the KV cache all use `dtype`.
 */
typedef struct {
  int   hidden;      /* H; multiple of 8 */
  int   n_heads;
  int   head_dim;    /* 64 or 128 */
  int   ffn;         /* F; multiple of 8 */
  int   n_layers;
  int   norm;        /* SARATHI_NORM_* */
  int   act;         /* SARATHI_ACT_* */
  int   rope;        /* 0 or 1 */
  float rope_base;
  float eps;
  int   dtype;       /* SARATHI_F32 or SARATHI_BF16 */
} sarathi_model_cfg;

/*
 * Device pointers to one layer's weights, row-major [out, in] (y = x W^T):
 *   w_qkv  [3*n_heads*head_dim, hidden]   (q rows, then k rows, then v rows;
 *                                          head h owns rows h*head_dim.. in each)
 *   w_o    [hidden, n_heads*head_dim]
 *   w_up   [2*ffn, hidden] (SwiGLU: gate rows then up rows) or [ffn, hidden] (GELU)
 *   w_down [hidden, ffn]
 *   norm*_g [hidden] gains; norm*_b [hidden] biases (LayerNorm only, else ignored).
 * No linear biases.
 */
typedef struct {
  const void* norm1_g;
  const void* norm1_b;
  const void* w_qkv;
  const void* w_o;
  const void* norm2_g;
  const void* norm2_b;
  const void* w_up;
  const void* w_down;
} sarathi_layer_weights;

/*
 * Decode-maximal hybrid batch (Sec. 4.3): at most one prefill chunk plus
 * decodes.  Host memory.
 *   chunk: chunk_len tokens of the request in slot prefill_slot, at
 *          positions chunk_offset .. chunk_offset+chunk_len-1; positions
 *          0..chunk_offset-1 of that slot must already hold its earlier
 *          chunks' K/V (Sec. 4.2).  chunk_len = 0: decode-only batch.
 *   decodes: n_decodes requests; decode b is in slot decode_slots[b] with
 *          decode_ctx_lens[b] tokens already cached; its new token sits at
 *          position decode_ctx_lens[b] and attends to ctx+1 keys.
 *          n_decodes = 0: prefill-only batch.
 * Rows of x_in / x_out ([chunk_len + n_decodes, hidden]): the chunk's rows
 * in position order, then the decodes in array order.  All slots distinct.
 */
typedef struct {
  int        prefill_slot;
  int        chunk_offset;
  int        chunk_len;
  int        n_decodes;
  const int* decode_slots;
  const int* decode_ctx_lens;
} sarathi_hybrid_batch;

/*
 * Mixed batch: any number of prompt chunks plus decodes (the iteration-level
 * batching of Orca, which Sec. 5.2 compares against; with n_chunks <= 1 it
 * is the hybrid batch above).  Host memory.
 *   chunk i: chunk_lens[i] >= 1 tokens of the request in slot chunk_slots[i]
 *            at positions chunk_offsets[i] .. + chunk_lens[i] - 1 (earlier
 *            positions of that slot already cached);
 *   decodes: as in sarathi_hybrid_batch.
 * Rows of x_in / x_out: chunk 0's rows in position order, then chunk 1's, ...,
 * then the decodes in array order.  All slots distinct.
 */
typedef struct {
  int        n_chunks;
  const int* chunk_slots;
  const int* chunk_offsets;
  const int* chunk_lens;
  int        n_decodes;
  const int* decode_slots;
  const int* decode_ctx_lens;
} sarathi_mixed_batch;

/* ------------------------------------------------------------------ KV cache */
/*
 * Pre-allocated per-request KV slabs (Sec. 4.5), laid out
 *   [layer][slot][K=0 | V=1][head][pos][head_dim]   (dtype elements),
 * pos < max_seq_len.  Each (slot, head) K or V stream is contiguous.
 * The handle is host-side; the memory is the caller's.
 */
typedef struct sarathi_kv sarathi_kv;

/* Bytes of KV memory for the layout above (0 on invalid arguments). */
size_t sarathi_kv_bytes(const sarathi_model_cfg* cfg, int n_slots, int max_seq_len);

/*
 * Bind caller-owned device memory `dev_mem` of `dev_bytes` bytes (>=
 * sarathi_kv_bytes) as the KV cache of `cfg`; *out receives a host handle.
 * The memory is not touched.  Errors: EINVAL (null, n_slots/max_seq_len < 1),
 * EUNSUPPORTED (cfg), ENOSPC (dev_bytes too small).
 */
int sarathi_kv_alloc(const sarathi_model_cfg* cfg, int n_slots, int max_seq_len,
                     void* dev_mem, size_t dev_bytes, sarathi_kv** out);

/* Free the host handle (not the device memory).  NULL is accepted. */
void sarathi_kv_free(sarathi_kv* kv);

/* Element strides of the layout (layer, slot, K/V, head, pos); 0 on null. */
typedef struct {
  size_t layer, slot, kv, head, pos;
} sarathi_kv_strides;
int sarathi_kv_get_strides(const sarathi_kv* kv, sarathi_kv_strides* out);

/* ------------------------------------------------------------------ workspace */
/*
 * Device workspace of one call: intermediates, decode-attention partial
 * results and the batch metadata.  Its layout depends only on
 * (cfg, n_tokens, n_decodes, max_seq_len); after a layer call the
 * intermediates below hold that layer's values (element offsets in bytes from
 * the workspace base):
 *   a    [T, hidden]            dtype   norm_2 output (norm_1's is overwritten)
 *   qkv  [T, 3*nh*hd]           dtype   preproj output: the q columns (rotated); the k and
 *                                       v columns are undefined (k, v go to the KV cache)
 *   o    [T, nh*hd]             dtype   attention output
 *   hres [T, hidden]            fp32    x + postproj(o)
 *   m    [T, ffn]               dtype   ffn_ln1 activation output
 *   ping[2] [T, hidden]         dtype   sarathi_model_step hands layer l's
 *                                       output to layer l+1 in ping[(l+1) % 2]
 * For sarathi_model_step they hold the last layer's values (so ping[(L-1) % 2]
 * holds the last layer's input when L > 1).
 */
typedef struct {
  size_t a, qkv, o, hres, m;
  size_t ping[2];
  size_t total;      /* bytes needed */
} sarathi_ws_layout;

size_t sarathi_workspace_bytes(const sarathi_model_cfg* cfg, int max_tokens, int max_decodes,
                               int max_seq_len);
int sarathi_workspace_layout(const sarathi_model_cfg* cfg, int n_tokens, int n_decodes,
                             int max_seq_len, sarathi_ws_layout* out);
/* The same for mixed batches of up to max_chunks (n_chunks) prompt chunks;
 * with one chunk these equal the functions above. */
size_t sarathi_mixed_workspace_bytes(const sarathi_model_cfg* cfg, int max_tokens, int max_chunks,
                                     int max_seq_len);
int sarathi_mixed_workspace_layout(const sarathi_model_cfg* cfg, int n_tokens, int n_chunks,
                                   int max_seq_len, sarathi_ws_layout* out);

/*
 * How a layer call splits a hybrid batch's attention into work items (for
 * measurement; nothing is launched, the batch is checked against cfg only):
 * the chunk-attention and decode-attention work items per head, the rows of
 * fp32 key-split partials they write (hd + 4 floats per row and head; a
 * chunk item that covers every key of its rows writes the attention output
 * directly), and the partial rows the combine pass reads back.  Errors:
 * EINVAL (NULL arguments, malformed batch).
 */
typedef struct {
  int chunk_items;
  int decode_items;
  long partial_rows_written;
  long partial_rows_read;
  int combine_rows;
} sarathi_attn_plan;
int sarathi_attention_plan(const sarathi_model_cfg* cfg, const sarathi_hybrid_batch* batch,
                           sarathi_attn_plan* out);

/* ------------------------------------------------------------------ forward */
/*
 * One decoder layer over a hybrid batch (Sec. 4.3; layer `layer` of the KV
 * cache):
 *   a = norm_1(x); [q|k|v] = a W_qkv^T (one matmul over all rows);
 *   rotate q, k; write k, v to the cache at each row's (slot, position);
 *   chunk rows attend to keys 0..position of the prefill slot (cached
 *   prefix + causal within the chunk, Sec. 4.2); each decode attends to keys
 *   0..ctx of its slot; h = x + o W_o^T; b = norm_2(h);
 *   m = act(b W_up^T); y = h + m W_down^T.
 * x_in, x_out: device [T, hidden] dtype, not aliasing each other or ws.
 * KV: reads positions < chunk_offset+chunk_len (prefill slot) and <= ctx
 * (decode slots) of layer `layer`; writes exactly the new positions
 * (chunk_offset..chunk_offset+chunk_len-1 of the prefill slot, ctx of each
 * decode slot); touches nothing else.
 * ws: device workspace of ws_bytes >= sarathi_workspace_layout(...).total
 * for this batch and the KV's max_seq_len.
 * Errors (host-side, before any launch): EINVAL (null, C+B = 0, slot out of
 * range or repeated, layer out of range, cfg differs from the KV's, x_in ==
 * x_out), ERANGE (offset/chunk/context beyond max_seq_len or negative),
 * ENOSPC (ws too small), EUNSUPPORTED; EHIP if a launch fails.
 */
int sarathi_hybrid_layer_forward(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w,
                                 sarathi_kv* kv, int layer, const sarathi_hybrid_batch* batch,
                                 const void* x_in, void* x_out, void* ws, size_t ws_bytes,
                                 void* hip_stream);

/*
 * One iteration of the whole model over a hybrid batch (Sec. 4.5): layers
 * 0..cfg->n_layers-1 in order, layer l using w[l] (host array of n_layers
 * weight sets) and KV layer l, each layer's output feeding the next.  Same
 * arguments, errors and KV contract as sarathi_hybrid_layer_forward, for
 * every layer.  The batch metadata is copied to the device once per step.
 */
int sarathi_model_step(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w,
                       sarathi_kv* kv, const sarathi_hybrid_batch* batch,
                       const void* x_in, void* x_out, void* ws, size_t ws_bytes,
                       void* hip_stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * sarathi_hybrid_layer_forward with its workspace in a static device array
 * of SARATHI_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it
 * runs on until the process ends (looked up on the first call on a device).
 * The call allocates nothing; the caller still passes x_in, x_out, the
 * weights and the KV cache, with the same meaning, layout and KV contract
 * as sarathi_hybrid_layer_forward, and gets the same results.
 * Every call on one GPU shares that GPU's array: calls that overlap on one
 * GPU (different streams, or different host threads without ordering) race.
 * Errors: as sarathi_hybrid_layer_forward; ENOSPC when the batch needs more
 * workspace than the array holds (sarathi_workspace_bytes(cfg, T, B,
 * max_seq_len) > SARATHI_NOALLOC_SCRATCH_BYTES); EHIP if the array's device
 * address cannot be looked up.
 */
#define SARATHI_NOALLOC_SCRATCH_BYTES (160ull << 20)
int sarathi_hybrid_layer_forward_noalloc(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w,
                                         sarathi_kv* kv, int layer, const sarathi_hybrid_batch* batch,
                                         const void* x_in, void* x_out, void* hip_stream);

/*
 * sarathi_hybrid_layer_forward / sarathi_model_step over a mixed batch (any
 * number of prompt chunks, Sec. 5.2's mixed batching): the linear ops run
 * over all rows, each chunk's attention over its own slot, each decode over
 * its slot.  Same contract; the workspace is sized by
 * sarathi_mixed_workspace_layout for this batch's rows and chunk count.
 * Extra errors: EINVAL (n_chunks < 0 or > 65536, NULL chunk arrays), ERANGE
 * (a chunk length < 1).
 */
int sarathi_mixed_layer_forward(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w,
                                sarathi_kv* kv, int layer, const sarathi_mixed_batch* batch,
                                const void* x_in, void* x_out, void* ws, size_t ws_bytes,
                                void* hip_stream);
int sarathi_mixed_model_step(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w,
                             sarathi_kv* kv, const sarathi_mixed_batch* batch,
                             const void* x_in, void* x_out, void* ws, size_t ws_bytes,
                             void* hip_stream);

/* ------------------------------------------------------------------ building block */
/*
 * One linear op of the layer on its own (the fused matmuls of Sec. 4.3 with
 * their epilogues), for tests and per-op measurement:
 *   SARATHI_LINEAR_PLAIN   out[M,N] (dtype) = x W^T            (preproj)
 *   SARATHI_LINEAR_RESID   out[M,N] (fp32)  = resid (dtype) + x W^T  (postproj)
 *   SARATHI_LINEAR_RESID_F32IN out[M,N] (dtype) = resid (fp32) + x W^T (ffn_ln2)
 *   SARATHI_LINEAR_SWIGLU  out[M,N] (dtype) = silu(x Wg^T) * (x Wu^T), W = [Wg; Wu] [2N, K]
 *   SARATHI_LINEAR_GELU    out[M,N] (dtype) = gelu(x W^T)
 * x [M,K] dtype row-major, W [N or 2N, K] dtype; K multiple of 8.
 * `scratch`/`scratch_bytes`: device memory (16-byte aligned) for split-K
 * partials of the two residual kinds; with NULL or too small a buffer the op
 * runs without split-K (same result up to fp32 summation order, lower
 * occupancy at small M).  sarathi_linear_scratch_bytes(M, N) is the most it
 * can use (6 splits of M x N fp32).  Results are deterministic either way.
 */
#define SARATHI_LINEAR_PLAIN        0
#define SARATHI_LINEAR_RESID        1
#define SARATHI_LINEAR_RESID_F32IN  2
#define SARATHI_LINEAR_SWIGLU       3
#define SARATHI_LINEAR_GELU         4

size_t sarathi_linear_scratch_bytes(int M, int N);
int sarathi_linear(int dtype, int kind, int M, int N, int K, const void* x, const void* w,
                   const void* resid, void* out, void* scratch, size_t scratch_bytes,
                   void* hip_stream);

/*
 * The block shape (*bm rows of x by *bn rows of W) and K-split count that
 * sarathi_linear would run the op with, given scratch_bytes of split-K
 * scratch; nothing is launched.  sarathi_layer_split_scratch_bytes(cfg, T)
 * is the split-K scratch a layer call of T rows gives its two residual ops
 * (postproj, ffn_ln2), so the plan of a layer's op is
 * sarathi_linear_plan(..., sarathi_layer_split_scratch_bytes(cfg, T), ...).
 * For measurement: the fp32 partials of a split op (n_split x M x N x 4
 * bytes written, then read back) are traffic beyond the method's own.
 * Errors: EINVAL (NULL outputs, bad kind or sizes), EUNSUPPORTED (dtype,
 * K not a multiple of 8).
 */
int sarathi_linear_plan(int dtype, int kind, int M, int N, int K, size_t scratch_bytes, int* bm, int* bn,
                        int* n_split);
size_t sarathi_layer_split_scratch_bytes(const sarathi_model_cfg* cfg, int n_tokens);

/*
 * Tile shapes of the bf16 matmul kernel, for tests and tuning:
 * sarathi_linear_tile_count() shapes, shape t = *bm rows of x by *bn rows of
 * W per block (sarathi_linear_tile_shape returns EINVAL for t out of range).
 * sarathi_linear_tiled is sarathi_linear with the shape and K-split count
 * given instead of chosen by the library's cost model: dtype must be BF16 and
 * K a multiple of 64 (else EUNSUPPORTED); n_split >= 1 is used for the two
 * residual kinds when `scratch` holds n_split x M x N fp32 (capped at 6 and
 * at one split per 128 of K), and ignored for the other kinds.  Results
 * differ from sarathi_linear only in the fp32 summation order.
 */
int sarathi_linear_tile_count(void);
int sarathi_linear_tile_shape(int tile, int* bm, int* bn);
int sarathi_linear_tiled(int kind, int M, int N, int K, const void* x, const void* w, const void* resid,
                         void* out, void* scratch, size_t scratch_bytes, int tile, int n_split,
                         void* hip_stream);

/* ------------------------------------------------------------------ stage timing */
/*
 * Measurement hook: between sarathi_profile_begin and sarathi_profile_end,
 * every layer call (also each layer of sarathi_model_step) records a HIP
 * event on its stream before each of the SARATHI_N_STAGES stages and after
 * the last, from a host-side pool of (SARATHI_N_STAGES + 1) * max_calls
 * events (no device memory).  Calls beyond max_calls are not recorded.
 * sarathi_profile_end waits for the last recorded event, writes the summed
 * elapsed milliseconds of each stage over all recorded calls into
 * stage_ms[SARATHI_N_STAGES] and the number of recorded layer calls into
 * *n_calls, and stops recording.  Errors: EINVAL (bad max_calls, end without
 * begin, NULL outputs), EHIP.
 * Stages: 0 norm_1, 1 preproj, 2 rotary embedding + KV append, 3 chunk
 * attention, 4 decode attention, 5 combine of the attention key-splits,
 * 6 postproj, 7 norm_2, 8 ffn_ln1, 9 ffn_ln2.
 */
#define SARATHI_N_STAGES 10
int sarathi_profile_begin(int max_calls);
int sarathi_profile_end(double* stage_ms, int* n_calls);

/* ------------------------------------------------------------------ misc */
const char* sarathi_last_error(void);
int sarathi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SARATHI_H */
