// Host-side launchers of the gfx950 kernels (implemented in the .hip files).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.h"

namespace sarathi {

// ---- batch metadata (int32 arrays in the workspace), written by a kernel
// whose arguments carry the host values (stream-ordered, no staging buffer).
// 8 KB of kernel arguments per launch: one launch covers the metadata of a
// batch of ~350 rows (5 ints per row plus the work lists); ROCm passes
// argument structs of this size (measured: one 8 KB launch costs about as much
// as one small launch, against three for 2.5 KB pieces).
constexpr int META_CHUNK = 2040;
struct MetaChunk {
  int count;
  int values[META_CHUNK];
};
hipError_t launch_meta_write(const MetaChunk& chunk, int* dst, hipStream_t s);

// ---- norms (one row per block).  in: [rows, H] of Tin; out: [rows, H] of dtype.
// With meta non-null the same launch also copies that metadata chunk to
// meta_dst (one extra block).
hipError_t launch_norm(int dtype, bool in_f32, bool layer_norm, const void* in, const void* g,
                       const void* b, void* out, int rows, int H, float eps, hipStream_t s,
                       const MetaChunk* meta = nullptr, int* meta_dst = nullptr);

// ---- rotary embedding of q, k in place of the preproj output and K/V append.
struct RopeArgs {
  void* qkv;            // [T, 3*nh*hd]
  int T, nh, hd;
  int rope;
  float base;
  const int* row_slot;  // [T]
  const int* row_pos;   // [T]
  void* kv_layer;       // base of this layer's cache
  KVStrides st;
};
hipError_t launch_rope_append(int dtype, const RopeArgs& a, hipStream_t s);

// ---- a norm applied to a linear op's output (rows of N): out = norm(y) * g (+ b).
struct NormArgs {
  const void* g;
  const void* b;        // LayerNorm only
  void* out;            // [M, N] dtype
  float eps;
  bool layer;           // LayerNorm (else RMSNorm)
};

// ---- linear ops (see sarathi.h for the kinds).
enum LinearKind { LIN_PLAIN = 0, LIN_RESID = 1, LIN_RESID_F32IN = 2, LIN_SWIGLU = 3, LIN_GELU = 4 };
struct LinearArgs {
  int kind;
  int M, N, K;          // N = output columns
  const void* x;        // [M, K]
  const void* w;        // [N or 2N, K]
  const void* resid;    // LIN_RESID: dtype [M,N]; LIN_RESID_F32IN: fp32 [M,N]
  void* out;            // LIN_RESID: fp32 [M,N]; others dtype [M,N]
  float* parts;         // residual kinds: fp32 scratch for split-K partials (null: no split-K)
  size_t parts_cap;     // its capacity in floats
  // LIN_PLAIN preproj (bf16), optional: rotary embedding + KV append fused
  // into the epilogue when head_dim is a multiple of 16 and N = 3 nh hd
  // (producer/consumer kernel; then *rope_done = true,
  // only the q columns of out are written; else the caller runs
  // launch_rope_append).
  const RopeArgs* rope;
  bool* rope_done;
  // LIN_RESID / LIN_RESID_F32IN (bf16), optional: the norm of the output
  // rows folded into the split-K reduction pass when the op runs split over
  // K (then *norm_done = true and norm->out holds the normalised rows; else
  // the caller runs the norm).
  const NormArgs* norm;
  bool* norm_done;
};
constexpr int MAX_SPLIT = 6;   // split-K partials: at most MAX_SPLIT x [M, N] fp32
// force_tile >= 0 (bf16, K a multiple of 64): run that producer/consumer tile
// shape with force_split K-splits (residual kinds with scratch) instead of the
// cost model's choice.
// With plan non-null nothing is launched: *plan receives the block shape and
// K-split count the op would run with (bm = bn = 0 for the fp32 kernel's
// 64 x 64 tiles is reported as 64, 64).
struct LinearPlan {
  int bm, bn, n_split;
};
hipError_t launch_linear(int dtype, const LinearArgs& a, hipStream_t s, int force_tile = -1, int force_split = 0,
                         LinearPlan* plan = nullptr);
int linear_tile_count();
bool linear_tile_shape(int tile, int* bm, int* bn);

// ---- attention
// Partial results (one per row x head x key split): [m, l, -, -, o[hd]] in
// fp32 (hd + PART_O floats, so o starts 16-byte aligned), m the running max
// of the log2-scaled scores, l the sum of 2^(s - m), o the unnormalised
// weighted sum of values.
constexpr int PART_O = 4;
// Chunk rows per chunk-attention work item: 256 (8 waves x 32 queries, two
// waves per SIMD) for long chunks and long prefixes, 128 (4 waves x 32, one
// per SIMD, a smaller block set-up and output) for short ones; the host's plan
// picks one per batch.  Buffers are sized for the larger.
constexpr int PREFILL_QBLOCK = 256;
constexpr int PREFILL_QBLOCK_SMALL = 128;
struct PrefillArgs {
  const void* qkv;      // all rows; chunk c's rows start at its first-row entry; q columns rotated
  int ld_qkv;
  const void* kv_layer;
  KVStrides st;
  const int* chunks;    // [n_chunks][slot, offset, len, first row]
  int nh, hd;
  const int* work;      // [n_work][chunk, q_block, partial slot p, (first key tile << 16) | end key tile]
  int n_work;
  int qblock;           // rows per q-block: PREFILL_QBLOCK or PREFILL_QBLOCK_SMALL
  float* part;          // row j of an item's q-block -> partial index p * qblock + j
  void* out;            // p < 0 (the item covers every key of its rows): normalised rows of O [T, nh*hd]
  int ld_out;
};
hipError_t launch_attn_prefill(int dtype, const PrefillArgs& a, hipStream_t s);

// Row attention: each row r in [row_base, row_base + n_rows) attends to keys
// 0..row_pos[r] of slot row_slot[r], split into work items of split_keys keys.
struct RowAttnArgs {
  const void* qkv;
  int ld_qkv;
  const void* kv_layer;
  KVStrides st;
  const int* row_slot;
  const int* row_pos;
  const int* work;      // [n_work] (row_rel << 12) | split
  int row_base, n_work, split_keys, nh, hd;
  float* part;          // work item w -> partial index part_base + w
  int part_base;
};
hipError_t launch_attn_rows(int dtype, const RowAttnArgs& a, hipStream_t s);

// Combine: row r's partials are comb[3r] + j * comb[3r + 2] for j < comb[3r + 1];
// rows with no partials (comb[3r + 1] == 0: written by their attention kernel)
// are left alone.  Rows row0 .. n_rows - 1 are visited.
struct CombineArgs {
  const float* part;
  const int* comb;
  int row0, n_rows, nh, hd;
  void* out;            // [n_rows, nh * hd]
  int ld_out;
};
hipError_t launch_attn_combine(int dtype, const CombineArgs& a, hipStream_t s);

// out[i] = resid[i] + sum_{s < n_split} parts[s * n + i], summed in split order
// (resid: fp32 if resid_f32 else dtype; out: fp32 if out_f32 else dtype).
hipError_t launch_split_reduce(int dtype, bool resid_f32, bool out_f32, const void* resid, const float* parts,
                               int n_split, size_t n, void* out, hipStream_t s);
// The same for rows x N plus the norm of each output row in the same pass
// (one block per row): bf16 residual and fp32 out, or (resid_f32) fp32
// residual and bf16 out, normalised as rounded.  Returns
// hipErrorNotSupported (nothing launched) when N does not fit one block.
hipError_t launch_split_reduce_norm(const void* resid, bool resid_f32, const float* parts, int n_split, int rows,
                                    int N, void* out, const NormArgs& norm, hipStream_t s);

}  // namespace sarathi
