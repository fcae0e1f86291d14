// Attention of the prompt chunk(s) of the hybrid batch, run separately from the
// decodes (Sec. 4.3).  It writes per-split partial results (max, sum,
// unnormalised o) that the combine pass of attention_combine.hip merges per row.
//
// Chunked-prefill attention (bf16, MFMA): the chunk's queries at positions
// off..off+C-1 attend to the prefill slot's keys 0..position (the earlier
// chunks' cached keys plus, causally, the chunk's own; Sec. 4.2).  Work item
// = (block of PREFILL_QBLOCK queries, a range of 64-key tiles), one head per
// block of PREFILL_QBLOCK / 16 waves x 16 query rows.  K and V tiles of 64
// keys are staged in a ring of LDS stages by LDS DMA (V read back transposed
// so P*V takes 16 contiguous bytes per lane); S = Q K^T and O += P V run on
// v_mfma_f32_16x16x32_bf16 with an fp32 online softmax.
#include "kernels.h"

namespace sarathi {

constexpr float LOG2E = 1.4426950408889634f;

// ============================================================================ prefill (bf16, MFMA)
typedef short v4i16 __attribute__((ext_vector_type(4)));

// Two fp32 -> one dword of two bf16 (round to nearest even; low half = a).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// LDS transpose read (gfx950): within each group of 16 lanes, output lane j
// element e is element (j % 4) of the 8 bytes addressed by lane 4e + j / 4.
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
__device__ __forceinline__ uint2 lds_read_tr16(const void* p) {
  const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p));
  return __builtin_bit_cast(uint2, v);
}

// One block = one head x (16 * NW queries of the chunk, one split of keys);
// wave w owns queries w*16..w*16+15.  Per 64-key tile:
//   S^T = K Q^T  (MFMA: A = K rows from LDS, B = the wave's Q fragments), so
//     each lane holds 16 scores of ONE query (lane % 16) for keys
//     nt*16 + 4*(lane/16) + i;
//   the online softmax runs on that query's own registers (+2 lane shuffles);
//   O^T += V^T P^T (MFMA: B = the lane's probabilities packed as bf16x8
//     straight from registers; A = V^T fragments read from the row-major V
//     tile with LDS transpose reads).  The k order of this product is a
//     permutation of the 32 keys of a block: lane group g holds keys
//     4g..4g+3 and 16+4g..16+4g+3, which is what two transpose reads of rows
//     4g..4g+3 and 16+4g..16+4g+3 deliver.
// K and V tiles are stored row-major (16-byte chunks XOR-swizzled by row) in
// an S-stage LDS ring filled by LDS DMA (global_load_lds_dwordx4: a wave
// instruction fills 1 KB = 1024 / (2 D) key rows; lane i takes LDS slot i of
// its row and so reads the chunk that the swizzle puts there), S - 1 tiles in
// flight while one is used; one barrier per tile.  Registers are capped at
// 128 per lane (four waves per SIMD) so that two blocks share a CU.
template <int D, int NW, int S>
__global__ __launch_bounds__(64 * NW, 4) void attn_prefill_bf16_kernel(PrefillArgs a, float scale_log2) {
  constexpr int QB = 16 * NW;            // the block's queries (chunk rows)
  constexpr int KT = 64;                 // keys per tile
  constexpr int DCH = D / 8;             // 16-byte chunks per K/V row
  constexpr int TILE = KT * DCH;         // 16-byte chunks per K (or V) tile
  constexpr int RPI = 64 / DCH;          // key rows per 1 KB DMA instruction
  constexpr int GRP = 2 * KT / RPI;      // 1 KB groups per K+V tile pair
  constexpr int NI = GRP / NW;           // DMA instructions per wave per tile
  static_assert(NI * NW == GRP && (S - 2) * NI < 64 && S >= 2, "tile DMA split");
  extern __shared__ u32x4 ring[];        // [S][K tile, V tile]

  const int per = gridDim.x / 8;
  const int t = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (t >= a.n_work * a.nh) return;
  const int item = t % a.n_work, h = t / a.n_work;
  const int* wk = a.work + 4 * item;
  const int* ch = a.chunks + 4 * wk[0];
  const int slot = ch[0], offset = ch[1], C = ch[2], row0 = ch[3];
  const int q0 = wk[1] * QB, pslot = wk[2];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = lane >> 4, ql = lane & 15;
  const bf16* qkv = reinterpret_cast<const bf16*>(a.qkv) + (size_t)row0 * a.ld_qkv;
  const bf16* cache = reinterpret_cast<const bf16*>(a.kv_layer);
  const bf16* kbase = cache + (size_t)slot * a.st.slot + (size_t)h * a.st.head;
  const bf16* vbase = kbase + a.st.kv;

  // This item's keys: tiles [t0, t1) of 0 .. off + min(q0 + QB, C) - 1.
  const int n_keys = offset + min(q0 + QB, C);
  const int kbeg = (wk[3] >> 16) * KT;
  const int kend = min(n_keys, (wk[3] & 0xffff) * KT);
  const int n_tiles = (kend - kbeg + KT - 1) / KT;

  // The lane's query (B operand of S^T): q = ql, d = ks*32 + 8*grp.
  const int myq = q0 + wave * 16 + ql;
  const int qpos = offset + myq;
  u32x4 qf[D / 32];
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(qkv + (size_t)min(myq, C - 1) * a.ld_qkv + h * D + ks * 32 + 8 * grp);
    qf[ks] = (myq < C) ? v : u32x4{0u, 0u, 0u, 0u};
  }

  float m_run = -INFINITY, l_run = 0.f;
  floatx4 o_acc[D / 16];                 // O^T[d = dt*16 + 4*grp + i][q = ql]
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) o_acc[dt] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Tile DMA: instruction j of wave w fills 1 KB group g = j * NW + w of the
  // tile pair (K groups first, then V).  Key addresses are clamped to the
  // item's last key (finite data; such keys are masked out of the softmax).
  const int lrow = lane / DCH, lslot = lane % DCH;
  const bf16* dsrc[NI];
  int drow[NI];
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    const int g = j * NW + wave;
    const int kv = g / (KT / RPI), row = (g % (KT / RPI)) * RPI + lrow;
    drow[j] = row;
    dsrc[j] = (kv ? vbase : kbase) + (lslot ^ (row & 7)) * 8;
  }
  auto issue = [&](int stage, int kt) {
    const int k0 = kbeg + kt * KT;
    uint4* dst = reinterpret_cast<uint4*>(ring + stage * 2 * TILE);
#pragma unroll
    for (int j = 0; j < NI; ++j)
      dma16(dsrc[j] + (size_t)min(k0 + drow[j], kend - 1) * a.st.pos, dst + (j * NW + wave) * 64);
  };

  // Transpose-read addressing of V^T fragments: lane i of group grp reads 8
  // bytes of row 4*grp + i/4 (+16 for the second half) at columns
  // dt*16 + 4*(i%4) .. +3.
  const int tr_row = 4 * grp + (ql >> 2);
  const int tr_c16 = (ql & 3) >> 1;      // 16-byte chunk within the 16 columns of dt
  const int tr_half = (ql & 1) * 8;      // byte offset inside the chunk

#pragma unroll
  for (int st = 0; st < S - 1; ++st)
    if (st < n_tiles) issue(st, st);
  int buf = 0, nbuf = S - 1;
  for (int kt = 0; kt < n_tiles; ++kt) {
    const int k0 = kbeg + kt * KT;
    if (kt + S - 2 < n_tiles) wait_vmcnt<(S - 2) * NI>();
    else wait_vmcnt<0>();
    lds_read_barrier();
    if (kt + S - 1 < n_tiles) issue(nbuf, kt + S - 1);
    const u32x4* ks_ = ring + buf * 2 * TILE;
    const u32x4* vs_ = ks_ + TILE;
    buf = (buf + 1 == S) ? 0 : buf + 1;
    nbuf = (nbuf + 1 == S) ? 0 : nbuf + 1;

    // ---- S^T = K Q^T: s[nt][i] = score of key k0 + nt*16 + 4*grp + i for query ql.
    floatx4 s[KT / 16];
#pragma unroll
    for (int nt = 0; nt < KT / 16; ++nt) {
      s[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
      const int key = nt * 16 + ql;
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        const int ch = ks * 4 + grp;
        const bf16x8_t kf = __builtin_bit_cast(bf16x8_t, ks_[key * DCH + (ch ^ (key & 7))]);
        s[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, __builtin_bit_cast(bf16x8_t, qf[ks]), s[nt], 0, 0, 0);
      }
    }

    // ---- online softmax (log2 units).  Keys past the query's position or the
    // item's end are masked; a tile entirely before every query of the wave
    // and inside the item needs no mask.
    const bool full = k0 + KT <= kend && k0 + KT - 1 <= offset + q0 + wave * 16;
    if (!full) {
#pragma unroll
      for (int nt = 0; nt < KT / 16; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int kp = k0 + nt * 16 + 4 * grp + i;
          if (!(kp <= qpos && kp < kend)) s[nt][i] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int nt = 0; nt < KT / 16; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) mx = fmaxf(mx, s[nt][i]);
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx * scale_log2);
    const float m_safe = (m_new == -INFINITY) ? 0.f : m_new;
    const float corr = __builtin_amdgcn_exp2f(m_run - m_safe);
    float sum = 0.f;
#pragma unroll
    for (int nt = 0; nt < KT / 16; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s[nt][i] = __builtin_amdgcn_exp2f(fmaf(s[nt][i], scale_log2, -m_safe));
        sum += s[nt][i];
      }
    sum += __shfl_xor(sum, 16, 64);
    sum += __shfl_xor(sum, 32, 64);
    l_run = l_run * corr + sum;
    m_run = m_new;
    if (__ballot(corr != 1.0f)) {
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) o_acc[dt] *= corr;
    }

    // ---- O^T += V^T P^T over two 32-key blocks.
    const char* vb = reinterpret_cast<const char*>(vs_);
#pragma unroll
    for (int kk = 0; kk < KT / 32; ++kk) {
      // probabilities to bf16 (round to nearest even, v_cvt_pk_bf16_f32)
      const u32x4 pw{pack_bf16x2(s[2 * kk][0], s[2 * kk][1]), pack_bf16x2(s[2 * kk][2], s[2 * kk][3]),
                     pack_bf16x2(s[2 * kk + 1][0], s[2 * kk + 1][1]), pack_bf16x2(s[2 * kk + 1][2], s[2 * kk + 1][3])};
      const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, pw);
      const int r0 = kk * 32 + tr_row, r1 = r0 + 16;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const int c16 = 2 * dt + tr_c16;
        const uint2 lo = lds_read_tr16(vb + (r0 * DCH + (c16 ^ (r0 & 7))) * 16 + tr_half);
        const uint2 hi = lds_read_tr16(vb + (r1 * DCH + (c16 ^ (r1 & 7))) * 16 + tr_half);
        const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, u32x4{lo.x, lo.y, hi.x, hi.y});
        o_acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, o_acc[dt], 0, 0, 0);
      }
    }
  }

  // ---- partial of the lane's query (rows < C): [m, l, o[D]].
  const int rb = wave * 16 + ql;
  if (q0 + rb < C) {
    float* dst = a.part + ((size_t)(pslot * QB + rb) * a.nh + h) * (D + 2);
    if (grp == 0) {
      dst[0] = m_run;
      dst[1] = l_run;
    }
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) dst[2 + dt * 16 + 4 * grp + i] = o_acc[dt][i];
  }
}

template <int D, int NW, int S>
static hipError_t run_prefill(const PrefillArgs& a, unsigned grid, float scale_log2, hipStream_t s) {
  const size_t lds_bytes = (size_t)S * 2 * 64 * (D / 8) * 16;
  static std::atomic<uint64_t> lds_set{0};   // devices on which this instance's LDS limit is raised
  hipError_t e = ensure_dynamic_lds((const void*)attn_prefill_bf16_kernel<D, NW, S>, (int)lds_bytes, lds_set);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_prefill_bf16_kernel<D, NW, S>), dim3(grid), dim3(64 * NW), lds_bytes, s, a, scale_log2);
  return hipGetLastError();
}

hipError_t launch_attn_prefill(int dtype, const PrefillArgs& a, hipStream_t s) {
  if (a.n_work <= 0) return hipSuccess;
  if (dtype != 1) return hipErrorInvalidValue;
  const float scale_log2 = LOG2E / sqrtf((float)a.hd);
  const unsigned grid = (unsigned)(((size_t)a.n_work * a.nh + 7) / 8 * 8);
  constexpr int NW = PREFILL_QBLOCK / 16;
  // two stages (64 KB for head_dim 128): two blocks per CU
  if (a.hd == 128) return run_prefill<128, NW, 2>(a, grid, scale_log2, s);
  return run_prefill<64, NW, 2>(a, grid, scale_log2, s);
}

}  // namespace sarathi
