// Attention of the decodes of the hybrid batch, run separately from the
// prompt chunk (Sec. 4.3).  It writes per-split partial results (max, sum,
// unnormalised o) that the combine pass of attention_combine.hip merges per
// row.
//
// Row attention (decodes; in fp32 runs also the chunk rows): each row attends
// to keys 0..pos of its slot.  Work item = (row, split of split_keys keys); a
// block of 4 (fp32) or 8 (bf16) waves streams its split, each wave 32 keys per
// pass with 16-byte non-temporal loads (a key row spread over hd*size/16
// lanes), partial dot products reduce-scattered across those lanes so each
// key's score ends up in two lanes, online softmax, then P*V accumulated per
// lane.  The block's wave states are merged in LDS into one partial.  attn_rows_kernel is the
// generic form (fp32 runs); attn_rows_bf16_kernel the bf16 one, with the
// arithmetic arranged for fewer vector-ALU instructions (see there).
#include "kernels.h"

namespace sarathi {

constexpr float LOG2E = 1.4426950408889634f;

// 16-byte load with the non-temporal hint (streamed data, read once).
typedef unsigned int u32x4_nt __attribute__((ext_vector_type(4)));
template <typename T>
__device__ __forceinline__ uint4 load_stream16(const T* p) {
  const u32x4_nt v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// ============================================================================ row attention
template <typename T, int D, int DUP>
__global__ __launch_bounds__(256) void attn_rows_kernel(RowAttnArgs a, float scale_log2) {
  constexpr int EPL = Vec16<T>::N;           // elements per lane per key (16 bytes)
  constexpr int LPK = D / EPL;               // lanes per key row
  constexpr int KPI = 64 / LPK;              // keys per wave load instruction
  constexpr int NI = LPK / DUP;              // load instructions per pass
  constexpr int KP = NI * KPI;               // keys per pass per wave (64 / DUP)
  static_assert(LPK * KPI == 64 && NI * DUP == LPK, "pass");
  __shared__ float red_m[4], red_l[4];
  __shared__ float red_o[4][D];

  const int item = blockIdx.x, h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane / LPK, j = lane % LPK;
  const int wv = a.work[item];
  const int row_rel = wv >> 12, split = wv & 4095;
  const int row = a.row_base + row_rel;
  const int slot = a.row_slot[row];
  const int nk = a.row_pos[row] + 1;
  const int kb = split * a.split_keys;
  const int ke = min(nk, kb + a.split_keys);

  const T* qkv = reinterpret_cast<const T*>(a.qkv);
  const T* cache = reinterpret_cast<const T*>(a.kv_layer);
  const T* kbase = cache + (size_t)slot * a.st.slot + (size_t)h * a.st.head + j * EPL;
  const T* vbase = kbase + a.st.kv;

  float q[EPL];
  Vec16<T>::unpack(*reinterpret_cast<const uint4*>(qkv + (size_t)row * a.ld_qkv + h * D + j * EPL), q);
#pragma unroll
  for (int e = 0; e < EPL; ++e) q[e] *= scale_log2;

  float m_run = -INFINITY, l_run = 0.f;
  float o[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) o[e] = 0.f;

  // Each wave takes passes of KP keys (pb, pb + 4*KP, ...).  All K loads are
  // issued first, then all V loads: the scores wait only for K (loads
  // complete in order) while V is still in flight.  Key addresses past the
  // split are clamped to its last key (finite data, masked below).  The KV
  // is read once per call, so its loads are non-temporal: they do not
  // allocate in the memory-side cache, which neither evicts what other
  // kernels left there nor forces the write-back of their dirty lines in the
  // middle of this stream (measured: 12% faster alone, and 32-128 MB of
  // writes by the kernel before it no longer slow it down).
  for (int pb = kb + wave * KP; pb < ke; pb += 4 * KP) {
    uint4 kr[NI], vr[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i)
      kr[i] = load_stream16(kbase + (size_t)min(pb + i * KPI + g, ke - 1) * a.st.pos);
#pragma unroll
    for (int i = 0; i < NI; ++i)
      vr[i] = load_stream16(vbase + (size_t)min(pb + i * KPI + g, ke - 1) * a.st.pos);
    // Keep all 2*NI loads in flight before any use (the scheduler would
    // otherwise sink each load next to its first use and serialise them).
    __builtin_amdgcn_sched_barrier(0);
    float part[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      float kf[EPL];
      Vec16<T>::unpack(kr[i], kf);
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc = fmaf(q[e], kf[e], acc);
      part[i] = acc;
    }
    // Reduce-scatter across the LPK lanes of a key group: afterwards the
    // DUP lanes j with j / DUP == i hold the full score of the key loaded
    // by instruction i.
#pragma unroll
    for (int n = NI, msk = LPK / 2; n > 1; n >>= 1, msk >>= 1) {
#pragma unroll
      for (int idx = 0; idx < n / 2; ++idx) {
        const bool upper = (j & msk) != 0;
        const float keep = upper ? part[idx + n / 2] : part[idx];
        const float send = upper ? part[idx] : part[idx + n / 2];
        part[idx] = keep + __shfl_xor(send, msk, 64);
      }
    }
#pragma unroll
    for (int msk = DUP / 2; msk >= 1; msk >>= 1) part[0] += __shfl_xor(part[0], msk, 64);
    const int mykey = pb + (j / DUP) * KPI + g;
    const bool own = (j % DUP) == 0;            // one lane per key counts in the sum
    const float sc = (mykey < ke) ? part[0] : -INFINITY;
    const float m_new = fmaxf(m_run, wave_max(sc));
    const float m_safe = (m_new == -INFINITY) ? 0.f : m_new;
    const float corr = exp2f(m_run - m_safe);
    const float pk = (mykey < ke) ? exp2f(sc - m_safe) : 0.f;
    l_run = l_run * corr + wave_sum(own ? pk : 0.f);
    m_run = m_new;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[e] *= corr;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const float w = __shfl(pk, g * LPK + i * DUP, 64);
      float vf[EPL];
      Vec16<T>::unpack(vr[i], vf);
#pragma unroll
      for (int e = 0; e < EPL; ++e) o[e] = fmaf(w, vf[e], o[e]);
    }
  }
  // Sum o over the KPI key groups of the wave.
#pragma unroll
  for (int msk = LPK; msk < 64; msk <<= 1)
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[e] += __shfl_xor(o[e], msk, 64);

  if (lane == 0) {
    red_m[wave] = m_run;
    red_l[wave] = l_run;
  }
  if (g == 0) {
#pragma unroll
    for (int e = 0; e < EPL; ++e) red_o[wave][j * EPL + e] = o[e];
  }
  __syncthreads();
  float M = fmaxf(fmaxf(red_m[0], red_m[1]), fmaxf(red_m[2], red_m[3]));
  const float Ms = (M == -INFINITY) ? 0.f : M;
  float* dst = a.part + ((size_t)(a.part_base + item) * a.nh + h) * (D + PART_O);
  for (int d = tid; d < D; d += 256) {
    float acc = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) acc += red_o[w][d] * exp2f(red_m[w] - Ms);
    dst[PART_O + d] = acc;
  }
  if (tid == 0) {
    float L = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) L += red_l[w] * exp2f(red_m[w] - Ms);
    dst[0] = M;
    dst[1] = L;
  }
}

// ---------------------------------------------------------------------------- bf16 row attention
// DPP lane exchanges inside 16-lane rows.  For mask bit b the partner differs
// from the lane in bit b (and only in bits <= b): b = 3 row_mirror (i <->
// 15 - i), b = 2 row_half_mirror (i <-> 7 - i within 8), b = 1 quad_perm
// [3,2,1,0], b = 0 quad_perm [1,0,3,2]; a butterfly over b = 3 .. 0 reaches all
// 16 lanes, over b = 2 .. 0 all 8 of a half row.
template <int MSK>
__device__ __forceinline__ float row_xchg(float v) {
  constexpr int CTRL = MSK == 8 ? 0x140 : MSK == 4 ? 0x141 : MSK == 2 ? 0x1B : 0xB1;
  return __builtin_amdgcn_update_dpp(0.f, v, CTRL, 0xf, 0xf, false);
}
// Lane l of each 16-lane row broadcast to the row (row_newbcast); l is a
// compile-time constant wherever the loops are unrolled.
template <int L>
__device__ __forceinline__ float row_bcast_c(float v) {
  return __builtin_amdgcn_update_dpp(0.f, v, 0x150 + L, 0xf, 0xf, false);
}
__device__ __forceinline__ float row_bcast(float v, int l) {
  switch (l & 15) {
    case 0: return row_bcast_c<0>(v);
    case 1: return row_bcast_c<1>(v);
    case 2: return row_bcast_c<2>(v);
    case 3: return row_bcast_c<3>(v);
    case 4: return row_bcast_c<4>(v);
    case 5: return row_bcast_c<5>(v);
    case 6: return row_bcast_c<6>(v);
    case 7: return row_bcast_c<7>(v);
    case 8: return row_bcast_c<8>(v);
    case 9: return row_bcast_c<9>(v);
    case 10: return row_bcast_c<10>(v);
    case 11: return row_bcast_c<11>(v);
    case 12: return row_bcast_c<12>(v);
    case 13: return row_bcast_c<13>(v);
    case 14: return row_bcast_c<14>(v);
    default: return row_bcast_c<15>(v);
  }
}
template <int LPK>
__device__ __forceinline__ float group_max(float v) {
  if constexpr (LPK >= 16) v = fmaxf(v, row_xchg<8>(v));
  v = fmaxf(v, row_xchg<4>(v));
  v = fmaxf(v, row_xchg<2>(v));
  return fmaxf(v, row_xchg<1>(v));
}
template <int LPK>
__device__ __forceinline__ float group_sum(float v) {
  if constexpr (LPK >= 16) v += row_xchg<8>(v);
  v += row_xchg<4>(v);
  v += row_xchg<2>(v);
  return v + row_xchg<1>(v);
}
// Reduce-scatter of part[0 .. N) over the lanes of a key row, levels
// MSK = N*DUP/2 .. DUP: after it, part[0] of the lanes j with j / DUP == i
// holds (half of) the sum of part[i] over the row.
template <int N, int MSK>
__device__ __forceinline__ void reduce_scatter(float* part, int j) {
  if constexpr (N > 1) {
    const bool upper = (j & MSK) != 0;
#pragma unroll
    for (int idx = 0; idx < N / 2; ++idx) {
      const float lo = part[idx], hi = part[idx + N / 2];
      const float keep = upper ? hi : lo, send = upper ? lo : hi;
      part[idx] = keep + row_xchg<MSK>(send);
    }
    reduce_scatter<N / 2, MSK / 2>(part, j);
  }
}

// a.lo * b.lo + a.hi * b.hi + c for two bf16 pairs (v_dot2_f32_bf16: the
// bf16 products are exact in fp32, the sums are fp32).
typedef __bf16 bf16x2_dot __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_dot, a), __builtin_bit_cast(bf16x2_dot, b), c,
                                         false);
}

// The bf16 kernel: same work items, lanes and partials as attn_rows_kernel,
// with half the vector-ALU instructions per pass:
//   q.k on v_dot2_f32_bf16 (two exact bf16 products per instruction, fp32
//   sums), the unscaled bf16 q straight from the workspace;
//   the reduce-scatter and the softmax reductions on DPP row exchanges (no
//   LDS round trips, no lane-index arithmetic);
//   each group of LPK lanes (the key rows of one load instruction) keeps its
//   own running max and sum, so a pass reduces over 16 lanes, not 64, and a
//   key's probability reaches the group's lanes by a row broadcast; the
//   groups are merged once at the end;
//   P V stays fp32 (probabilities and V unpacked to fp32).
template <int D, int NWV>
__global__ __launch_bounds__(64 * NWV) void attn_rows_bf16_kernel(RowAttnArgs a, float scale_log2) {
  constexpr int LPK = D / 8;                 // lanes per key row (8 bf16 per lane)
  constexpr int KPI = 64 / LPK;              // keys per wave load instruction
  constexpr int DUP = 2;                     // lanes holding each key's score
  constexpr int NI = LPK / DUP;              // load instructions per pass (K, and V)
  constexpr int KP = NI * KPI;               // keys per pass per wave
  static_assert(LPK == 16 || LPK == 8, "head_dim 128 or 64");
  __shared__ float red_m[NWV], red_l[NWV];
  __shared__ float red_o[NWV][D];

  // one block per (work item, head), heads fastest: the blocks in flight
  // stream the same key range of one slot for all its heads (measured ~2%
  // faster than items fastest)
  const int item = blockIdx.x / a.nh, h = blockIdx.x % a.nh;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane / LPK, j = lane % LPK;
  const int wv = a.work[item];
  const int row_rel = wv >> 12, split = wv & 4095;
  const int row = a.row_base + row_rel;
  const int slot = a.row_slot[row];
  const int nk = a.row_pos[row] + 1;
  const int kb = split * a.split_keys;
  const int ke = min(nk, kb + a.split_keys);

  const bf16* qkv = reinterpret_cast<const bf16*>(a.qkv);
  const bf16* cache = reinterpret_cast<const bf16*>(a.kv_layer);
  const bf16* kbase = cache + (size_t)slot * a.st.slot + (size_t)h * a.st.head + j * 8;
  const bf16* vbase = kbase + a.st.kv;
  const uint4 qv = *reinterpret_cast<const uint4*>(qkv + (size_t)row * a.ld_qkv + h * D + j * 8);
  const uint32_t pos_stride = (uint32_t)a.st.pos;

  float m_run = -INFINITY, l_run = 0.f;     // of this lane's key group
  float o[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = 0.f;

  // Passes of KP keys per wave (pb, pb + NWV*KP, ...): all K loads, then all V
  // loads, non-temporal (see attn_rows_kernel); addresses past the split are
  // clamped to its last key (finite data, masked below).
  for (int pb = kb + wave * KP; pb < ke; pb += NWV * KP) {
    uint4 kr[NI], vr[NI];
    // element offsets in 32 bits: positions < 2^20, position stride = head_dim
    uint32_t off[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) off[i] = (uint32_t)min(pb + i * KPI + g, ke - 1) * pos_stride;
#pragma unroll
    for (int i = 0; i < NI; ++i) kr[i] = load_stream16(kbase + off[i]);
#pragma unroll
    for (int i = 0; i < NI; ++i) vr[i] = load_stream16(vbase + off[i]);
    __builtin_amdgcn_sched_barrier(0);
    float part[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      float acc = dot2_bf16(qv.x, kr[i].x, 0.f);
      acc = dot2_bf16(qv.y, kr[i].y, acc);
      acc = dot2_bf16(qv.z, kr[i].z, acc);
      part[i] = dot2_bf16(qv.w, kr[i].w, acc);
    }
    reduce_scatter<NI, LPK / 2>(part, j);
    part[0] += row_xchg<1>(part[0]);         // the DUP = 2 lanes of a key
    const int mykey = pb + (j / DUP) * KPI + g;
    const bool valid = mykey < ke;
    const float sc = valid ? part[0] * scale_log2 : -INFINITY;
    const float m_new = fmaxf(m_run, group_max<LPK>(sc));
    const float m_safe = (m_new == -INFINITY) ? 0.f : m_new;
    const float corr = exp2f(m_run - m_safe);
    const float pk = valid ? exp2f(sc - m_safe) : 0.f;
    l_run = l_run * corr + group_sum<LPK>((j % DUP) == 0 ? pk : 0.f);
    m_run = m_new;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] *= corr;
    // P V: key i's probability sits in lane i * DUP of the group.
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      float w;
      if constexpr (LPK == 16) w = row_bcast(pk, i * DUP);
      else w = __shfl(pk, g * LPK + i * DUP, 64);
      float vf[8];
      Vec16<bf16>::unpack(vr[i], vf);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = fmaf(w, vf[e], o[e]);
    }
  }
  // Merge the KPI key groups of the wave (lanes j, j + LPK, ...).
  float M = m_run;
#pragma unroll
  for (int msk = LPK; msk < 64; msk <<= 1) M = fmaxf(M, __shfl_xor(M, msk, 64));
  const float Mw = (M == -INFINITY) ? 0.f : M;
  const float sg = exp2f(m_run - Mw);
  float L = l_run * sg;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] *= sg;
#pragma unroll
  for (int msk = LPK; msk < 64; msk <<= 1) {
    L += __shfl_xor(L, msk, 64);
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] += __shfl_xor(o[e], msk, 64);
  }

  if (lane == 0) {
    red_m[wave] = M;
    red_l[wave] = L;
  }
  if (g == 0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) red_o[wave][j * 8 + e] = o[e];
  }
  __syncthreads();
  float Mb = red_m[0];
#pragma unroll
  for (int w = 1; w < NWV; ++w) Mb = fmaxf(Mb, red_m[w]);
  const float Ms = (Mb == -INFINITY) ? 0.f : Mb;
  float* dst = a.part + ((size_t)(a.part_base + item) * a.nh + h) * (D + PART_O);
  for (int d = tid; d < D; d += 64 * NWV) {
    float acc = 0.f;
#pragma unroll
    for (int w = 0; w < NWV; ++w) acc += red_o[w][d] * exp2f(red_m[w] - Ms);
    dst[PART_O + d] = acc;
  }
  if (tid == 0) {
    float Lb = 0.f;
#pragma unroll
    for (int w = 0; w < NWV; ++w) Lb += red_l[w] * exp2f(red_m[w] - Ms);
    dst[0] = Mb;
    dst[1] = Lb;
  }
}

template <typename T, int D>
static hipError_t run_rows(const RowAttnArgs& a, hipStream_t s) {
  const float scale_log2 = LOG2E / sqrtf((float)D);
  hipLaunchKernelGGL((attn_rows_kernel<T, D, 2>), dim3(a.n_work, a.nh), dim3(256), 0, s, a, scale_log2);
  return hipGetLastError();
}

hipError_t launch_attn_rows(int dtype, const RowAttnArgs& a, hipStream_t s) {
  if (a.n_work <= 0) return hipSuccess;
  if (dtype == 0) return a.hd == 128 ? run_rows<float, 128>(a, s) : run_rows<float, 64>(a, s);
  const float scale_log2 = LOG2E / sqrtf((float)a.hd);
  constexpr int NWV = 8;
  const unsigned grid = (unsigned)((size_t)a.n_work * a.nh);
  if (a.hd == 128)
    hipLaunchKernelGGL((attn_rows_bf16_kernel<128, NWV>), dim3(grid), dim3(64 * NWV), 0, s, a, scale_log2);
  else
    hipLaunchKernelGGL((attn_rows_bf16_kernel<64, NWV>), dim3(grid), dim3(64 * NWV), 0, s, a, scale_log2);
  return hipGetLastError();
}

}  // namespace sarathi
