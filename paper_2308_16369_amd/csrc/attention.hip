// Attention of the hybrid batch, run separately for the prefill chunk and for
// the decodes (Sec. 4.3).  Both write per-split partial results
// (max, sum, unnormalised o) that one combine pass merges per row.
//
// Chunked-prefill attention (bf16, MFMA): the chunk's queries at positions
// off..off+C-1 attend to the prefill slot's keys 0..position (the earlier
// chunks' cached keys plus, causally, the chunk's own; Sec. 4.2).  Work item
// = (64-query block, split of split_keys keys), one head per block of 4
// waves x 16 query rows.  K and V tiles of 64 keys are staged in LDS (V
// transposed so P*V reads 16 contiguous bytes per lane), the next tile is
// prefetched into registers while the current one is used; S = Q K^T and
// O += P V run on v_mfma_f32_16x16x32_bf16 with an fp32 online softmax.
//
// Row attention (decodes; in fp32 runs also the chunk rows): each row attends
// to keys 0..pos of its slot.  Work item = (row, split of split_keys keys); a
// block of 4 waves streams its split, each wave 64 keys per pass with 16-byte
// loads (a key row spread over hd*size/16 lanes), partial dot products
// reduce-scattered across those lanes so every lane ends up with one key's
// score, wave-level online softmax, then P*V accumulated per lane.  The
// block's four wave states are merged in LDS into one partial.
#include "kernels.h"

namespace sarathi {

constexpr float LOG2E = 1.4426950408889634f;

// ============================================================================ prefill (bf16, MFMA)
template <int D>
__global__ __launch_bounds__(256) void attn_prefill_bf16_kernel(PrefillArgs a, float scale_log2) {
  constexpr int KT = 64;                 // keys per tile
  constexpr int DCH = D / 8;             // 16-byte chunks per K/V row
  constexpr int LD = KT * DCH / 256;     // chunks of K (and of V) per thread per tile
  __shared__ uint4 ks_[KT * DCH];        // K tile [key][D], chunk ^ (key & 7)
  __shared__ uint4 vt_[D * (KT / 8)];    // V^T tile [d][KT keys], chunk ^ (d & 7)
  __shared__ uint4 ps_[4][16 * (KT / 8)];// per-wave P [16 rows][KT], chunk ^ (row & 7)

  const int item = blockIdx.x, h = blockIdx.y;
  const int wv = a.work[item];
  const int q0 = (wv >> 12) * 64, ksplit = wv & 4095;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bf16* qkv = reinterpret_cast<const bf16*>(a.qkv);
  const bf16* cache = reinterpret_cast<const bf16*>(a.kv_layer);
  const bf16* kbase = cache + (size_t)a.slot * a.st.slot + (size_t)h * a.st.head;
  const bf16* vbase = kbase + a.st.kv;

  // This item's keys: [kbeg, kend) within 0 .. off + min(q0 + 64, C) - 1.
  const int n_keys = a.offset + min(q0 + 64, a.C);
  const int kbeg = ksplit * a.split_keys;
  const int kend = min(n_keys, kbeg + a.split_keys);
  const int n_tiles = (kend - kbeg + KT - 1) / KT;

  // Q fragments (A operand): row = wave*16 + lane%16, d = ks*32 + 8*(lane/16).
  const int qrow = q0 + wave * 16 + (lane & 15);
  uint4 qf[D / 32];
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks)
    qf[ks] = (qrow < a.C) ? *reinterpret_cast<const uint4*>(qkv + (size_t)qrow * a.ld_qkv + h * D + ks * 32 + 8 * (lane >> 4))
                          : make_uint4(0, 0, 0, 0);

  // Rows held by this lane in the C layout: 4*(lane/16) + i of the wave's 16.
  float m_run[4], l_run[4];
  int qpos[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m_run[i] = -INFINITY;
    l_run[i] = 0.f;
    qpos[i] = a.offset + q0 + wave * 16 + 4 * (lane >> 4) + i;
  }
  floatx4 o_acc[D / 16];
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) o_acc[dt] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Tile loads into registers; key addresses are clamped to the last key of
  // the item (finite data; such keys are masked out of the softmax).
  uint4 kreg[LD], vreg[LD];
  auto gload = [&](int kt) {
#pragma unroll
    for (int j = 0; j < LD; ++j) {
      const int c = tid + 256 * j;
      const int kp = min(kbeg + kt * KT + c / DCH, kend - 1);
      const size_t off = (size_t)kp * a.st.pos + (c % DCH) * 8;
      kreg[j] = *reinterpret_cast<const uint4*>(kbase + off);
      vreg[j] = *reinterpret_cast<const uint4*>(vbase + off);
    }
  };
  auto sstore = [&]() {
    bf16* vt = reinterpret_cast<bf16*>(vt_);
#pragma unroll
    for (int j = 0; j < LD; ++j) {
      const int c = tid + 256 * j;
      const int key = c / DCH, ch = c % DCH;
      ks_[key * DCH + (ch ^ (key & 7))] = kreg[j];
      const bf16* vv = reinterpret_cast<const bf16*>(&vreg[j]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = ch * 8 + e;
        vt[(d * (KT / 8) + ((key >> 3) ^ (d & 7))) * 8 + (key & 7)] = vv[e];
      }
    }
  };

  if (n_tiles > 0) gload(0);
  for (int kt = 0; kt < n_tiles; ++kt) {
    const int k0 = kbeg + kt * KT;
    sstore();
    __syncthreads();
    if (kt + 1 < n_tiles) gload(kt + 1);

    // ---- S = Q K^T for the wave's 16 rows x 64 keys.
    floatx4 s[KT / 16];
#pragma unroll
    for (int nt = 0; nt < KT / 16; ++nt) {
      s[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
      const int key = nt * 16 + (lane & 15);
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        const int ch = ks * 4 + (lane >> 4);
        const bf16x8_t kf = __builtin_bit_cast(bf16x8_t, ks_[key * DCH + (ch ^ (key & 7))]);
        s[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, qf[ks]), kf, s[nt], 0, 0, 0);
      }
    }

    // ---- mask (key position <= query position, key in this item), online softmax.
    float p[KT / 16][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mx = -INFINITY;
#pragma unroll
      for (int nt = 0; nt < KT / 16; ++nt) {
        const int kp = k0 + nt * 16 + (lane & 15);
        const float v = (kp <= qpos[i] && kp < kend) ? s[nt][i] * scale_log2 : -INFINITY;
        p[nt][i] = v;
        mx = fmaxf(mx, v);
      }
#pragma unroll
      for (int m = 8; m >= 1; m >>= 1) mx = fmaxf(mx, __shfl_xor(mx, m, 64));
      const float m_new = fmaxf(m_run[i], mx);
      const float m_safe = (m_new == -INFINITY) ? 0.f : m_new;
      const float corr = exp2f(m_run[i] - m_safe);
      float sum = 0.f;
#pragma unroll
      for (int nt = 0; nt < KT / 16; ++nt) {
        const float e = exp2f(p[nt][i] - m_safe);
        p[nt][i] = e;
        sum += e;
      }
#pragma unroll
      for (int m = 8; m >= 1; m >>= 1) sum += __shfl_xor(sum, m, 64);
      l_run[i] = l_run[i] * corr + sum;
      m_run[i] = m_new;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) o_acc[dt][i] *= corr;
    }

    // ---- P (bf16) to the wave's LDS slab, row-major [16][KT].
    bf16* pw = reinterpret_cast<bf16*>(ps_[wave]);
#pragma unroll
    for (int nt = 0; nt < KT / 16; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * (lane >> 4) + i, key = nt * 16 + (lane & 15);
        pw[(r * (KT / 8) + ((key >> 3) ^ (r & 7))) * 8 + (key & 7)] = f2bf(p[nt][i]);
      }
    __syncthreads();

    // ---- O += P V.
#pragma unroll
    for (int kk = 0; kk < KT / 32; ++kk) {
      const int r = lane & 15, ch = kk * 4 + (lane >> 4);
      const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, ps_[wave][r * (KT / 8) + (ch ^ (r & 7))]);
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const int d = dt * 16 + (lane & 15);
        const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, vt_[d * (KT / 8) + (ch ^ (d & 7))]);
        o_acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pf, vf, o_acc[dt], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  // ---- partials of rows < C: [m, l, o[D]].
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int rb = wave * 16 + 4 * (lane >> 4) + i;
    if (q0 + rb >= a.C) continue;
    float* dst = a.part + ((size_t)(item * 64 + rb) * a.nh + h) * (D + 2);
    if ((lane & 15) == 0) {
      dst[0] = m_run[i];
      dst[1] = l_run[i];
    }
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) dst[2 + dt * 16 + (lane & 15)] = o_acc[dt][i];
  }
}

hipError_t launch_attn_prefill(int dtype, const PrefillArgs& a, hipStream_t s) {
  if (a.C <= 0 || a.n_work <= 0) return hipSuccess;
  if (dtype != 1) return hipErrorInvalidValue;
  const float scale_log2 = LOG2E / sqrtf((float)a.hd);
  dim3 grid(a.n_work, a.nh);
  if (a.hd == 128)
    hipLaunchKernelGGL(attn_prefill_bf16_kernel<128>, grid, dim3(256), 0, s, a, scale_log2);
  else
    hipLaunchKernelGGL(attn_prefill_bf16_kernel<64>, grid, dim3(256), 0, s, a, scale_log2);
  return hipGetLastError();
}

// ============================================================================ row attention
template <typename T, int D>
__global__ __launch_bounds__(256) void attn_rows_kernel(RowAttnArgs a, float scale_log2) {
  constexpr int EPL = Vec16<T>::N;           // elements per lane per key (16 bytes)
  constexpr int LPK = D / EPL;               // lanes per key row
  constexpr int KPI = 64 / LPK;              // keys per wave load instruction
  constexpr int NI = LPK;                    // load instructions per pass (64 keys)
  static_assert(LPK * KPI == 64 && NI * KPI == 64, "pass");
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

  for (int pb = kb + wave * 64; pb < ke; pb += 256) {
    uint4 kr[NI], vr[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int key = pb + i * KPI + g;
      const bool ok = key < ke;
      kr[i] = ok ? *reinterpret_cast<const uint4*>(kbase + (size_t)key * a.st.pos) : make_uint4(0, 0, 0, 0);
      vr[i] = ok ? *reinterpret_cast<const uint4*>(vbase + (size_t)key * a.st.pos) : make_uint4(0, 0, 0, 0);
    }
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
    // Reduce-scatter across the LPK lanes of a key group: after it, lane j
    // holds the full score of the key loaded by instruction j.
#pragma unroll
    for (int n = NI, msk = LPK / 2; msk >= 1; n >>= 1, msk >>= 1) {
#pragma unroll
      for (int idx = 0; idx < n / 2; ++idx) {
        const bool upper = (j & msk) != 0;
        const float keep = upper ? part[idx + n / 2] : part[idx];
        const float send = upper ? part[idx] : part[idx + n / 2];
        part[idx] = keep + __shfl_xor(send, msk, 64);
      }
    }
    const int mykey = pb + j * KPI + g;
    const float sc = (mykey < ke) ? part[0] : -INFINITY;
    const float m_new = fmaxf(m_run, wave_max(sc));
    const float m_safe = (m_new == -INFINITY) ? 0.f : m_new;
    const float corr = exp2f(m_run - m_safe);
    const float pk = (mykey < ke) ? exp2f(sc - m_safe) : 0.f;
    l_run = l_run * corr + wave_sum(pk);
    m_run = m_new;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[e] *= corr;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const float w = __shfl(pk, g * LPK + i, 64);
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
  float* dst = a.part + ((size_t)(a.part_base + item) * a.nh + h) * (D + 2);
  for (int d = tid; d < D; d += 256) {
    float acc = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) acc += red_o[w][d] * exp2f(red_m[w] - Ms);
    dst[2 + d] = acc;
  }
  if (tid == 0) {
    float L = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) L += red_l[w] * exp2f(red_m[w] - Ms);
    dst[0] = M;
    dst[1] = L;
  }
}

template <typename T, int D>
static hipError_t run_rows(const RowAttnArgs& a, hipStream_t s) {
  const float scale_log2 = LOG2E / sqrtf((float)D);
  hipLaunchKernelGGL((attn_rows_kernel<T, D>), dim3(a.n_work, a.nh), dim3(256), 0, s, a, scale_log2);
  return hipGetLastError();
}

hipError_t launch_attn_rows(int dtype, const RowAttnArgs& a, hipStream_t s) {
  if (a.n_work <= 0) return hipSuccess;
  if (dtype == 0) return a.hd == 128 ? run_rows<float, 128>(a, s) : run_rows<float, 64>(a, s);
  return a.hd == 128 ? run_rows<bf16, 128>(a, s) : run_rows<bf16, 64>(a, s);
}

// ============================================================================ combine
// O = sum_s o_s 2^(m_s - M) / sum_s l_s 2^(m_s - M), M = max_s m_s.
template <typename T, int D>
__global__ __launch_bounds__(64) void attn_combine_kernel(CombineArgs a) {
  const int r = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int start = a.comb[3 * r], cnt = a.comb[3 * r + 1], stride = a.comb[3 * r + 2];
  float M = -INFINITY;
  for (int j = 0; j < cnt; ++j) M = fmaxf(M, a.part[((size_t)(start + j * stride) * a.nh + h) * (D + 2)]);
  const float Ms = (M == -INFINITY) ? 0.f : M;
  float L = 0.f;
  float acc[D / 64];
#pragma unroll
  for (int e = 0; e < D / 64; ++e) acc[e] = 0.f;
  for (int j = 0; j < cnt; ++j) {
    const float* src = a.part + ((size_t)(start + j * stride) * a.nh + h) * (D + 2);
    const float w = exp2f(src[0] - Ms);
    L += src[1] * w;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) acc[e] += src[2 + lane + 64 * e] * w;
  }
  const float inv = 1.0f / L;
  T* out = reinterpret_cast<T*>(a.out) + (size_t)r * a.ld_out + h * D;
#pragma unroll
  for (int e = 0; e < D / 64; ++e) out[lane + 64 * e] = from_f<T>(acc[e] * inv);
}

hipError_t launch_attn_combine(int dtype, const CombineArgs& a, hipStream_t s) {
  if (a.n_rows <= 0) return hipSuccess;
  dim3 grid(a.n_rows, a.nh);
  if (dtype == 0) {
    if (a.hd == 128) hipLaunchKernelGGL((attn_combine_kernel<float, 128>), grid, dim3(64), 0, s, a);
    else hipLaunchKernelGGL((attn_combine_kernel<float, 64>), grid, dim3(64), 0, s, a);
  } else {
    if (a.hd == 128) hipLaunchKernelGGL((attn_combine_kernel<bf16, 128>), grid, dim3(64), 0, s, a);
    else hipLaunchKernelGGL((attn_combine_kernel<bf16, 64>), grid, dim3(64), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace sarathi
