// The combine pass of the attention: merges the per-split partial results
// (max, sum, unnormalised o) of every row -- chunk rows and decodes -- into
// the attention output.
#include "kernels.h"

namespace sarathi {

// ============================================================================ combine
// O = sum_s o_s 2^(m_s - M) / sum_s l_s 2^(m_s - M), M = max_s m_s.  One wave
// per (row, head), four heads per block.  The lanes read the splits' (m, l)
// in parallel while every lane already loads its D/64 columns of the first
// U splits; later splits follow in groups of U, each group's loads issued
// together, so a row of up to U splits costs one round trip to memory.  The
// splits are added in split order (deterministic).
template <typename T, int D>
__global__ __launch_bounds__(256) void attn_combine_kernel(CombineArgs a) {
  constexpr int E = D / 64, U = 8;
  const int r = a.row0 + blockIdx.x, lane = threadIdx.x & 63;
  const int h = blockIdx.y * 4 + (threadIdx.x >> 6);
  if (h >= a.nh) return;
  const int start = a.comb[3 * r], cnt = a.comb[3 * r + 1], stride = a.comb[3 * r + 2];
  if (cnt == 0) return;   // written directly by its attention kernel
  auto src_of = [&](int j) { return a.part + ((size_t)(start + j * stride) * a.nh + h) * (D + PART_O); };
  float v[U][E];
  auto load_group = [&](int j0) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < E; ++e) v[u][e] = (j0 + u < cnt) ? src_of(j0 + u)[PART_O + lane + 64 * e] : 0.f;
  };
  // first chunk of up to 64 splits: (m, l) per lane, o of the first U splits
  const int n0 = min(64, cnt);
  const float* mine = src_of(min(lane, n0 - 1));
  float m_l = lane < n0 ? mine[0] : -INFINITY;
  float l_l = lane < n0 ? mine[1] : 0.f;
  load_group(0);
  float M = m_l;
  for (int j0 = 64; j0 < cnt; j0 += 64)
    if (j0 + lane < cnt) M = fmaxf(M, src_of(j0 + lane)[0]);
  M = wave_max(M);
  const float Ms = (M == -INFINITY) ? 0.f : M;
  float wl = lane < n0 ? exp2f(m_l - Ms) : 0.f;
  float L = wl * l_l;
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  for (int j0 = 0; j0 < cnt; j0 += U) {
    if (j0 > 0) {
      if (j0 % 64 == 0) {   // next chunk of 64 splits: its (m, l) per lane
        const int nj = min(64, cnt - j0);
        const float* mj = src_of(j0 + min(lane, nj - 1));
        wl = lane < nj ? exp2f(mj[0] - Ms) : 0.f;
        L += wl * (lane < nj ? mj[1] : 0.f);
      }
      load_group(j0);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (j0 + u < cnt) {
        const float w = __shfl(wl, (j0 + u) % 64, 64);
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = fmaf(v[u][e], w, acc[e]);
      }
    }
  }
  L = wave_sum(L);
  const float inv = 1.0f / L;
  T* out = reinterpret_cast<T*>(a.out) + (size_t)r * a.ld_out + h * D;
#pragma unroll
  for (int e = 0; e < E; ++e) out[lane + 64 * e] = from_f<T>(acc[e] * inv);
}

hipError_t launch_attn_combine(int dtype, const CombineArgs& a, hipStream_t s) {
  if (a.n_rows <= a.row0) return hipSuccess;
  dim3 grid(a.n_rows - a.row0, (a.nh + 3) / 4);
  if (dtype == 0) {
    if (a.hd == 128) hipLaunchKernelGGL((attn_combine_kernel<float, 128>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((attn_combine_kernel<float, 64>), grid, dim3(256), 0, s, a);
  } else {
    if (a.hd == 128) hipLaunchKernelGGL((attn_combine_kernel<bf16, 128>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((attn_combine_kernel<bf16, 64>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace sarathi
