// The "others" ops of the decoder block (norms, rotary embedding + KV append,
// casts) and the batch-metadata writer.  All memory-bound; one pass each.
#include "kernels.h"

namespace sarathi {

// ------------------------------------------------------------------ metadata
// All loads of a thread are issued before its stores, so the copy costs one
// round trip to the argument buffer rather than one per value.
__global__ __launch_bounds__(256) void meta_write_kernel(MetaChunk c, int* dst) {
  constexpr int PER = (META_CHUNK + 255) / 256;
  int v[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) v[j] = c.values[min((int)threadIdx.x + 256 * j, META_CHUNK - 1)];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int i = threadIdx.x + 256 * j;
    if (i < c.count) dst[i] = v[j];
  }
}

hipError_t launch_meta_write(const MetaChunk& chunk, int* dst, hipStream_t s) {
  hipLaunchKernelGGL(meta_write_kernel, dim3(1), dim3(256), 0, s, chunk, dst);
  return hipGetLastError();
}

// ------------------------------------------------------------------ norms
// Block-wide sum over 256 threads (4 waves).
__device__ __forceinline__ float block_sum_256(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// One row per block, one read of the row: every thread keeps its 16-byte
// chunks (at most NC of them) in registers across the reductions.
// RMS: x / sqrt(mean(x^2) + eps) * g.
// LayerNorm: (x - mean) / sqrt(mean((x - mean)^2) + eps) * g + b.
template <typename T> struct Store16;
template <> struct Store16<bf16> {
  __device__ __forceinline__ static uint4 pack(const float* f) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = (uint32_t)f2bf(f[2 * i]) | ((uint32_t)f2bf(f[2 * i + 1]) << 16);
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
};
template <> struct Store16<float> {
  __device__ __forceinline__ static uint4 pack(const float* f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]), __float_as_uint(f[3]));
  }
};

constexpr int NORM_NC = 12;   // most units per thread

// A unit is CE = max(16 bytes of input, 16 bytes of output) elements, so
// loads and stores are whole 16-byte vectors; H up to NC * 256 * CE, NC the
// units per thread of the instance (registers scale with NC, so the launch
// takes the smallest instance that holds the row).
template <typename Tin, typename Tout, bool LAYER, int NC>
__device__ __forceinline__ void norm_row(const Tin* __restrict__ in, const Tout* __restrict__ g,
                                         const Tout* __restrict__ b, Tout* __restrict__ out, int H, float eps,
                                         size_t row) {
  __shared__ float red[4];
  constexpr int EI = Vec16<Tin>::N, EO = Vec16<Tout>::N;
  constexpr int CE = EI > EO ? EI : EO;
  constexpr int GV = CE / EO;                 // 16-byte gain vectors per unit
  const Tin* x = in + row * (size_t)H;
  const int nunit = H / CE;
  float v[NC][CE];
  // gains (and biases) are loaded up front, beside the row, so that the
  // output pass waits on no load
  uint4 graw[NC][GV], braw[LAYER ? NC : 1][GV];
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const int u = threadIdx.x + 256 * j;
    if (u < nunit) {
#pragma unroll
      for (int o = 0; o < CE; o += EI) Vec16<Tin>::unpack(*reinterpret_cast<const uint4*>(x + u * CE + o), &v[j][o]);
#pragma unroll
      for (int k = 0; k < GV; ++k) {
        graw[j][k] = *reinterpret_cast<const uint4*>(g + u * CE + k * EO);
        if (LAYER) braw[LAYER ? j : 0][k] = *reinterpret_cast<const uint4*>(b + u * CE + k * EO);
      }
#pragma unroll
      for (int e = 0; e < CE; ++e) s += v[j][e];
    } else {
#pragma unroll
      for (int e = 0; e < CE; ++e) v[j][e] = 0.f;
    }
  }
  float mean = 0.f;
  if (LAYER) mean = block_sum_256(s, red) / (float)H;
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    if (threadIdx.x + 256 * j < nunit) {
#pragma unroll
      for (int e = 0; e < CE; ++e) {
        const float d = v[j][e] - mean;
        ss += d * d;
      }
    }
  }
  const float r = 1.0f / sqrtf(block_sum_256(ss, red) / (float)H + eps);
  Tout* y = out + row * (size_t)H;
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const int u = threadIdx.x + 256 * j;
    if (u >= nunit) continue;
    const int i0 = u * CE;
#pragma unroll
    for (int k = 0; k < GV; ++k) {
      const int o = k * EO;
      float gv[EO], bv[EO], f[EO];
      Vec16<Tout>::unpack(graw[j][k], gv);
      if (LAYER) Vec16<Tout>::unpack(braw[LAYER ? j : 0][k], bv);
#pragma unroll
      for (int e = 0; e < EO; ++e) f[e] = (v[j][o + e] - mean) * r * gv[e] + (LAYER ? bv[e] : 0.f);
      *reinterpret_cast<uint4*>(y + i0 + o) = Store16<Tout>::pack(f);
    }
  }
}

template <typename Tin, typename Tout, bool LAYER, int NC>
__global__ __launch_bounds__(256) void norm_kernel(const Tin* __restrict__ in, const Tout* __restrict__ g,
                                                   const Tout* __restrict__ b, Tout* __restrict__ out, int H,
                                                   float eps) {
  norm_row<Tin, Tout, LAYER, NC>(in, g, b, out, H, eps, blockIdx.x);
}

// The first norm of a layer call with the metadata upload riding along:
// block 0 copies the metadata chunk (as meta_write_kernel), blocks 1..rows
// normalise rows 0..rows-1.  One launch instead of two.
template <typename Tin, typename Tout, bool LAYER, int NC>
__global__ __launch_bounds__(256) void norm_meta_kernel(const Tin* __restrict__ in, const Tout* __restrict__ g,
                                                        const Tout* __restrict__ b, Tout* __restrict__ out, int H,
                                                        float eps, MetaChunk c, int* __restrict__ dst) {
  if (blockIdx.x == 0) {
    constexpr int PER = (META_CHUNK + 255) / 256;
    int v[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) v[j] = c.values[min((int)threadIdx.x + 256 * j, META_CHUNK - 1)];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int i = threadIdx.x + 256 * j;
      if (i < c.count) dst[i] = v[j];
    }
    return;
  }
  norm_row<Tin, Tout, LAYER, NC>(in, g, b, out, H, eps, blockIdx.x - 1);
}

template <typename Tin, typename Tout, bool LAYER, int NC>
static void norm_launch_nc(const void* in, const void* g, const void* b, void* out, int rows, int H, float eps,
                           hipStream_t s, const MetaChunk* meta, int* meta_dst) {
  if (meta)
    hipLaunchKernelGGL((norm_meta_kernel<Tin, Tout, LAYER, NC>), dim3(rows + 1), dim3(256), 0, s, (const Tin*)in,
                       (const Tout*)g, (const Tout*)b, (Tout*)out, H, eps, *meta, meta_dst);
  else
    hipLaunchKernelGGL((norm_kernel<Tin, Tout, LAYER, NC>), dim3(rows), dim3(256), 0, s, (const Tin*)in,
                       (const Tout*)g, (const Tout*)b, (Tout*)out, H, eps);
}

template <typename Tin, typename Tout, bool LAYER>
static void norm_launch(const void* in, const void* g, const void* b, void* out, int rows, int H, float eps,
                        hipStream_t s, const MetaChunk* meta, int* meta_dst) {
  constexpr int EI = Vec16<Tin>::N, EO = Vec16<Tout>::N;
  constexpr int CE = EI > EO ? EI : EO;
  const int nc = (H / CE + 255) / 256;
  if (nc <= 2) norm_launch_nc<Tin, Tout, LAYER, 2>(in, g, b, out, rows, H, eps, s, meta, meta_dst);
  else if (nc <= 4) norm_launch_nc<Tin, Tout, LAYER, 4>(in, g, b, out, rows, H, eps, s, meta, meta_dst);
  else if (nc <= 6) norm_launch_nc<Tin, Tout, LAYER, 6>(in, g, b, out, rows, H, eps, s, meta, meta_dst);
  else norm_launch_nc<Tin, Tout, LAYER, NORM_NC>(in, g, b, out, rows, H, eps, s, meta, meta_dst);
}

template <typename Tin, typename Tout>
static void norm_dispatch(bool layer, const void* in, const void* g, const void* b, void* out, int rows, int H,
                          float eps, hipStream_t s, const MetaChunk* meta, int* meta_dst) {
  if (layer)
    norm_launch<Tin, Tout, true>(in, g, b, out, rows, H, eps, s, meta, meta_dst);
  else
    norm_launch<Tin, Tout, false>(in, g, b, out, rows, H, eps, s, meta, meta_dst);
}

hipError_t launch_norm(int dtype, bool in_f32, bool layer_norm, const void* in, const void* g,
                       const void* b, void* out, int rows, int H, float eps, hipStream_t s,
                       const MetaChunk* meta, int* meta_dst) {
  if (rows <= 0) return meta ? launch_meta_write(*meta, meta_dst, s) : hipSuccess;
  if (dtype == 0)
    norm_dispatch<float, float>(layer_norm, in, g, b, out, rows, H, eps, s, meta, meta_dst);
  else if (in_f32)
    norm_dispatch<float, bf16>(layer_norm, in, g, b, out, rows, H, eps, s, meta, meta_dst);
  else
    norm_dispatch<bf16, bf16>(layer_norm, in, g, b, out, rows, H, eps, s, meta, meta_dst);
  return hipGetLastError();
}

// ------------------------------------------------------------------ RoPE + KV append
// One thread per (row, head, group of P consecutive pair indices), P = 16
// bytes of T: it rotates the pairs (i, i + hd/2), i in [i0, i0 + P), of q and
// k by angle pos * base^(-2i/hd) (angle reduced in fp64, sin/cos in fp32),
// writes q back in place and k, v to the cache at (slot, pos), all with
// 16-byte accesses.
template <typename T>
__global__ __launch_bounds__(256) void rope_append_kernel(RopeArgs a) {
  constexpr int P = Vec16<T>::N;
  const int half = a.hd / 2, groups = half / P;
  const size_t t = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  if (t >= (size_t)a.T * a.nh * groups) return;
  const int grp = (int)(t % groups);
  const int h = (int)((t / groups) % a.nh);
  const int row = (int)(t / ((size_t)groups * a.nh));
  const int i0 = grp * P;
  const int slot = a.row_slot[row];
  const int pos = a.row_pos[row];
  T* base = reinterpret_cast<T*>(a.qkv) + (size_t)row * (3 * a.nh * a.hd);
  T* q = base + h * a.hd;
  const T* k = base + a.nh * a.hd + h * a.hd;
  const T* v = base + 2 * a.nh * a.hd + h * a.hd;
  T* cache = reinterpret_cast<T*>(a.kv_layer);
  T* kd = cache + (size_t)slot * a.st.slot + (size_t)h * a.st.head + (size_t)pos * a.st.pos;
  T* vd = kd + a.st.kv;
  const uint4 k_lo = *reinterpret_cast<const uint4*>(k + i0), k_hi = *reinterpret_cast<const uint4*>(k + half + i0);
  *reinterpret_cast<uint4*>(vd + i0) = *reinterpret_cast<const uint4*>(v + i0);
  *reinterpret_cast<uint4*>(vd + half + i0) = *reinterpret_cast<const uint4*>(v + half + i0);
  if (!a.rope) {
    *reinterpret_cast<uint4*>(kd + i0) = k_lo;
    *reinterpret_cast<uint4*>(kd + half + i0) = k_hi;
    return;
  }
  float q0[P], q1[P], k0[P], k1[P];
  Vec16<T>::unpack(*reinterpret_cast<const uint4*>(q + i0), q0);
  Vec16<T>::unpack(*reinterpret_cast<const uint4*>(q + half + i0), q1);
  Vec16<T>::unpack(k_lo, k0);
  Vec16<T>::unpack(k_hi, k1);
  const double lb = log2((double)a.base);
#pragma unroll
  for (int e = 0; e < P; ++e) {
    float sn, c;
    rope_sincos(pos, rope_theta(i0 + e, a.hd, lb), &sn, &c);
    const float nq0 = q0[e] * c - q1[e] * sn, nq1 = q0[e] * sn + q1[e] * c;
    const float nk0 = k0[e] * c - k1[e] * sn, nk1 = k0[e] * sn + k1[e] * c;
    q0[e] = nq0; q1[e] = nq1; k0[e] = nk0; k1[e] = nk1;
  }
  *reinterpret_cast<uint4*>(q + i0) = Store16<T>::pack(q0);
  *reinterpret_cast<uint4*>(q + half + i0) = Store16<T>::pack(q1);
  *reinterpret_cast<uint4*>(kd + i0) = Store16<T>::pack(k0);
  *reinterpret_cast<uint4*>(kd + half + i0) = Store16<T>::pack(k1);
}

hipError_t launch_rope_append(int dtype, const RopeArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  const int P = dtype == 0 ? 4 : 8;   // pairs per thread (16 bytes)
  const size_t threads = (size_t)a.T * a.nh * (a.hd / 2 / P);
  const dim3 grid((unsigned)((threads + 255) / 256));
  if (dtype == 0)
    hipLaunchKernelGGL(rope_append_kernel<float>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(rope_append_kernel<bf16>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

// ------------------------------------------------------------------ split-K reduction
// out = resid + parts[0] + parts[1] + ... (fixed order: deterministic).  Four
// elements per thread when n is a multiple of 4, else one.
template <typename Tr, typename To, int V>
__global__ __launch_bounds__(256) void split_reduce_kernel(const Tr* __restrict__ resid, const float* __restrict__ parts,
                                                           int n_split, size_t n, To* __restrict__ out) {
  const size_t nv = n / V;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < nv; i += (size_t)gridDim.x * blockDim.x) {
    // every split's partial is loaded before the first add (one memory
    // round trip, not n_split), then added in split order
    float q[MAX_SPLIT][V];
#pragma unroll
    for (int sp = 0; sp < MAX_SPLIT; ++sp) {
      if (sp >= n_split) break;
      const float* pp = parts + (size_t)sp * n + i * V;
      if constexpr (V == 4) {
        const float4 f = *reinterpret_cast<const float4*>(pp);
        q[sp][0] = f.x; q[sp][1] = f.y; q[sp][2] = f.z; q[sp][3] = f.w;
      } else {
#pragma unroll
        for (int e = 0; e < V; ++e) q[sp][e] = pp[e];
      }
    }
    float acc[V];
#pragma unroll
    for (int e = 0; e < V; ++e) acc[e] = to_f<Tr>(resid[i * V + e]);
#pragma unroll
    for (int sp = 0; sp < MAX_SPLIT; ++sp) {
      if (sp >= n_split) break;
#pragma unroll
      for (int e = 0; e < V; ++e) acc[e] += q[sp][e];
    }
#pragma unroll
    for (int e = 0; e < V; ++e) out[i * V + e] = from_f<To>(acc[e]);
  }
}

template <typename Tr, typename To>
static void split_reduce_dispatch(const void* resid, const float* parts, int n_split, size_t n, void* out,
                                  hipStream_t s) {
  const bool vec = (n % 4) == 0;
  const size_t items = vec ? n / 4 : n;
  const int blocks = (int)((items + 255) / 256 < 8192 ? (items + 255) / 256 : 8192);
  if (vec)
    hipLaunchKernelGGL((split_reduce_kernel<Tr, To, 4>), dim3(blocks), dim3(256), 0, s, (const Tr*)resid, parts,
                       n_split, n, (To*)out);
  else
    hipLaunchKernelGGL((split_reduce_kernel<Tr, To, 1>), dim3(blocks), dim3(256), 0, s, (const Tr*)resid, parts,
                       n_split, n, (To*)out);
}

// Split-K reduction of rows of N followed by the norm of each row, one block
// per row: the row's sums stay in registers between the reduction and the
// norm, so the norm reads nothing back.  RF32 = false: bf16 residual, fp32
// out (a layer's postproj, then its norm_2); RF32 = true: fp32 residual, bf16
// out (a layer's ffn_ln2, then the next layer's norm_1, which normalises the
// bf16-rounded row).  The sums are formed in split order as in
// split_reduce_kernel, and the norm accumulates over the same units in the
// same order as norm_row, so both outputs are bit-identical to the two
// separate passes.
template <bool LAYER, int NC, bool RF32>
__global__ __launch_bounds__(256) void split_reduce_norm_kernel(const void* __restrict__ resid_,
                                                                const float* __restrict__ parts, int n_split, int N,
                                                                void* __restrict__ out_, const bf16* __restrict__ g,
                                                                const bf16* __restrict__ b, bf16* __restrict__ nout,
                                                                float eps) {
  __shared__ float red[4];
  constexpr int CE = 8;                       // elements per unit: 16 bytes of bf16, 2 x 16 of fp32
  const size_t row = blockIdx.x;
  const size_t n = (size_t)gridDim.x * N;     // elements per split
  const int nunit = N / CE;
  float v[NC][CE];
  uint4 graw[NC], braw[LAYER ? NC : 1];
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const int u = threadIdx.x + 256 * j;
    if (u < nunit) {
      const size_t at = row * N + (size_t)u * CE;
      float q[MAX_SPLIT][CE];
#pragma unroll
      for (int sp = 0; sp < MAX_SPLIT; ++sp) {
        if (sp >= n_split) break;
        const float4* pp = reinterpret_cast<const float4*>(parts + (size_t)sp * n + at);
        const float4 lo = pp[0], hi = pp[1];
        q[sp][0] = lo.x; q[sp][1] = lo.y; q[sp][2] = lo.z; q[sp][3] = lo.w;
        q[sp][4] = hi.x; q[sp][5] = hi.y; q[sp][6] = hi.z; q[sp][7] = hi.w;
      }
      graw[j] = *reinterpret_cast<const uint4*>(g + (size_t)u * CE);
      if (LAYER) braw[LAYER ? j : 0] = *reinterpret_cast<const uint4*>(b + (size_t)u * CE);
      if constexpr (RF32) {
        const float4* rp = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(resid_) + at);
        const float4 lo = rp[0], hi = rp[1];
        v[j][0] = lo.x; v[j][1] = lo.y; v[j][2] = lo.z; v[j][3] = lo.w;
        v[j][4] = hi.x; v[j][5] = hi.y; v[j][6] = hi.z; v[j][7] = hi.w;
      } else {
        Vec16<bf16>::unpack(*reinterpret_cast<const uint4*>(reinterpret_cast<const bf16*>(resid_) + at), v[j]);
      }
#pragma unroll
      for (int sp = 0; sp < MAX_SPLIT; ++sp) {
        if (sp >= n_split) break;
#pragma unroll
        for (int e = 0; e < CE; ++e) v[j][e] += q[sp][e];
      }
      if constexpr (RF32) {
        const uint4 w = Store16<bf16>::pack(v[j]);
        *reinterpret_cast<uint4*>(reinterpret_cast<bf16*>(out_) + at) = w;
        Vec16<bf16>::unpack(w, v[j]);      // the norm sees the stored (rounded) row
      } else {
        float4* op = reinterpret_cast<float4*>(reinterpret_cast<float*>(out_) + at);
        op[0] = make_float4(v[j][0], v[j][1], v[j][2], v[j][3]);
        op[1] = make_float4(v[j][4], v[j][5], v[j][6], v[j][7]);
      }
#pragma unroll
      for (int e = 0; e < CE; ++e) s += v[j][e];
    } else {
#pragma unroll
      for (int e = 0; e < CE; ++e) v[j][e] = 0.f;
    }
  }
  float mean = 0.f;
  if (LAYER) mean = block_sum_256(s, red) / (float)N;
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    if (threadIdx.x + 256 * j < nunit) {
#pragma unroll
      for (int e = 0; e < CE; ++e) {
        const float d = v[j][e] - mean;
        ss += d * d;
      }
    }
  }
  const float r = 1.0f / sqrtf(block_sum_256(ss, red) / (float)N + eps);
  bf16* y = nout + row * (size_t)N;
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const int u = threadIdx.x + 256 * j;
    if (u >= nunit) continue;
    float gv[CE], bv[CE], f[CE];
    Vec16<bf16>::unpack(graw[j], gv);
    if (LAYER) Vec16<bf16>::unpack(braw[LAYER ? j : 0], bv);
#pragma unroll
    for (int e = 0; e < CE; ++e) f[e] = (v[j][e] - mean) * r * gv[e] + (LAYER ? bv[e] : 0.f);
    *reinterpret_cast<uint4*>(y + (size_t)u * CE) = Store16<bf16>::pack(f);
  }
}

template <bool LAYER, bool RF32>
static hipError_t split_reduce_norm_layer(const void* resid, const float* parts, int n_split, int rows, int N,
                                          void* out, const NormArgs& nm, hipStream_t s) {
  const int nc = (N / 8 + 255) / 256;
#define SRN_LAUNCH(NCV)                                                                                          \
  hipLaunchKernelGGL((split_reduce_norm_kernel<LAYER, NCV, RF32>), dim3(rows), dim3(256), 0, s, resid, parts, n_split, \
                     N, out, (const bf16*)nm.g, (const bf16*)nm.b, (bf16*)nm.out, nm.eps)
  if (nc <= 4) SRN_LAUNCH(4);
  else if (nc <= 8) SRN_LAUNCH(8);
  else SRN_LAUNCH(12);
#undef SRN_LAUNCH
  return hipGetLastError();
}

hipError_t launch_split_reduce_norm(const void* resid, bool resid_f32, const float* parts, int n_split, int rows,
                                    int N, void* out, const NormArgs& norm, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (N % 8 != 0 || N / 8 > 12 * 256 || n_split < 1 || n_split > MAX_SPLIT) return hipErrorNotSupported;
  if (resid_f32)
    return norm.layer ? split_reduce_norm_layer<true, true>(resid, parts, n_split, rows, N, out, norm, s)
                      : split_reduce_norm_layer<false, true>(resid, parts, n_split, rows, N, out, norm, s);
  return norm.layer ? split_reduce_norm_layer<true, false>(resid, parts, n_split, rows, N, out, norm, s)
                    : split_reduce_norm_layer<false, false>(resid, parts, n_split, rows, N, out, norm, s);
}

hipError_t launch_split_reduce(int dtype, bool resid_f32, bool out_f32, const void* resid, const float* parts,
                               int n_split, size_t n, void* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (n_split < 1 || n_split > MAX_SPLIT) return hipErrorInvalidValue;
  if (dtype == 0 || (resid_f32 && out_f32))
    split_reduce_dispatch<float, float>(resid, parts, n_split, n, out, s);
  else if (resid_f32)
    split_reduce_dispatch<float, bf16>(resid, parts, n_split, n, out, s);
  else if (out_f32)
    split_reduce_dispatch<bf16, float>(resid, parts, n_split, n, out, s);
  else
    split_reduce_dispatch<bf16, bf16>(resid, parts, n_split, n, out, s);
  return hipGetLastError();
}

}  // namespace sarathi
