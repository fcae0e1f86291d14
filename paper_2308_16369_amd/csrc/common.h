// Shared device helpers for the gfx950 kernels of libsarathi.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <cmath>

namespace sarathi {

typedef uint16_t bf16;   // bf16 storage (bit pattern)
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));   // 16 bytes kept in registers

__device__ __forceinline__ float bf2f(bf16 b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ bf16 f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16)0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16)(u >> 16);
}

template <typename T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<bf16>(bf16 v) { return bf2f(v); }

template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float v) { return f2bf(v); }

// 16-byte vector <-> float lanes.
template <typename T> struct Vec16;
template <> struct Vec16<bf16> {
  static constexpr int N = 8;
  __device__ __forceinline__ static void unpack(const uint4& v, float* f) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
};
template <> struct Vec16<float> {
  static constexpr int N = 4;
  __device__ __forceinline__ static void unpack(const uint4& v, float* f) {
    f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
  }
};

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + __expf(-z)); }
__device__ __forceinline__ float gelu_f(float z) { return 0.5f * z * (1.0f + erff(z * 0.70710678118654752f)); }

// Wave-level (64 lanes) reductions.
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// Rotary embedding: frequency of pair index i (of head_dim hd),
// base^(-2i/hd) with lb = log2(base), in fp64; the angle pos * theta is
// reduced to [-pi, pi] in fp64, then sin / cos in fp32.
__device__ __forceinline__ double rope_theta(int i, int hd, double lb) {
  return exp2(-2.0 * (double)i / (double)hd * lb);
}
__device__ __forceinline__ void rope_sincos(int pos, double theta, float* sn, float* cs) {
  const double ang = (double)pos * theta;
  const double red = ang - 6.283185307179586 * rint(ang * 0.15915494309189535);
  __sincosf((float)red, sn, cs);
}

// KV cache element strides: [layer][slot][K|V][head][pos][head_dim].
struct KVStrides {
  size_t layer, slot, kv, head, pos;
};

// Raises a kernel's dynamic-LDS limit to `bytes` once per device (the
// attribute belongs to the current device; `done` records the devices already
// set, so concurrent callers may both set it, harmlessly).
inline hipError_t ensure_dynamic_lds(const void* kernel, int bytes, std::atomic<uint64_t>& done) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = (dev >= 0 && dev < 64) ? (1ull << dev) : 0;
  if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
  e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_acq_rel);
  return e;
}

// LDS DMA and its waits.
typedef __attribute__((address_space(3))) void lds_void_t;

// One wave instruction: lane i copies 16 bytes from src (its own address) to
// dst + 16 i (dst is the same for the whole wave), global_load_lds_dwordx4.
__device__ __forceinline__ void dma16(const void* src, uint4* dst) {
  __builtin_amdgcn_global_load_lds(src, (lds_void_t*)dst, 16, 0, 0);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // gfx9 s_waitcnt: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] at [15:14]
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier without the fence of __syncthreads(): the fence would
// make the compiler wait for every outstanding LDS DMA load (vmcnt 0) and
// drain the ring.  The memory clobber keeps LDS accesses on their side.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }
// The same after this wave's LDS reads have returned, so a stage it has read
// can be refilled by DMA once every wave has passed the barrier.
__device__ __forceinline__ void lds_read_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

}  // namespace sarathi
