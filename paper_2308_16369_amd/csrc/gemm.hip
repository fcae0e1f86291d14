// Linear ops of the hybrid batch: one matmul over all C+B rows (Sec. 4.3,
// "fuse all the linear operations"), y = x W^T with W stored [N, K].
//
// bf16: MFMA v_mfma_f32_16x16x32_bf16, 256 threads = 2x2 waves, block tile
// BM x BN x 64, both operands staged through LDS (double-buffered, 16-byte
// chunks XOR-swizzled by row so the MFMA operand reads are bank-conflict
// free).  Both operands are K-contiguous, so every lane reads 16 contiguous
// bytes for either MFMA operand.  Epilogues fuse the residual add
// (postproj, ffn_ln2), SiLU*mul (SwiGLU ffn_ln1) and GELU.  Split-K
// accumulates fp32 partials atomically into a buffer that already holds the
// residual.
//
// fp32: a plain LDS-tiled FMA kernel with the same epilogues.
#include "kernels.h"

namespace sarathi {

enum Epi { EPI_STORE = 0, EPI_GELU = 1, EPI_SWIGLU = 2, EPI_RESID_TO_F32 = 3, EPI_RESIDF32_TO_ACT = 4,
           EPI_ATOMIC = 5 };

struct GemmP {
  const void* A;        // [M, K]
  const void* W;        // [N or 2N, K]
  int M, N, K;          // N = output columns (SwiGLU: F)
  int k_split, n_split; // K elements per split; number of splits
  int tiles_m, tiles_n, n_tiles;
  void* out;            // [M, N]: dtype, or fp32 for EPI_RESID_TO_F32 / EPI_ATOMIC
  const void* resid;    // EPI_RESID_TO_F32: dtype [M,N]; EPI_RESIDF32_TO_ACT: fp32 [M,N]
};

// Output element handling shared by both kernels.
template <typename T, int EPI>
__device__ __forceinline__ void epi_store(const GemmP& p, int r, int c, float v) {
  const size_t idx = (size_t)r * p.N + c;
  if (EPI == EPI_STORE) {
    reinterpret_cast<T*>(p.out)[idx] = from_f<T>(v);
  } else if (EPI == EPI_GELU) {
    reinterpret_cast<T*>(p.out)[idx] = from_f<T>(gelu_f(v));
  } else if (EPI == EPI_RESID_TO_F32) {
    reinterpret_cast<float*>(p.out)[idx] = to_f<T>(reinterpret_cast<const T*>(p.resid)[idx]) + v;
  } else if (EPI == EPI_RESIDF32_TO_ACT) {
    reinterpret_cast<T*>(p.out)[idx] = from_f<T>(reinterpret_cast<const float*>(p.resid)[idx] + v);
  } else if (EPI == EPI_ATOMIC) {
    unsafeAtomicAdd(reinterpret_cast<float*>(p.out) + idx, v);
  }
}

// ============================================================================ bf16 MFMA
template <int BM, int BN, int EPI>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmP p) {
  constexpr int BK = 64;
  constexpr int WTM = BM / 2, WTN = BN / 2;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int AL = BM / 32, BL = BN / 32;
  static_assert(BM % 32 == 0 && BN % 64 == 0, "tile");
  extern __shared__ uint4 lds[];   // [2][(BM + BN) * 8] 16-byte chunks

  // XCD-aware order: block b runs on XCD b % 8.  Consecutive tiles (the
  // M-tiles that share a W panel) are given to blocks of one XCD so the panel
  // is fetched into that XCD's L2 once.
  const int per = gridDim.x / 8;
  const int t = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (t >= p.n_tiles) return;
  const int tile_m = t % p.tiles_m;
  const int rest = t / p.tiles_m;
  const int split = rest % p.n_split;
  const int tile_n = rest / p.n_split;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = tile_m * BM;
  const int n0_out = tile_n * (EPI == EPI_SWIGLU ? BN / 2 : BN);
  const int kbeg = split * p.k_split;
  const int kend = min(p.K, kbeg + p.k_split);
  const int nk = (kend - kbeg + BK - 1) / BK;

  const bf16* A = reinterpret_cast<const bf16*>(p.A);
  const bf16* W = reinterpret_cast<const bf16*>(p.W);
  const int lc = tid & 7, lr = tid >> 3;

  const bf16* a_src[AL];
  bool a_ok[AL];
#pragma unroll
  for (int i = 0; i < AL; ++i) {
    const int r = m0 + lr + 32 * i;
    a_ok[i] = r < p.M;
    a_src[i] = A + (size_t)(a_ok[i] ? r : 0) * p.K + kbeg + lc * 8;
  }
  const bf16* b_src[BL];
  bool b_ok[BL];
#pragma unroll
  for (int i = 0; i < BL; ++i) {
    const int nl = lr + 32 * i;
    int wrow;
    if (EPI == EPI_SWIGLU) {
      const int q = nl / WTN, w = nl % WTN, half = WTN / 2;
      const int j = n0_out + q * half + (w % half);
      b_ok[i] = j < p.N;
      wrow = (w < half) ? j : p.N + j;
    } else {
      wrow = n0_out + nl;
      b_ok[i] = wrow < p.N;
    }
    b_src[i] = W + (size_t)(b_ok[i] ? wrow : 0) * p.K + kbeg + lc * 8;
  }

  uint4 ra[AL], rb[BL];
  auto gload = [&](int kt) {
    const bool kok = kbeg + kt * BK + lc * 8 < kend;
#pragma unroll
    for (int i = 0; i < AL; ++i)
      ra[i] = (a_ok[i] && kok) ? *reinterpret_cast<const uint4*>(a_src[i] + kt * BK) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < BL; ++i)
      rb[i] = (b_ok[i] && kok) ? *reinterpret_cast<const uint4*>(b_src[i] + kt * BK) : make_uint4(0, 0, 0, 0);
  };
  auto sstore = [&](int buf) {
    uint4* s = lds + buf * (BM + BN) * 8;
#pragma unroll
    for (int i = 0; i < AL; ++i) {
      const int r = lr + 32 * i;
      s[r * 8 + (lc ^ (r & 7))] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BL; ++i) {
      const int r = BM + lr + 32 * i;
      s[r * 8 + (lc ^ (r & 7))] = rb[i];
    }
  };

  floatx4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  if (nk > 0) {
    gload(0);
    sstore(0);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    const uint4* s = lds + cur * (BM + BN) * 8;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int ch = ks * 4 + (lane >> 4);
      bf16x8_t af[FM], bfr[FN];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
        const int r = wm * WTM + fm * 16 + (lane & 15);
        af[fm] = __builtin_bit_cast(bf16x8_t, s[r * 8 + (ch ^ (r & 7))]);
      }
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        const int r = BM + wn * WTN + fn * 16 + (lane & 15);
        bfr[fn] = __builtin_bit_cast(bf16x8_t, s[r * 8 + (ch ^ (r & 7))]);
      }
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
          acc[fm][fn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[fm], bfr[fn], acc[fm][fn], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  // Epilogue.  acc[fm][fn][i] = C[row 4*(lane/16)+i][col lane%16] of the 16x16 tile.
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = m0 + wm * WTM + fm * 16 + 4 * (lane >> 4) + i;
      if (r >= p.M) continue;
      if (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int fn = 0; fn < FN / 2; ++fn) {
          const int c = n0_out + wn * (WTN / 2) + fn * 16 + (lane & 15);
          if (c < p.N) {
            const float v = silu_f(acc[fm][fn][i]) * acc[fm][fn + FN / 2][i];
            reinterpret_cast<bf16*>(p.out)[(size_t)r * p.N + c] = f2bf(v);
          }
        }
      } else {
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          const int c = n0_out + wn * WTN + fn * 16 + (lane & 15);
          if (c < p.N) epi_store<bf16, EPI>(p, r, c, acc[fm][fn][i]);
        }
      }
    }
  }
}

// ============================================================================ fp32 FMA
// 64x64 tile of W rows (SwiGLU: 32 gate + 32 up rows -> 32 outputs), BK 16,
// 16x16 threads with 4x4 results each.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmP p) {
  constexpr int BK = 16;
  __shared__ float As[BK][64 + 4];
  __shared__ float Ws[BK][64 + 4];
  const int tile_m = blockIdx.x, tile_n = blockIdx.y;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = tile_m * 64;
  const int n0_out = tile_n * (EPI == EPI_SWIGLU ? 32 : 64);
  const float* A = reinterpret_cast<const float*>(p.A);
  const float* W = reinterpret_cast<const float*>(p.W);
  int cols[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) cols[j] = (EPI == EPI_SWIGLU) ? ((j < 2) ? 2 * tx + j : 32 + 2 * tx + j - 2) : 4 * tx + j;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < p.K; k0 += BK) {
    for (int e = threadIdx.x; e < 64 * BK; e += 256) {
      const int r = e / BK, kk = e % BK;
      const int gr = m0 + r, gk = k0 + kk;
      As[kk][r] = (gr < p.M && gk < p.K) ? A[(size_t)gr * p.K + gk] : 0.f;
      int wrow;
      bool ok;
      if (EPI == EPI_SWIGLU) {
        const int j = n0_out + (r % 32);
        ok = j < p.N;
        wrow = (r < 32) ? j : p.N + j;
      } else {
        wrow = n0_out + r;
        ok = wrow < p.N;
      }
      Ws[kk][r] = (ok && gk < p.K) ? W[(size_t)wrow * p.K + gk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][4 * ty + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Ws[kk][cols[j]];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = m0 + 4 * ty + i;
    if (r >= p.M) continue;
    if (EPI == EPI_SWIGLU) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int c = n0_out + 2 * tx + j;
        if (c < p.N)
          reinterpret_cast<float*>(p.out)[(size_t)r * p.N + c] = silu_f(acc[i][j]) * acc[i][j + 2];
      }
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int c = n0_out + 4 * tx + j;
        if (c < p.N) epi_store<float, EPI>(p, r, c, acc[i][j]);
      }
    }
  }
}

// ============================================================================ launch
template <int BM, int BN, int EPI>
static hipError_t run_bf16(GemmP p, hipStream_t s) {
  const size_t lds_bytes = 2 * (BM + BN) * 8 * sizeof(uint4);
  static bool attr_set = false;   // per process; the attribute is per function
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)gemm_bf16_kernel<BM, BN, EPI>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int grid = (p.n_tiles + 7) / 8 * 8;
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, EPI>), dim3(grid), dim3(256), lds_bytes, s, p);
  return hipGetLastError();
}

template <int BM>
static hipError_t run_bf16_epi(int epi, const GemmP& p, hipStream_t s) {
  switch (epi) {
    case EPI_STORE: return run_bf16<BM, 128, EPI_STORE>(p, s);
    case EPI_GELU: return run_bf16<BM, 128, EPI_GELU>(p, s);
    case EPI_SWIGLU: return run_bf16<BM, 128, EPI_SWIGLU>(p, s);
    case EPI_RESID_TO_F32: return run_bf16<BM, 128, EPI_RESID_TO_F32>(p, s);
    case EPI_RESIDF32_TO_ACT: return run_bf16<BM, 128, EPI_RESIDF32_TO_ACT>(p, s);
    default: return run_bf16<BM, 128, EPI_ATOMIC>(p, s);
  }
}

template <int EPI>
static hipError_t run_f32(const GemmP& p, hipStream_t s) {
  const int out_per_tile = (EPI == EPI_SWIGLU) ? 32 : 64;
  dim3 grid((p.M + 63) / 64, (p.N + out_per_tile - 1) / out_per_tile);
  hipLaunchKernelGGL(gemm_f32_kernel<EPI>, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

// Block rows for the bf16 kernel: the candidate that pads M least, larger on ties.
static int pick_bm(int M) {
  if (M <= 64) return 64;
  const int cands[3] = {160, 128, 96};
  int best = 160, best_pad = 1 << 30;
  for (int c : cands) {
    const int pad = (M + c - 1) / c * c;
    if (pad < best_pad) { best_pad = pad; best = c; }
  }
  return best;
}

hipError_t launch_linear(int dtype, const LinearArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  GemmP p{};
  p.A = a.x; p.W = a.w; p.M = a.M; p.N = a.N; p.K = a.K;
  p.out = a.out; p.resid = a.resid;
  p.k_split = a.K; p.n_split = 1;

  if (dtype == 0) {
    switch (a.kind) {
      case LIN_PLAIN: return run_f32<EPI_STORE>(p, s);
      case LIN_GELU: return run_f32<EPI_GELU>(p, s);
      case LIN_SWIGLU: return run_f32<EPI_SWIGLU>(p, s);
      case LIN_RESID: return run_f32<EPI_RESID_TO_F32>(p, s);
      default: return run_f32<EPI_RESIDF32_TO_ACT>(p, s);
    }
  }

  const int BM = pick_bm(a.M), BN = 128;
  p.tiles_m = (a.M + BM - 1) / BM;
  p.tiles_n = (a.kind == LIN_SWIGLU) ? (a.N + BN / 2 - 1) / (BN / 2) : (a.N + BN - 1) / BN;
  int epi;
  switch (a.kind) {
    case LIN_PLAIN: epi = EPI_STORE; break;
    case LIN_GELU: epi = EPI_GELU; break;
    case LIN_SWIGLU: epi = EPI_SWIGLU; break;
    case LIN_RESID: epi = EPI_RESID_TO_F32; break;
    default: epi = EPI_RESIDF32_TO_ACT; break;
  }
  // Split-K for the residual ops when the tile grid leaves CUs idle: fp32
  // partials are added atomically into an accumulator that starts out holding
  // the residual (LIN_RESID: the fp32 output itself; LIN_RESID_F32IN: a.acc,
  // cast to the output afterwards).
  const int tiles = p.tiles_m * p.tiles_n;
  const bool resid_kind = a.kind == LIN_RESID || a.kind == LIN_RESID_F32IN;
  const bool can_split = resid_kind && a.allow_split && (a.kind == LIN_RESID || a.acc != nullptr);
  if (can_split && tiles < 160) {
    int ns = (240 + tiles - 1) / tiles;
    const int max_ns = a.K / 256 > 0 ? a.K / 256 : 1;
    if (ns > max_ns) ns = max_ns;
    if (ns > 1) {
      const int kt = (a.K + 63) / 64;
      const int kt_per = (kt + ns - 1) / ns;
      p.k_split = kt_per * 64;
      p.n_split = (kt + kt_per - 1) / kt_per;
      epi = EPI_ATOMIC;
      float* accbuf = (a.kind == LIN_RESID) ? reinterpret_cast<float*>(a.out) : a.acc;
      if (!a.acc_ready) {
        hipError_t e = launch_to_f32(a.kind == LIN_RESID ? dtype : 0, a.resid, accbuf,
                                     (size_t)a.M * a.N, s);
        if (e != hipSuccess) return e;
      }
      p.out = accbuf;
    }
  }
  p.n_tiles = p.tiles_m * p.tiles_n * p.n_split;
  hipError_t e;
  switch (BM) {
    case 64: e = run_bf16_epi<64>(epi, p, s); break;
    case 96: e = run_bf16_epi<96>(epi, p, s); break;
    case 128: e = run_bf16_epi<128>(epi, p, s); break;
    default: e = run_bf16_epi<160>(epi, p, s); break;
  }
  if (e != hipSuccess) return e;
  if (epi == EPI_ATOMIC && a.kind == LIN_RESID_F32IN)
    return launch_cast_out(dtype, a.acc, a.out, (size_t)a.M * a.N, s);
  return hipSuccess;
}

}  // namespace sarathi
