// Linear ops of the hybrid batch: one matmul over all C+B rows (Sec. 4.3,
// "fuse all the linear operations"), y = x W^T with W stored [N, K].
//
// bf16, K a multiple of 64 (every LLaMA / GPT-3 shape): gemm_ws_kernel, a
// block of producer waves that move both operands from global memory into an
// LDS ring with LDS DMA (global_load_lds_dwordx4) and consumer waves that run
// v_mfma_f32_16x16x32_bf16 on LDS-staged tiles (16-byte chunks XOR-swizzled
// by row so the operand reads are bank-conflict free).  Both operands are
// K-contiguous, so every lane moves 16 contiguous bytes.  Epilogues fuse the
// residual add (postproj, ffn_ln2), SiLU*mul (SwiGLU ffn_ln1) and GELU.
// Split-K stores one fp32 partial per split; a separate pass adds residual +
// partials in a fixed order, so results do not depend on scheduling.
//
// bf16 with a ragged K: gemm_bf16_kernel, the same tiles loaded through
// registers (k-chunks past K zeroed).  fp32: a plain LDS-tiled FMA kernel
// with the same epilogues.
#include "kernels.h"

#include <algorithm>

namespace sarathi {

enum Epi { EPI_STORE = 0, EPI_GELU = 1, EPI_SWIGLU = 2, EPI_RESID_TO_F32 = 3, EPI_RESIDF32_TO_ACT = 4,
           EPI_PARTIAL = 5, EPI_ROPE_KV = 6 };

struct GemmP {
  const void* A;        // [M, K]
  const void* W;        // [N or 2N, K]
  int M, N, K;          // N = output columns (SwiGLU: F)
  int k_split, n_split; // K elements per split; number of splits
  int tiles_m, tiles_n, n_tiles;
  int rotate_k;         // gemm_ws_kernel: 0, or the distance (in k-tiles) by which the M-tiles of a W panel
                        // rotate their k-tile order
  void* out;            // [M, N]: dtype, or fp32 for EPI_RESID_TO_F32; EPI_PARTIAL: fp32 [n_split][M, N]
  const void* resid;    // EPI_RESID_TO_F32: dtype [M,N]; EPI_RESIDF32_TO_ACT: fp32 [M,N]
  RopeArgs rope;        // EPI_ROPE_KV: rotary embedding + KV append of the preproj output
};

// Output element handling shared by both kernels.
template <typename T, int EPI>
__device__ __forceinline__ void epi_store(const GemmP& p, int r, int c, float v, int split = 0) {
  const size_t idx = (size_t)r * p.N + c;
  if (EPI == EPI_STORE) {
    reinterpret_cast<T*>(p.out)[idx] = from_f<T>(v);
  } else if (EPI == EPI_GELU) {
    reinterpret_cast<T*>(p.out)[idx] = from_f<T>(gelu_f(v));
  } else if (EPI == EPI_RESID_TO_F32) {
    reinterpret_cast<float*>(p.out)[idx] = to_f<T>(reinterpret_cast<const T*>(p.resid)[idx]) + v;
  } else if (EPI == EPI_RESIDF32_TO_ACT) {
    reinterpret_cast<T*>(p.out)[idx] = from_f<T>(reinterpret_cast<const float*>(p.resid)[idx] + v);
  } else if (EPI == EPI_PARTIAL) {
    reinterpret_cast<float*>(p.out)[(size_t)split * p.M * p.N + idx] = v;
  }
}

// ============================================================================ bf16 MFMA, register-staged
// Block tile BM x BN (W rows) x 64, WGM x WGN waves, PD register stages of
// prefetch.  Loads are unconditional (addresses clamped into the operands) so
// the compiler can keep PD tiles in flight with partial vmcnt waits; rows and
// k-chunks outside the operands are zeroed when the registers are written to
// LDS.  The k-loop runs whole groups of U tiles (tiles past the end are zero
// and add nothing), keeping every register-stage index static.
__device__ __forceinline__ uint4 mask4(const uint4& v, bool ok) {
  return make_uint4(ok ? v.x : 0u, ok ? v.y : 0u, ok ? v.z : 0u, ok ? v.w : 0u);
}

template <int BM, int BN, int WGM, int WGN, int PD, int EPI>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_bf16_kernel(GemmP p) {
  constexpr int NT = 64 * WGM * WGN;
  constexpr int BK = 64;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int RPL = NT / 8;                  // rows covered by one 16-byte load per thread
  constexpr int AL = BM / RPL, BL = BN / RPL;
  constexpr int U = (PD % 2 == 0) ? PD : 2 * PD;
  static_assert(BM % RPL == 0 && BN % RPL == 0, "load split");
  static_assert(WTM % 16 == 0 && WTN % 16 == 0 && (EPI != EPI_SWIGLU || FN % 2 == 0), "wave tile");
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
  const int wm = wave / WGN, wn = wave % WGN;
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
    const int r = m0 + lr + RPL * i;
    a_ok[i] = r < p.M;
    a_src[i] = A + (size_t)(a_ok[i] ? r : 0) * p.K;
  }
  const bf16* b_src[BL];
  bool b_ok[BL];
#pragma unroll
  for (int i = 0; i < BL; ++i) {
    const int nl = lr + RPL * i;
    int wrow;
    if (EPI == EPI_SWIGLU) {
      // each wave's WTN columns: first half gate rows, second half up rows
      const int q = nl / WTN, w = nl % WTN, half = WTN / 2;
      const int j = n0_out + q * half + (w % half);
      b_ok[i] = j < p.N;
      wrow = (w < half) ? j : p.N + j;
    } else {
      wrow = n0_out + nl;
      b_ok[i] = wrow < p.N;
    }
    b_src[i] = W + (size_t)(b_ok[i] ? wrow : 0) * p.K;
  }

  uint4 R[PD][AL + BL];
  auto gload = [&](uint4* r, int kt) {
    const int kc = min(kt, nk - 1);
    const int kk = min(kbeg + kc * BK + lc * 8, p.K - 8);
#pragma unroll
    for (int i = 0; i < AL; ++i) r[i] = *reinterpret_cast<const uint4*>(a_src[i] + kk);
#pragma unroll
    for (int i = 0; i < BL; ++i) r[AL + i] = *reinterpret_cast<const uint4*>(b_src[i] + kk);
  };
  auto sstore = [&](int buf, const uint4* r, int kt) {
    uint4* s = lds + buf * (BM + BN) * 8;
    const bool kok = kbeg + kt * BK + lc * 8 < kend;
#pragma unroll
    for (int i = 0; i < AL; ++i) {
      const int row = lr + RPL * i;
      s[row * 8 + (lc ^ (row & 7))] = mask4(r[i], a_ok[i] && kok);
    }
#pragma unroll
    for (int i = 0; i < BL; ++i) {
      const int row = BM + lr + RPL * i;
      s[row * 8 + (lc ^ (row & 7))] = mask4(r[AL + i], b_ok[i] && kok);
    }
  };

  floatx4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int buf) {
    const uint4* s = lds + buf * (BM + BN) * 8;
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
  };

  if (nk > 0) {
#pragma unroll
    for (int st = 0; st < PD; ++st) gload(R[st], st);
    sstore(0, R[0], 0);
    gload(R[0], PD);
    __syncthreads();
    for (int kb = 0; kb < nk; kb += U) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int kt = kb + u;
        compute(u & 1);
        sstore((u + 1) & 1, R[(u + 1) % PD], kt + 1);
        gload(R[(u + 1) % PD], kt + 1 + PD);
        __syncthreads();
      }
    }
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
          if (c < p.N) epi_store<bf16, EPI>(p, r, c, acc[fm][fn][i], split);
        }
      }
    }
  }
}

// ============================================================================ bf16 MFMA, producer/consumer waves
// The memory pipeline of a CU holds a bounded number of outstanding cache-line
// requests, and a wave that issues a load while it is full stalls at the
// issue.  When the same waves load and multiply, those stalls serialise the
// operand feed with the MFMAs.  Here NP producer waves only issue LDS DMA
// loads (and wait for them) while WGM x WGN consumer waves only read LDS and
// run MFMAs; one barrier per k-tile hands a filled stage to the consumers
// and the consumed stage back to the producers.  S-stage LDS ring, K a
// multiple of 64.
template <int EPI, int WTN>
__device__ __forceinline__ int w_row_of(int nl, int n0_out, int N) {
  if (EPI == EPI_SWIGLU) {
    // each consumer wave's WTN columns: first half gate rows, second half up rows
    const int q = nl / WTN, w = nl % WTN, half = WTN / 2;
    const int jj = n0_out + q * half + (w % half);
    return jj < N ? ((w < half) ? jj : N + jj) : 0;
  }
  return min(n0_out + nl, N - 1);
}

// Preproj with the rotary embedding and the KV append fused (the "others" of
// Sec. 2.1 that follow the QKV matmul).  The rotary pairs are (d, d + hd/2)
// of a head; so that any tile holds whole pairs, the producers load W's rows
// in pair order: within each head, logical columns 16g .. 16g+7 are physical
// columns 8g .. 8g+7 and logical 16g+8 .. 16g+15 are physical hd/2 + 8g ..
// hd/2 + 8g+7.  Every 16-column group of a tile is then 8 complete pairs of
// one head of q, k or v (hd a multiple of 16).
__device__ __forceinline__ int rope_w_row(int n, int N, int hd) {
  n = min(n, N - 1);
  const int c = n % hd;
  return n - c + ((c >> 3) & 1) * (hd / 2) + (c >> 4) * 8 + (c & 7);
}

// The epilogue: the block's tile goes to LDS as bf16 (the rounding the
// separate kernel would read); each thread then keeps one 16-column group
// (one head, 8 frequencies computed once in fp64) and walks rows: q is
// rotated into the output, k rotated and v copied into the KV cache at the
// row's (slot, position), 16 bytes per access, both halves of the pairs
// back at their physical columns.  The k and v columns of the output are not
// written (attention reads them from the cache).
template <int BM, int BN, int WGM, int WGN, int WTM, int WTN, int FM, int FN>
__device__ __forceinline__ void rope_kv_epilogue(const GemmP& p, floatx4 (&acc)[FM][FN], int m0, int n0, int wm,
                                                 int wn, int lane, int tid) {
  extern __shared__ uint4 lds[];
  bf16* t = reinterpret_cast<bf16*>(lds);                  // [BM][BN] bf16
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = wm * WTM + fm * 16 + 4 * (lane >> 4) + i;
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) t[r * BN + wn * WTN + fn * 16 + (lane & 15)] = f2bf(acc[fm][fn][i]);
    }
  lds_read_barrier();                                       // the producers pass their last barrier too
  constexpr int JG = BN / 16;                               // 16-column groups per tile row
  constexpr int RS = (64 * WGM * WGN) / JG;                 // rows in flight
  static_assert(BN % 16 == 0 && RS > 0, "16-column groups");
  const int j = tid % JG, r0 = tid / JG;
  const int n = n0 + 16 * j;
  if (r0 >= RS || n >= p.N) return;
  const RopeArgs& a = p.rope;
  const int hd = a.hd, half = hd / 2, QD = a.nh * hd;
  const int part = n / QD, head = (n % QD) / hd;            // part 0 q, 1 k, 2 v
  const int d0 = (n % hd) / 2;                              // first pair of the group
  const bool rot = part < 2 && a.rope;
  double theta[8];
  if (rot) {
    const double lb = log2((double)a.base);
#pragma unroll
    for (int e = 0; e < 8; ++e) theta[e] = rope_theta(d0 + e, hd, lb);
  }
  bf16* cache = reinterpret_cast<bf16*>(a.kv_layer);
  const size_t kv_off = (part == 2 ? a.st.kv : 0) + (size_t)head * a.st.head;
  for (int r = r0; r < BM; r += RS) {
    const int row = m0 + r;
    if (row >= p.M) break;
    uint4 lo = *reinterpret_cast<const uint4*>(t + r * BN + 16 * j);
    uint4 hi = *reinterpret_cast<const uint4*>(t + r * BN + 16 * j + 8);
    const int slot = a.row_slot[row], pos = a.row_pos[row];
    if (rot) {
      float x0[8], x1[8];
      Vec16<bf16>::unpack(lo, x0);
      Vec16<bf16>::unpack(hi, x1);
      uint32_t w0[4], w1[4];
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        float s0, c0, s1, c1;
        rope_sincos(pos, theta[e], &s0, &c0);
        rope_sincos(pos, theta[e + 1], &s1, &c1);
        const bf16 a0 = f2bf(x0[e] * c0 - x1[e] * s0), b0 = f2bf(x0[e] * s0 + x1[e] * c0);
        const bf16 a1 = f2bf(x0[e + 1] * c1 - x1[e + 1] * s1), b1 = f2bf(x0[e + 1] * s1 + x1[e + 1] * c1);
        w0[e / 2] = (uint32_t)a0 | ((uint32_t)a1 << 16);
        w1[e / 2] = (uint32_t)b0 | ((uint32_t)b1 << 16);
      }
      lo = make_uint4(w0[0], w0[1], w0[2], w0[3]);
      hi = make_uint4(w1[0], w1[1], w1[2], w1[3]);
    }
    bf16* dst = part == 0 ? reinterpret_cast<bf16*>(p.out) + (size_t)row * p.N + (n - n % hd)
                          : cache + (size_t)slot * a.st.slot + kv_off + (size_t)pos * a.st.pos;
    *reinterpret_cast<uint4*>(dst + d0) = lo;
    *reinterpret_cast<uint4*>(dst + half + d0) = hi;
  }
}

template <int BM, int BN, int WGM, int WGN, int NP, int S, int EPI>
__global__ __launch_bounds__(64 * (WGM * WGN + NP)) void gemm_ws_kernel(GemmP p) {
  constexpr int NC = WGM * WGN;
  constexpr int BK = 64;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int ROWS = BM + BN;
  constexpr int G = ROWS / 8, GA = BM / 8;
  constexpr int IHI = (G + NP - 1) / NP, ILO = G / NP, RHI = G % NP;
  static_assert(BM % 8 == 0 && BN % 8 == 0 && ILO > 0, "8-row groups");
  static_assert(WTM % 16 == 0 && WTN % 16 == 0 && (EPI != EPI_SWIGLU || FN % 2 == 0), "wave tile");
  static_assert((S - 2) * IHI < 64 && S >= 2, "stages");
  static_assert(BM * BN * 2 <= S * ROWS * 128, "the RoPE epilogue stages the bf16 tile in the ring's LDS");
  extern __shared__ uint4 lds[];                 // [S][ROWS * 8] 16-byte chunks

  const int per = gridDim.x / 8;
  const int t = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (t >= p.n_tiles) return;
  const int tile_m = t % p.tiles_m;
  const int rest = t / p.tiles_m;
  const int split = rest % p.n_split;
  const int tile_n = rest / p.n_split;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = tile_m * BM;
  const int n0_out = tile_n * (EPI == EPI_SWIGLU ? BN / 2 : BN);
  const int kbeg = split * p.k_split;
  const int kend = min(p.K, kbeg + p.k_split);
  const int nk = (kend - kbeg) / BK;

  if (wave >= NC) {
    // ---------------- producer
    // The wave index is uniform: the LDS destinations (m0) and the matrix
    // bases are scalar, and each lane keeps one 32-bit byte offset per row
    // group, so a request costs no vector instruction (global_load_lds with
    // a scalar base; the launcher keeps both matrices below 4 GiB).
    const int q = __builtin_amdgcn_readfirstlane(wave - NC);
    const char* A = reinterpret_cast<const char*>(p.A) + (size_t)kbeg * 2;
    const char* W = reinterpret_cast<const char*>(p.W) + (size_t)kbeg * 2;
    const int lchunk = (lane & 7) ^ (lane >> 3);
    uint32_t off[IHI];
#pragma unroll
    for (int j = 0; j < IHI; ++j) {
      const int g = min(j * NP + q, G - 1);
      const int row = g * 8 + (lane >> 3);
      const int nl = row - BM;
      const size_t r = g < GA                  ? (size_t)min(m0 + row, p.M - 1)
                       : EPI == EPI_ROPE_KV ? (size_t)rope_w_row(n0_out + nl, p.N, p.rope.hd)
                                            : (size_t)w_row_of<EPI, WTN>(nl, n0_out, p.N);
      off[j] = (uint32_t)(r * p.K * 2 + lchunk * 16);
    }
    const bool extra = q < RHI;
    // With rotate_k, the G = tiles_m blocks that share a W panel take each
    // group of G k-tiles in rotated orders (block m starts at m), so every
    // k-tile of the panel is first requested by one block -- which pays the
    // HBM latency -- and found in L2 by the others a step later, instead of
    // all G waiting on the same miss.
    const int G = p.rotate_k ? p.tiles_m : 1, RD = p.rotate_k, GR = G * RD;
    auto issue = [&](int stage, int kt) {
      if (G > 1) {
        const int base = kt / GR * GR;
        if (base + GR <= nk) kt = base + (kt - base + tile_m * RD) % GR;
      }
      uint4* dst = lds + stage * ROWS * 8;
      const char* a_k = A + (size_t)kt * BK * 2;
      const char* w_k = W + (size_t)kt * BK * 2;
#pragma unroll
      for (int j = IHI - 1; j >= 0; --j)
        if (j < ILO || extra) dma16((min(j * NP + q, ROWS / 8 - 1) < GA ? a_k : w_k) + off[j], dst + (j * NP + q) * 64);
    };
    auto wait_next = [&](bool all) {   // all but the newest S - 2 stages landed
      if (all) wait_vmcnt<0>();
      else if (extra) wait_vmcnt<(S - 2) * IHI>();
      else wait_vmcnt<(S - 2) * ILO>();
    };
#pragma unroll
    for (int st = 0; st < S - 1; ++st)
      if (st < nk) issue(st, st);
    wait_next(S - 2 >= nk);
    lds_barrier();
    int nbuf = S - 1;
    for (int kt = 0; kt < nk; ++kt) {
      const bool more = kt + S - 1 < nk;
      if (more) issue(nbuf, kt + S - 1);
      wait_next(!more);
      lds_barrier();
      nbuf = (nbuf + 1 == S) ? 0 : nbuf + 1;
    }
    if constexpr (EPI == EPI_ROPE_KV) lds_barrier();   // pairs with the consumers' epilogue barrier
    return;
  }

  // ---------------- consumer
  const int wm = wave / WGN, wn = wave % WGN;
  floatx4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  lds_barrier();
  int buf = 0;
  for (int kt = 0; kt < nk; ++kt) {
    const uint4* s = lds + buf * ROWS * 8;
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
    lds_read_barrier();
    buf = (buf + 1 == S) ? 0 : buf + 1;
  }

  if constexpr (EPI == EPI_ROPE_KV) {
    rope_kv_epilogue<BM, BN, WGM, WGN, WTM, WTN, FM, FN>(p, acc, m0, tile_n * BN, wm, wn, lane, tid);
    return;
  }
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
          if (c < p.N) epi_store<bf16, EPI>(p, r, c, acc[fm][fn][i], split);
        }
      }
    }
  }
}

// ============================================================================ fp32 FMA
// 64x64 tile of W rows (SwiGLU: 32 gate + 32 up rows -> 32 outputs), BK 64
// (few k-steps: the small fp32 matmuls run few blocks and are latency-bound),
// 16x16 threads with 4x4 results each.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmP p) {
  constexpr int BK = 64;
  __shared__ float As[BK][64 + 4];
  __shared__ float Ws[BK][64 + 4];
  const int tile_m = blockIdx.x, tile_n = blockIdx.y;
  // split-K (EPI_PARTIAL): blockIdx.z takes k in [z * k_split, (z + 1) * k_split)
  const int split = blockIdx.z;
  const int kbeg = split * p.k_split, kend = min(p.K, kbeg + p.k_split);
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = tile_m * 64;
  const int n0_out = tile_n * (EPI == EPI_SWIGLU ? 32 : 64);
  const float* A = reinterpret_cast<const float*>(p.A);
  const float* W = reinterpret_cast<const float*>(p.W);
  int cols[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) cols[j] = (EPI == EPI_SWIGLU) ? ((j < 2) ? 2 * tx + j : 32 + 2 * tx + j - 2) : 4 * tx + j;
  float acc[4][4] = {};
  // Each thread stages PER elements of A and of W per k-step.  All loads are
  // issued before any is used (addresses clamped into the operands, values
  // outside them zeroed afterwards), so a k-step waits for one memory round
  // trip rather than one per element.
  constexpr int PER = 64 * BK / 256;
  for (int k0 = kbeg; k0 < kend; k0 += BK) {
    float ra[PER], rw[PER];
    bool oka[PER], okw[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = threadIdx.x + i * 256;
      const int r = e / BK, kk = e % BK;
      const int gr = m0 + r, gk = k0 + kk;
      const int ck = min(gk, p.K - 1);
      int wrow, jn;
      if (EPI == EPI_SWIGLU) {
        jn = n0_out + (r % 32);
        wrow = (r < 32) ? min(jn, p.N - 1) : p.N + min(jn, p.N - 1);
      } else {
        jn = n0_out + r;
        wrow = min(jn, p.N - 1);
      }
      oka[i] = gr < p.M && gk < kend;
      okw[i] = jn < p.N && gk < kend;
      ra[i] = A[(size_t)min(gr, p.M - 1) * p.K + ck];
      rw[i] = W[(size_t)wrow * p.K + ck];
    }
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = threadIdx.x + i * 256;
      const int r = e / BK, kk = e % BK;
      As[kk][r] = oka[i] ? ra[i] : 0.f;
      Ws[kk][r] = okw[i] ? rw[i] : 0.f;
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
        if (c < p.N) epi_store<float, EPI>(p, r, c, acc[i][j], split);
      }
    }
  }
}

// ============================================================================ launch
// Tile configurations of the bf16 kernel (BM x BN W rows, waves, prefetch stages).
enum TileCfg { CFG_160x128 = 0, CFG_320x128 = 1, CFG_64x128 = 2, CFG_96x128 = 3 };

template <int BM, int BN, int WGM, int WGN, int PD, int EPI>
static hipError_t run_bf16(GemmP p, hipStream_t s) {
  const size_t lds_bytes = 2 * (BM + BN) * 8 * sizeof(uint4);
  static std::atomic<uint64_t> lds_set{0};   // devices on which this instance's LDS limit is raised
  hipError_t e = ensure_dynamic_lds((const void*)gemm_bf16_kernel<BM, BN, WGM, WGN, PD, EPI>, (int)lds_bytes, lds_set);
  if (e != hipSuccess) return e;
  const int grid = (p.n_tiles + 7) / 8 * 8;
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WGM, WGN, PD, EPI>), dim3(grid), dim3(64 * WGM * WGN), lds_bytes,
                     s, p);
  return hipGetLastError();
}

template <int BM, int BN, int WGM, int WGN, int NP, int S, int EPI>
static hipError_t run_ws(GemmP p, hipStream_t s) {
  const size_t lds_bytes = (size_t)S * (BM + BN) * 8 * sizeof(uint4);
  static std::atomic<uint64_t> lds_set{0};   // devices on which this instance's LDS limit is raised
  hipError_t e = ensure_dynamic_lds((const void*)gemm_ws_kernel<BM, BN, WGM, WGN, NP, S, EPI>, (int)lds_bytes, lds_set);
  if (e != hipSuccess) return e;
  const int grid = (p.n_tiles + 7) / 8 * 8;
  hipLaunchKernelGGL((gemm_ws_kernel<BM, BN, WGM, WGN, NP, S, EPI>), dim3(grid), dim3(64 * (WGM * WGN + NP)),
                     lds_bytes, s, p);
  return hipGetLastError();
}

template <int BM, int BN, int WGM, int WGN, int PD>
static hipError_t run_bf16_epi(int epi, const GemmP& p, hipStream_t s) {
  switch (epi) {
    case EPI_STORE: return run_bf16<BM, BN, WGM, WGN, PD, EPI_STORE>(p, s);
    case EPI_GELU: return run_bf16<BM, BN, WGM, WGN, PD, EPI_GELU>(p, s);
    case EPI_SWIGLU: return run_bf16<BM, BN, WGM, WGN, PD, EPI_SWIGLU>(p, s);
    case EPI_RESID_TO_F32: return run_bf16<BM, BN, WGM, WGN, PD, EPI_RESID_TO_F32>(p, s);
    case EPI_RESIDF32_TO_ACT: return run_bf16<BM, BN, WGM, WGN, PD, EPI_RESIDF32_TO_ACT>(p, s);
    default: return run_bf16<BM, BN, WGM, WGN, PD, EPI_PARTIAL>(p, s);
  }
}

template <int EPI>
static hipError_t run_f32(const GemmP& p, hipStream_t s) {
  const int out_per_tile = (EPI == EPI_SWIGLU) ? 32 : 64;
  dim3 grid((p.M + 63) / 64, (p.N + out_per_tile - 1) / out_per_tile, p.n_split);
  hipLaunchKernelGGL(gemm_f32_kernel<EPI>, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

static int cfg_bm(int cfg) {
  switch (cfg) {
    case CFG_320x128: return 320;
    case CFG_64x128: return 64;
    case CFG_96x128: return 96;
    default: return 160;
  }
}

// Tile choice for the skinny matmuls of the hybrid batch (M = C + B rows).
// Many W panels (>= 180 tiles of 128 rows) and M in (160, 320]: one block
// covers all rows (W read once per block, 8 waves).  A middle count: 160-row
// blocks.  Few panels (postproj / ffn_ln2 at N = hidden): 64-row blocks with
// split-K -- or, when split-K scratch is available and M in (160, 320],
// 320-row blocks split over K (chosen by the caller).  Small M: the block
// height that pads M least.
static int pick_cfg(int M, int n_panels) {
  if (M <= 64) return CFG_64x128;
  if (M <= 96) return CFG_96x128;
  if (n_panels >= 180 && M > 160 && M <= 320) return CFG_320x128;
  if (n_panels >= 100) {
    const int pad160 = (M + 159) / 160 * 160, pad96 = (M + 95) / 96 * 96;
    return pad96 < pad160 ? CFG_96x128 : CFG_160x128;
  }
  return CFG_64x128;
}

// Producer/consumer tiles (BM x BN W rows; consumer waves 2 x (BN / 32), or
// 2 x 2 for BN = 64; 4 producer waves, 2 beside 14 consumers) and their LDS
// ring depth (~100-156 KB).
struct WsTile {
  int bm, bn;
};
constexpr WsTile kWsTiles[] = {{64, 64},   {64, 128},  {64, 256},  {96, 128},  {96, 192},
                               {96, 256},  {160, 128}, {160, 192}, {160, 224}, {160, 256}};
constexpr int kNumWsTiles = sizeof(kWsTiles) / sizeof(kWsTiles[0]);

template <int EPI>
static hipError_t run_ws_cfg(int cfg, const GemmP& p, hipStream_t s) {
  switch (cfg) {
    case 0: return run_ws<64, 64, 2, 2, 4, 6, EPI>(p, s);
    case 1: return run_ws<64, 128, 2, 4, 4, 6, EPI>(p, s);
    case 2: return run_ws<64, 256, 2, 4, 4, 3, EPI>(p, s);
    case 3: return run_ws<96, 128, 2, 4, 4, 5, EPI>(p, s);
    case 4: return run_ws<96, 192, 2, 6, 4, 4, EPI>(p, s);
    case 5: return run_ws<96, 256, 2, 4, 4, 3, EPI>(p, s);
    case 6: return run_ws<160, 128, 2, 4, 4, 4, EPI>(p, s);
    case 7: return run_ws<160, 192, 2, 6, 4, 3, EPI>(p, s);
    case 8: return run_ws<160, 224, 2, 7, 2, 3, EPI>(p, s);
    default: return run_ws<160, 256, 2, 4, 4, 3, EPI>(p, s);
  }
}

static hipError_t run_ws_epi(int epi, int cfg, const GemmP& p, hipStream_t s) {
  switch (epi) {
    case EPI_STORE: return run_ws_cfg<EPI_STORE>(cfg, p, s);
    case EPI_GELU: return run_ws_cfg<EPI_GELU>(cfg, p, s);
    case EPI_SWIGLU: return run_ws_cfg<EPI_SWIGLU>(cfg, p, s);
    case EPI_RESID_TO_F32: return run_ws_cfg<EPI_RESID_TO_F32>(cfg, p, s);
    case EPI_RESIDF32_TO_ACT: return run_ws_cfg<EPI_RESIDF32_TO_ACT>(cfg, p, s);
    case EPI_ROPE_KV: return run_ws_cfg<EPI_ROPE_KV>(cfg, p, s);
    default: return run_ws_cfg<EPI_PARTIAL>(cfg, p, s);
  }
}

// Tile (and K-split) choice from a cost model of the operand feed, fitted to
// MI355X measurements of the LLaMA-13B / 33B shapes.  Each CU runs one block
// at a time and is bound by its outstanding memory requests: a 64-wide k-tile
// costs ~1.9 ns per A row (L2 hits) and ~3.1 ns per W row when two M-tiles
// share the W panel (~4.2 ns when one block streams it alone: every row an
// HBM miss); a block adds ~3 us of pipeline fill plus its output writes
// (~40 GB/s per CU); blocks beyond the first 256 run as another round.  A
// split-K op's reduction pass reads the fp32 partials and writes the result
// at ~5.5 TB/s.
struct WsChoice {
  int cfg, n_split;
};
static WsChoice pick_ws(int M, int N, int K, bool swiglu, int max_split) {
  WsChoice best{6, 1};
  double best_t = 1e300;
  const int nk = K / 64;
  for (int c = 0; c < kNumWsTiles; ++c) {
    const int bm = kWsTiles[c].bm, bn = kWsTiles[c].bn;
    if (bm == 64 && M > 64) continue;    // 64-row tiles only for short batches
    const int per = swiglu ? bn / 2 : bn;
    const int tiles_m = (M + bm - 1) / bm;
    const long tiles = (long)tiles_m * ((N + per - 1) / per);
    const double per_k = 1.9e-3 * bm + (tiles_m >= 2 ? 3.1e-3 : 4.2e-3) * bn;   // us per k-tile
    for (int ns = 1; ns <= max_split; ++ns) {
      const double rounds = (double)((tiles * ns + 255) / 256);
      const double k_tiles = 2.0 * ((nk / 2 + ns - 1) / ns);               // whole pairs per split
      const double out_bytes = (double)bm * (swiglu ? bn / 2 : bn) * (ns > 1 ? 4.0 : 2.0);
      double t = rounds * (k_tiles * per_k + 3.0 + out_bytes / 4.0e4);
      if (ns > 1) t += (ns * 4.0 + 6.0) * (double)M * N / 5.5e6 + 2.0;
      if (t < best_t * 0.999) {
        best_t = t;
        best = {c, ns};
      }
    }
  }
  return best;
}

int linear_tile_count() { return kNumWsTiles; }
bool linear_tile_shape(int tile, int* bm, int* bn) {
  if (tile < 0 || tile >= kNumWsTiles) return false;
  *bm = kWsTiles[tile].bm;
  *bn = kWsTiles[tile].bn;
  return true;
}

hipError_t launch_linear(int dtype, const LinearArgs& a, hipStream_t s, int force_tile, int force_split,
                         LinearPlan* plan) {
  if (plan) *plan = LinearPlan{0, 0, 0};
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  GemmP p{};
  p.A = a.x; p.W = a.w; p.M = a.M; p.N = a.N; p.K = a.K;
  p.out = a.out; p.resid = a.resid;
  p.k_split = a.K; p.n_split = 1;

  if (dtype == 0) {
    // Split-K for the residual ops when the 64x64 tiles leave most CUs idle:
    // fp32 partials per split of whole 64-wide k-steps, then residual +
    // partials added in split order (deterministic).
    const bool resid_kind = a.kind == LIN_RESID || a.kind == LIN_RESID_F32IN;
    const int tiles = ((a.M + 63) / 64) * ((a.N + 63) / 64);
    if (resid_kind && a.parts != nullptr && tiles < 64) {
      int ns = std::min(std::min(MAX_SPLIT, (64 + tiles - 1) / tiles), (a.K + 127) / 128);
      ns = (int)std::min<size_t>((size_t)ns, a.parts_cap / ((size_t)a.M * a.N));
      if (ns > 1) {
        const int steps = (a.K + 63) / 64;
        p.k_split = (steps + ns - 1) / ns * 64;
        p.n_split = (a.K + p.k_split - 1) / p.k_split;
        p.out = a.parts;
        if (plan) {
          *plan = LinearPlan{64, 64, p.n_split};
          return hipSuccess;
        }
        hipError_t e = run_f32<EPI_PARTIAL>(p, s);
        if (e != hipSuccess) return e;
        return launch_split_reduce(0, a.kind == LIN_RESID_F32IN, a.kind == LIN_RESID, a.resid, a.parts, p.n_split,
                                   (size_t)a.M * a.N, a.out, s);
      }
    }
    if (plan) {
      *plan = LinearPlan{64, 64, 1};
      return hipSuccess;
    }
    switch (a.kind) {
      case LIN_PLAIN: return run_f32<EPI_STORE>(p, s);
      case LIN_GELU: return run_f32<EPI_GELU>(p, s);
      case LIN_SWIGLU: return run_f32<EPI_SWIGLU>(p, s);
      case LIN_RESID: return run_f32<EPI_RESID_TO_F32>(p, s);
      default: return run_f32<EPI_RESIDF32_TO_ACT>(p, s);
    }
  }

  int epi;
  switch (a.kind) {
    case LIN_PLAIN: epi = EPI_STORE; break;
    case LIN_GELU: epi = EPI_GELU; break;
    case LIN_SWIGLU: epi = EPI_SWIGLU; break;
    case LIN_RESID: epi = EPI_RESID_TO_F32; break;
    default: epi = EPI_RESIDF32_TO_ACT; break;
  }
  const bool swiglu = a.kind == LIN_SWIGLU;
  const bool resid_kind = a.kind == LIN_RESID || a.kind == LIN_RESID_F32IN;
  // producer/consumer kernel: whole 64-wide k-tiles, and x and W each under
  // 4 GiB (its producers address rows by 32-bit byte offsets)
  const size_t w_rows = swiglu ? 2 * (size_t)a.N : (size_t)a.N;
  const bool ws = (a.K % 64) == 0 && (size_t)a.M * a.K * 2 < (1ull << 32) && w_rows * a.K * 2 < (1ull << 32);

  // splits available to the residual ops: whole groups of two k-tiles per
  // split, partials must fit the scratch
  int max_split = 1;
  if (resid_kind && a.parts != nullptr) {
    max_split = std::min(MAX_SPLIT, (a.K + 127) / 128 / 2);
    max_split = (int)std::min<size_t>((size_t)max_split, a.parts_cap / ((size_t)a.M * a.N));
    max_split = std::max(max_split, 1);
  }
  int cfg, BM, BN, ws_split = 1;
  if (ws) {
    WsChoice ch = pick_ws(a.M, a.N, a.K, swiglu, max_split);
    if (force_tile >= 0 && force_tile < kNumWsTiles) ch = {force_tile, std::min(std::max(force_split, 1), max_split)};
    cfg = ch.cfg;
    ws_split = ch.n_split;
    BM = kWsTiles[cfg].bm;
    BN = kWsTiles[cfg].bn;
  } else {
    BN = 128;
    const int n_panels = (a.N + (swiglu ? BN / 2 : BN) - 1) / (swiglu ? BN / 2 : BN);
    const bool split_kind = resid_kind && a.parts != nullptr;
    cfg = (split_kind && a.M > 160 && a.M <= 320 && n_panels < 256) ? CFG_320x128 : pick_cfg(a.M, n_panels);
    BM = cfg_bm(cfg);
  }
  const int out_per_tile = swiglu ? BN / 2 : BN;
  p.tiles_m = (a.M + BM - 1) / BM;
  p.tiles_n = (a.N + out_per_tile - 1) / out_per_tile;
  // preproj with the rotary embedding and KV append in its epilogue (W rows
  // loaded in rotary-pair order, any tile)
  if (ws && a.kind == LIN_PLAIN && a.rope != nullptr) {
    const int hd = a.rope->hd, QD = a.rope->nh * hd;
    if (hd % 16 == 0 && a.N == 3 * QD) {
      epi = EPI_ROPE_KV;
      p.rope = *a.rope;
      if (a.rope_done) *a.rope_done = true;
    }
  }

  // Split-K for the residual ops when the tile grid leaves CUs idle: every
  // split stores its fp32 partial, then one pass adds residual + partials in
  // split order (deterministic).  Each split covers whole groups of two
  // 64-wide k-tiles.  Blocks of ~150 KB of LDS run one per CU, so the split
  // count keeps the grid within one wave of blocks over the 256 CUs.
  const int tiles = p.tiles_m * p.tiles_n;
  int n_split = 1;
  if (resid_kind && a.parts != nullptr && (ws ? ws_split > 1 : tiles < 256)) {
    const int kgroups = (a.K + 127) / 128;
    int ns = ws ? ws_split : (cfg == CFG_320x128 ? 256 / tiles : (400 + tiles - 1) / tiles);
    if (ns > kgroups / 2) ns = kgroups / 2;
    if (ns > MAX_SPLIT) ns = MAX_SPLIT;
    if ((size_t)ns * a.M * a.N > a.parts_cap) ns = (int)(a.parts_cap / ((size_t)a.M * a.N));
    if (ns > 1) {
      const int g_per = (kgroups + ns - 1) / ns;
      p.k_split = g_per * 128;
      p.n_split = (a.K + p.k_split - 1) / p.k_split;
      n_split = p.n_split;
      epi = EPI_PARTIAL;
      p.out = a.parts;
    }
  }
  p.n_tiles = p.tiles_m * p.tiles_n * p.n_split;
  // Rotated k order for the two M-tiles of a W panel, when a block runs at
  // most 192 k-tiles.  Measured in the layers: LLaMA-13B preproj -13% and
  // ffn_ln1 -2%; LLaMA-33B at 288 rows every op -2..-5% (layer -4%); GPT-3
  // preproj, postproj and ffn_ln1 -2..-6% (96-192 k-tiles); but GPT-3 ffn_ln2
  // (384 k-tiles per split) +6%.  Four M-tiles: no gain.
  {
    const int nk_block = (n_split > 1 ? p.k_split : a.K) / 64;
    p.rotate_k = (ws && p.tiles_m == 2 && nk_block <= 192) ? 1 : 0;
  }
  if (plan) {
    *plan = LinearPlan{BM, BN, p.n_split};
    return hipSuccess;
  }
  hipError_t e;
  if (ws) {
    e = run_ws_epi(epi, cfg, p, s);
  } else {
    switch (cfg) {
      case CFG_320x128: e = run_bf16_epi<320, 128, 4, 2, 2>(epi, p, s); break;
      case CFG_64x128: e = run_bf16_epi<64, 128, 2, 2, 2>(epi, p, s); break;
      case CFG_96x128: e = run_bf16_epi<96, 128, 2, 2, 2>(epi, p, s); break;
      default: e = run_bf16_epi<160, 128, 2, 2, 2>(epi, p, s); break;
    }
  }
  if (e != hipSuccess) return e;
  if (n_split > 1) {
    if (a.norm != nullptr && resid_kind && dtype == 1) {
      e = launch_split_reduce_norm(a.resid, a.kind == LIN_RESID_F32IN, a.parts, n_split, a.M, a.N, a.out, *a.norm, s);
      if (e == hipSuccess && a.norm_done) *a.norm_done = true;
      if (e != hipErrorNotSupported) return e;
    }
    return launch_split_reduce(dtype, a.kind == LIN_RESID_F32IN, a.kind == LIN_RESID, a.resid, a.parts, n_split,
                               (size_t)a.M * a.N, a.out, s);
  }
  return hipSuccess;
}

}  // namespace sarathi
