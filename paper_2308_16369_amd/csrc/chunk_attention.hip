// Attention of the prompt chunk(s) of the hybrid batch, run separately from the
// decodes (Sec. 4.3).  A work item that sees every key of its rows writes
// their attention output directly; a key range of a split item is written as
// a partial result (max, sum, unnormalised o) that the combine pass of
// attention_combine.hip merges per row.
//
// Chunked-prefill attention (bf16, MFMA): the chunk's queries at positions
// off..off+C-1 attend to the prefill slot's keys 0..position (the earlier
// chunks' cached keys plus, causally, the chunk's own; Sec. 4.2).  Work item
// = (block of qblock queries, a range of 64-key tiles), one head per block of
// qblock / 32 waves x 32 query rows; qblock is PREFILL_QBLOCK (8 waves) or
// PREFILL_QBLOCK_SMALL (4 waves), chosen per batch by the plan.  K and V tiles of 64
// keys are staged in LDS rings by LDS DMA (V read back transposed so P*V
// takes 16 contiguous bytes per lane); S = Q K^T and O += P V run on
// v_mfma_f32_32x32x16_bf16 with an fp32 online softmax.
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
//
// The chunk-attention loop issues its LDS reads as inline assembly, with the
// LDS-counter wait written out (lds_wait): the compiler treats every LDS
// read as possibly overlapping the tile stages that LDS DMA is still filling
// and would otherwise wait for all outstanding DMA (vmcnt 0) before the
// first read of V, which would drain the K/V prefetch every tile.  The
// stages a tile reads are made complete by the vmcnt wait and barrier at the
// top of its iteration.  The wait takes the loaded registers as operands so
// that no use of them can be scheduled before it.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }
template <int OFF>
__device__ __forceinline__ u32x2 lds_tr16_asm(uint32_t addr) {
  u32x2 v;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
  return v;
}
template <int OFF>
__device__ __forceinline__ u32x4 lds_b128_asm(uint32_t addr) {
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
  return v;
}
template <int N, typename T>
__device__ __forceinline__ void lds_wait(T (&r)[N]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(r[i]));
}
// The same, leaving the newest K LDS reads in flight (they complete in issue
// order): the N registers of the group issued before them have landed.
template <int K, int N, typename T>
__device__ __forceinline__ void lds_wait_but(T (&r)[N]) {
  static_assert(K >= 0 && K < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(K) : "memory");
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(r[i]));
}

// 16-byte chunk swizzle of a K/V row (D / 8 chunks): key row r keeps
// logical chunk c at c ^ f(r).  For head_dim 128 (256-byte rows, one row
// per pass over the 64 banks) f is a bijection of r mod 16 that moves
// aligned groups of four chunks together: 16 consecutive rows read at one
// chunk (the K operand) land on 16 distinct chunk positions, and the four
// consecutive rows x four chunks of a transposed V read by 32 lanes land on
// four distinct groups of four.
template <int D>
__device__ __forceinline__ int kv_swz(int c, int r) {
  if (D == 128) return c ^ (((r & 3) << 2) | ((r >> 2) & 3));
  return c ^ (r & 7);
}

typedef float floatx16 __attribute__((ext_vector_type(16)));

// Max and sum of the values of lanes l and l ^ 32 (v_permlane32_swap hands
// each lane both values; no LDS traffic).
__device__ __forceinline__ f32x2_t lanes_pair(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return f32x2_t{__uint_as_float(r[0]), __uint_as_float(r[1])};
}
// Maximum that propagates NaN (v_maximum3_f32; fmaxf would first quieten
// every matrix-core output).  No score is NaN.
__device__ __forceinline__ float fmax_nan(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float pair_max(float x) { const f32x2_t p = lanes_pair(x); return fmax_nan(p.x, p.y); }
__device__ __forceinline__ float pair_sum(float x) { const f32x2_t p = lanes_pair(x); return p.x + p.y; }

// One block = one head x (32 * NW queries of the chunk, one range of keys);
// wave w owns queries w*32 .. w*32+31.  Per 64-key tile:
//   S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (A = 32 key rows of the K tile,
//     B = the wave's Q^T fragments held in registers), two 32-key blocks;
//     lane l holds, per block, the 16 scores of query l % 32 for keys
//     8*(v/4) + 4*(l/32) + v%4;
//   the online softmax runs on each query's registers (the query's other
//     keys sit in lane l ^ 32: one lane swap for the max, one for the sum
//     at the end);
//   O^T += V^T P^T (32x32x16: B = the lane's probabilities packed as bf16x8
//     straight from registers, A = V^T fragments from transposed LDS reads).
//     The product's k order is a permutation of each 16-key step: lane
//     group g = l / 32 supplies keys 4g..4g+3 and 8+4g..8+4g+3, which is what
//     two transposed reads of those four rows deliver.
// Each LDS byte of K and V feeds 32 queries (twice the 16 of a 16x16 tile).
// Software pipeline, per tile k: the matrix cores compute the scores of
// tile k + 1 while the vector ALU turns the scores of tile k into
// probabilities; then O += P V of tile k while the vector ALU masks the
// scores of tile k + 1 and takes their max.  K and V tiles sit
// in two R-stage LDS rings; iteration k reads K(k + 1) and V(k) and
// requests V(k + R - 1) and K(k + R) into the stages of V(k - 1) and K(k),
// so R - 2 tiles of each are in flight while one is used (R = 4: 128 KB
// for head_dim 128, one block of 8 waves per CU; the depth covers the
// latency of tiles that come from HBM).  Tiles arrive by LDS DMA
// (global_load_lds_dwordx4: a wave instruction fills 1 KB = 1024 / (2 D) key
// rows; lane i takes LDS slot i of its row and so reads the chunk that the
// swizzle puts there); one barrier per tile.  A wave skips the arithmetic
// of tiles wholly past its last query (the causal triangle of the chunk).
// Output: a work item with partial index p >= 0 writes the partial
// [m, l, -, -, o[D]] of each of its rows (merged by the combine pass); p < 0 means
// the item covers all of its rows' keys, and it writes the normalised rows
// of O (dtype bf16) directly.
template <int D, int NW, int R>
__global__ __launch_bounds__(64 * NW) void attn_prefill_bf16_kernel(PrefillArgs a, float scale_log2) {
  constexpr int QB = 32 * NW;            // the block's queries (chunk rows)
  constexpr int KT = 64;                 // keys per tile
  constexpr int DCH = D / 8;             // 16-byte chunks per K/V row
  constexpr int TILE = KT * DCH;         // 16-byte chunks per K (or V) tile
  constexpr int RPI = 64 / DCH;          // key rows per 1 KB DMA instruction
  constexpr int NI = KT / RPI / NW;      // DMA instructions per wave per tile (K or V)
  static_assert(NI * NW * RPI == KT && 2 * (R - 1) * NI < 64 && R >= 3, "tile DMA split");
  extern __shared__ u32x4 ring[];        // [R] K tiles, then [R] V tiles
  u32x4* kring = ring;
  u32x4* vring = ring + R * TILE;

  const int per = gridDim.x / 8;
  const int t = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (t >= a.n_work * a.nh) return;
  const int item = t % a.n_work, h = t / a.n_work;
  const int* wk = a.work + 4 * item;
  const int* ch = a.chunks + 4 * wk[0];
  const int slot = ch[0], offset = ch[1], C = ch[2], row0 = ch[3];
  const int q0 = wk[1] * QB, pslot = wk[2];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, ql = lane & 31;
  const bf16* qkv = reinterpret_cast<const bf16*>(a.qkv) + (size_t)row0 * a.ld_qkv;
  const bf16* cache = reinterpret_cast<const bf16*>(a.kv_layer);
  const bf16* kbase = cache + (size_t)slot * a.st.slot + (size_t)h * a.st.head;
  const bf16* vbase = kbase + a.st.kv;

  // This item's keys: tiles [t0, t1) of 0 .. off + min(q0 + QB, C) - 1.
  const int n_keys = offset + min(q0 + QB, C);
  const int kbeg = (wk[3] >> 16) * KT;
  const int kend = min(n_keys, (wk[3] & 0xffff) * KT);
  const int n_tiles = (kend - kbeg + KT - 1) / KT;

  // The lane's query (B operand of S^T): q = ql, d = ks*16 + 8*g.
  const int wq0 = q0 + wave * 32;        // the wave's first query
  const int myq = wq0 + ql;
  const int qpos = offset + myq;
  const int last_key = offset + wq0 + 31;   // keys past it are masked for the whole wave
  u32x4 qf[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(qkv + (size_t)min(myq, C - 1) * a.ld_qkv + h * D + ks * 16 + 8 * g);
    qf[ks] = (myq < C) ? v : u32x4{0u, 0u, 0u, 0u};
  }

  float m_run = -INFINITY, l_run = 0.f;
  floatx16 o_acc[D / 32];                // O^T[d = db*32 + 8*(v/4) + 4*g + v%4][q = ql]
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) o_acc[db][v] = 0.f;

  // Tile DMA: instruction j of wave w fills 1 KB group gi = j * NW + w of a
  // K or V tile.  Key addresses are clamped to the item's last key (finite
  // data; such keys are masked out of the softmax).
  const int lrow = lane / DCH, lslot = lane % DCH;
  int drow[NI];
  size_t doff[NI];                       // element offset of the lane's 16 bytes in key row drow[j]
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    drow[j] = (j * NW + wave) * RPI + lrow;
    doff[j] = (size_t)drow[j] * a.st.pos + kv_swz<D>(lslot, drow[j]) * 8;
  }
  auto issue = [&](const bf16* base, u32x4* stage, int kt) {
    const int k0 = kbeg + kt * KT;
    uint4* dst = reinterpret_cast<uint4*>(stage);
    const bf16* tb = base + (size_t)k0 * a.st.pos;
    if (k0 + KT <= kend) {
#pragma unroll
      for (int j = 0; j < NI; ++j) dma16(tb + doff[j], dst + (j * NW + wave) * 64);
    } else {
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int over = max(k0 + drow[j] - (kend - 1), 0);   // rows past the item's last key re-read it
        dma16(tb + doff[j] - (size_t)over * a.st.pos, dst + (j * NW + wave) * 64);
      }
    }
  };

  // Transposed-read addressing of V^T fragments: within its 16-lane group
  // G = lane / 16, lane i = 4e + q reads 8 bytes of key row 8h + 4g + e
  // (+16 per key step) at columns db*32 + 16*(G % 2) + 4q .. +3.
  // The swizzle depends on the row only through its index mod 16, so each
  // lane's byte offsets are fixed for the whole loop: the 16-key steps and
  // 32-key blocks add constants (the LDS reads' immediate offsets).
  const int G = lane >> 4, li = lane & 15;
  const int tr_e = li >> 2, tr_q = li & 3;
  const int tr_c16 = 2 * (G & 1) + (tr_q >> 1);   // 16-byte chunk within the 32 columns of db
  const int tr_half = (tr_q & 1) * 8;              // byte offset inside the chunk
  int voff[2][D / 32];                             // rows 4g + tr_e (+8) of a V tile
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const int r = 4 * g + tr_e + 8 * hh;
      voff[hh][db] = (r * DCH + kv_swz<D>(4 * db + tr_c16, r)) * 16 + tr_half;
    }
  int koff[D / 16];                                // row ql of a K tile, chunk 2 ks + g
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) koff[ks] = (ql * DCH + kv_swz<D>(2 * ks + g, ql)) * 16;

  // scores of one tile: s[kb][v] = score of key k0 + kb*32 + 8*(v/4) + 4*g + v%4 for query ql
  auto scores = [&](const u32x4* ks_, floatx16* s) {
    const uint32_t kb_ = lds_addr(ks_);
    u32x4 kf[2][D / 16];
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) kf[0][ks] = lds_b128_asm<0>(kb_ + koff[ks]);
    lds_wait(kf[0]);
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) kf[1][ks] = lds_b128_asm<32 * DCH * 16>(kb_ + koff[ks]);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      if (kb == 1) lds_wait(kf[1]);
#pragma unroll
      for (int v = 0; v < 16; ++v) s[kb][v] = 0.f;
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks)
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kf[kb][ks]),
                                                        __builtin_bit_cast(bf16x8_t, qf[ks]), s[kb], 0, 0, 0);
    }
  };

  const int n = n_tiles;
  floatx16 s_cur[2], s_next[2];
  // Requests come in batches, batch j = {V(j + R - 1), K(j + R)} (tiles past
  // the item's end are skipped); iteration k needs K(k + 1) and V(k), both
  // of batch k - R + 1, so the batches after it may stay in flight: the LDS
  // DMA of a wave completes in issue order.  in_flight(k) counts those
  // instructions (V tiles k + 1 .. k + R - 2, K tiles k + 2 .. k + R - 1).
  auto cnt = [&](int lo, int hi) { return max(0, min(hi, n - 1) - lo + 1); };   // tiles in [lo, hi] below n
  auto wait_in_flight = [&](int c) {          // c: instructions that may remain outstanding
    switch (c / NI) {
      case 0: wait_vmcnt<0>(); break;
      case 1: wait_vmcnt<NI>(); break;
      case 2: wait_vmcnt<2 * NI>(); break;
      case 3: wait_vmcnt<3 * NI>(); break;
      case 4: wait_vmcnt<4 * NI>(); break;
      case 5: wait_vmcnt<5 * NI>(); break;
      case 6: wait_vmcnt<6 * NI>(); break;
      case 7: wait_vmcnt<7 * NI>(); break;
      default: wait_vmcnt<8 * NI>(); break;
    }
  };
  static_assert(2 * (R - 1) <= 8 && 8 * NI < 64, "wait cases");
  // prologue: K(0), then batches 1 - R .. -1 = V(0 .. R - 2), K(1 .. R - 1);
  // scores of tile 0 once K(0) has landed
  issue(kbase, kring, 0);
  for (int j = 0; j < R - 1; ++j) {
    if (j < n) issue(vbase, vring + j * TILE, j);
    if (j + 1 < n) issue(kbase, kring + (j + 1) * TILE, j + 1);
  }
  wait_in_flight(NI * (cnt(0, R - 2) + cnt(1, R - 1)));
  lds_read_barrier();
  // ---- mask and running max of one tile's scores.  Keys past the query's
  // position or the item's end are masked (a tile wholly before every query
  // of the wave and inside the item needs no mask).  The running max moves
  // only when a tile's max exceeds it by more than 2^8 (the probabilities of
  // a tile stay below 256: fp32 sums and bf16 products keep their relative
  // precision; O and l are rescaled together).
  auto mask = [&](int kt, floatx16* s) {
    const int k0 = kbeg + kt * KT;
    const bool full = k0 + KT <= kend && k0 + KT - 1 <= offset + wq0;
    if (!full) {
      const int lim = min(qpos, kend - 1) - k0;   // the lane's last unmasked key, tile-relative
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (kb * 32 + 8 * (v >> 2) + 4 * g + (v & 3) > lim) s[kb][v] = -INFINITY;
    }
  };
  auto tile_max = [&](const floatx16* s) {
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmax_nan(mx, s[kb][v]);
    return pair_max(mx) * scale_log2;   // the query's other keys sit in lane l ^ 32
  };
  auto move_max = [&](float mx) {
    if (__ballot(mx > m_run + 8.0f)) {
      const float m_new = fmaxf(m_run, mx);
      // 0 while m_run is -inf; a lane whose keys are all masked so far keeps 1
      const float corr = (m_new == -INFINITY) ? 1.0f : __builtin_amdgcn_exp2f(m_run - m_new);
#pragma unroll
      for (int db = 0; db < D / 32; ++db) o_acc[db] *= corr;
      l_run *= corr;
      m_run = m_new;
    }
  };
  if (kbeg <= last_key) {
    scores(kring, s_cur);
    mask(0, s_cur);
    move_max(tile_max(s_cur));
  }

  // One tile: the scores of tile kt are in sc, masked, with the running max
  // already moved for them; the scores of tile kt + 1 go to sn.  Phase 1:
  // the matrix cores compute S(kt + 1) while the vector ALU turns S(kt) into
  // probabilities; phase 2: O += P V of tile kt while the vector ALU masks
  // S(kt + 1) and takes its max.
  const f32x2_t ones{1.0f, 1.0f};
  auto step = [&](int kt, floatx16* sc, floatx16* sn) {
    const int k0 = kbeg + kt * KT;
    // K(kt + 1) and V(kt) have landed; after the barrier every wave is done
    // with K(kt) and V(kt - 1), whose stages take V(kt + R - 1) and K(kt + R)
    wait_in_flight(NI * (cnt(kt + 1, kt + R - 2) + cnt(kt + 2, kt + R - 1)));
    lds_read_barrier();
    if (kt + R - 1 < n) issue(vbase, vring + ((kt + R - 1) % R) * TILE, kt + R - 1);
    if (kt + R < n) issue(kbase, kring + (kt % R) * TILE, kt + R);
    // every key of the tile lies past the wave's last query: nothing to add
    // (and none of the later tiles adds anything either)
    if (k0 > last_key) return;
    // K fragments of tile kt + 1 (its stage exists in every iteration; past
    // the item's end its stale values are computed on and then masked)
    const uint32_t kn = lds_addr(kring + ((kt + 1) % R) * TILE);
    u32x4 kf[2][D / 16];
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) kf[0][ks] = lds_b128_asm<0>(kn + koff[ks]);
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) kf[1][ks] = lds_b128_asm<32 * DCH * 16>(kn + koff[ks]);

    // ---- phase 1.  Probabilities p = 2^(s * scale * log2 e - m), rounded to
    // bf16 (v_cvt_pk_bf16_f32, nearest even); the lane's share of the row
    // sum adds the rounded pairs (the same values that multiply V).
    const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
    float sum = 0.f;
    u32x4 pw[4];
    auto probs = [&](int kb) {
#pragma unroll
      for (int v = 0; v < 16; ++v) sc[kb][v] = __builtin_amdgcn_exp2f(fmaf(sc[kb][v], scale_log2, -m_use));
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const int vo = h2 * 8;
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          w[i] = pack_bf16x2(sc[kb][vo + 2 * i], sc[kb][vo + 2 * i + 1]);
          sum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w[i]),
                                                __builtin_convertvector(ones, bf16x2_t), sum, false);
        }
        pw[2 * kb + h2] = u32x4{w[0], w[1], w[2], w[3]};
      }
    };
    probs(0);                                  // while the K fragments arrive
    asm volatile("" : "+v"(pw[0]), "+v"(pw[1]), "+v"(sum));
    lds_wait(kf[0]);
    lds_wait(kf[1]);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) sn[kb][v] = 0.f;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        sn[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kf[kb][ks]),
                                                         __builtin_bit_cast(bf16x8_t, qf[ks]), sn[kb], 0, 0, 0);
    probs(1);
    // one matrix product, then three vector instructions, in turn
#pragma unroll
    for (int i = 0; i < D / 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
    }
    // the probabilities are complete here (else the compiler would move
    // their arithmetic next to their use, among the products of phase 2)
#pragma unroll
    for (int i = 0; i < 4; ++i) asm volatile("" : "+v"(pw[i]));
    asm volatile("" : "+v"(sum));
    l_run += sum;

    // ---- phase 2.  O^T += V^T P^T over four 16-key steps; the V fragments
    // of a step are read while the previous step's products run.
    mask(kt + 1, sn);
    const uint32_t vb = lds_addr(vring + (kt % R) * TILE);
    uint32_t va[2][D / 32];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int db = 0; db < D / 32; ++db) va[hh][db] = vb + voff[hh][db];
    constexpr int STEP = 16 * DCH * 16;   // bytes of 16 key rows
    auto vread = [&](u32x2* vr, int ks2) {
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        switch (ks2) {
          case 0: vr[2 * db] = lds_tr16_asm<0>(va[0][db]); vr[2 * db + 1] = lds_tr16_asm<0>(va[1][db]); break;
          case 1: vr[2 * db] = lds_tr16_asm<STEP>(va[0][db]); vr[2 * db + 1] = lds_tr16_asm<STEP>(va[1][db]); break;
          case 2: vr[2 * db] = lds_tr16_asm<2 * STEP>(va[0][db]); vr[2 * db + 1] = lds_tr16_asm<2 * STEP>(va[1][db]); break;
          default: vr[2 * db] = lds_tr16_asm<3 * STEP>(va[0][db]); vr[2 * db + 1] = lds_tr16_asm<3 * STEP>(va[1][db]); break;
        }
      }
    };
    u32x2 vr[2][2 * (D / 32)];
    vread(vr[0], 0);
    float mx = -INFINITY;
#pragma unroll
    for (int ks2 = 0; ks2 < KT / 16; ++ks2) {
      // the next step's V fragments are requested before this step's products
      if (ks2 + 1 < KT / 16) {
        vread(vr[(ks2 + 1) & 1], ks2 + 1);
        lds_wait_but<2 * (D / 32)>(vr[ks2 & 1]);   // the next step's reads may stay in flight
      } else {
        lds_wait(vr[ks2 & 1]);
      }
      const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, pw[ks2]);
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        const u32x2* vc = vr[ks2 & 1];
        const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, u32x4{vc[2 * db].x, vc[2 * db].y, vc[2 * db + 1].x,
                                                               vc[2 * db + 1].y});
        o_acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, o_acc[db], 0, 0, 0);
      }
      // a quarter of the next tile's max between the products
#pragma unroll
      for (int v = 4 * ks2; v < 4 * ks2 + 4; ++v) mx = fmax_nan(fmax_nan(mx, sn[0][v]), sn[1][v]);
    }
    move_max(pair_max(mx) * scale_log2);
  };

  // two tiles per trip, the score buffers alternating
  for (int kt = 0; kt < n; kt += 2) {
    step(kt, s_cur, s_next);
    if (kt + 1 < n) step(kt + 1, s_next, s_cur);
  }
  l_run = pair_sum(l_run);               // both halves of the query's keys

  // ---- epilogue.  The lane holds column block d of query ql; rows of O (or
  // of the partial) are contiguous in memory, so each wave first transposes
  // its 32 x D tile through LDS (16-byte chunks XOR-swizzled by row), then
  // writes whole rows, 16 bytes per lane.  The K/V rings are free once every
  // wave has passed the barrier.
  lds_read_barrier();
  const int nrows = min(32, C - wq0);     // the wave's rows inside the chunk
  if (pslot < 0) {
    // the item saw every key of its rows: normalised O in the output dtype
    constexpr int RC = D / 8;             // 16-byte chunks per bf16 row
    char* T = reinterpret_cast<char*>(ring) + wave * 32 * D * 2;
    const float inv = 1.0f / l_run;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        const uint2 w{pack_bf16x2(o_acc[db][4 * v4] * inv, o_acc[db][4 * v4 + 1] * inv),
                      pack_bf16x2(o_acc[db][4 * v4 + 2] * inv, o_acc[db][4 * v4 + 3] * inv)};
        const int c = db * 4 + v4;        // 16-byte chunk of columns db*32 + 8*v4 .. +7
        *reinterpret_cast<uint2*>(T + ql * D * 2 + (c ^ (ql & (RC - 1))) * 16 + g * 8) = w;
      }
    __builtin_amdgcn_s_waitcnt(0xc07f);   // this wave's LDS writes done (lgkmcnt 0)
#pragma unroll
    for (int i = 0; i < 32 * RC / 64; ++i) {
      const int idx = i * 64 + lane, r = idx / RC, c = idx % RC;
      const u32x4 v = *reinterpret_cast<const u32x4*>(T + r * D * 2 + (c ^ (r & (RC - 1))) * 16);
      if (r < nrows)
        *reinterpret_cast<u32x4*>(reinterpret_cast<bf16*>(a.out) + (size_t)(row0 + wq0 + r) * a.ld_out + h * D +
                                  c * 8) = v;
    }
    return;
  }
  // partial of each row: [m, l, -, -, o[D]]
  constexpr int RC = D / 4;               // 16-byte chunks per fp32 row
  float* T = reinterpret_cast<float*>(ring) + wave * 32 * D;
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4) {
      const int c = db * 8 + 2 * v4 + g;  // 16-byte chunk of columns db*32 + 8*v4 + 4*g .. +3
      *reinterpret_cast<floatx4*>(T + ql * D + (c ^ (ql & 15)) * 4) =
          floatx4{o_acc[db][4 * v4], o_acc[db][4 * v4 + 1], o_acc[db][4 * v4 + 2], o_acc[db][4 * v4 + 3]};
    }
  float* prow = a.part + (size_t)(pslot * QB + wave * 32) * a.nh * (D + PART_O) + (size_t)h * (D + PART_O);
  const size_t rstride = (size_t)a.nh * (D + PART_O);
  if (g == 0 && ql < nrows) {
    prow[ql * rstride] = m_run;
    prow[ql * rstride + 1] = l_run;
  }
  __builtin_amdgcn_s_waitcnt(0xc07f);     // this wave's LDS writes done (lgkmcnt 0)
#pragma unroll
  for (int i = 0; i < 32 * RC / 64; ++i) {
    const int idx = i * 64 + lane, r = idx / RC, c = idx % RC;
    const floatx4 v = *reinterpret_cast<const floatx4*>(T + r * D + (c ^ (r & 15)) * 4);
    if (r < nrows) *reinterpret_cast<floatx4*>(prow + r * rstride + PART_O + c * 4) = v;
  }
}

template <int D, int NW, int R>
static hipError_t run_prefill(const PrefillArgs& a, unsigned grid, float scale_log2, hipStream_t s) {
  const size_t lds_bytes = (size_t)2 * R * 64 * (D / 8) * 16;   // R K + R V tile stages
  static std::atomic<uint64_t> lds_set{0};   // devices on which this instance's LDS limit is raised
  hipError_t e = ensure_dynamic_lds((const void*)attn_prefill_bf16_kernel<D, NW, R>, (int)lds_bytes, lds_set);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_prefill_bf16_kernel<D, NW, R>), dim3(grid), dim3(64 * NW), lds_bytes, s, a, scale_log2);
  return hipGetLastError();
}

hipError_t launch_attn_prefill(int dtype, const PrefillArgs& a, hipStream_t s) {
  if (a.n_work <= 0) return hipSuccess;
  if (dtype != 1) return hipErrorInvalidValue;
  const float scale_log2 = LOG2E / sqrtf((float)a.hd);
  const unsigned grid = (unsigned)(((size_t)a.n_work * a.nh + 7) / 8 * 8);
  // 256-row q-blocks: 8 waves, 4-deep K and V rings (128 KB for head_dim 128,
  // one block per CU); 128-row q-blocks: 4 waves, 3-deep rings (96 KB)
  if (a.qblock == PREFILL_QBLOCK_SMALL) {
    if (a.hd == 128) return run_prefill<128, PREFILL_QBLOCK_SMALL / 32, 3>(a, grid, scale_log2, s);
    return run_prefill<64, PREFILL_QBLOCK_SMALL / 32, 3>(a, grid, scale_log2, s);
  }
  if (a.qblock != PREFILL_QBLOCK) return hipErrorInvalidValue;
  if (a.hd == 128) return run_prefill<128, PREFILL_QBLOCK / 32, 4>(a, grid, scale_log2, s);
  return run_prefill<64, PREFILL_QBLOCK / 32, 4>(a, grid, scale_log2, s);
}

}  // namespace sarathi
