// Host runtime of libsarathi: argument validation (entirely on the host,
// before anything is enqueued), workspace layout, batch metadata upload and
// the launch sequence of one decoder layer over a decode-maximal hybrid batch
// (Sec. 4.3: one matmul per linear op over all rows; chunk attention and
// decode attention separately).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "host_error.h"
#include "kernels.h"
#include "runtime_internal.h"
#include "sarathi.h"

using namespace sarathi;

struct sarathi_kv {
  sarathi_model_cfg cfg;
  int n_slots;
  int max_seq_len;
  void* mem;
  size_t bytes;
  KVStrides st;
};

namespace {
thread_local std::string g_err;
}  // namespace

int sarathi::fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

namespace {

int hip_fail(hipError_t e, const char* what) {
  return fail(SARATHI_EHIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int SPLIT_KEYS = 512;   // keys per decode-attention work item
constexpr int PRE_SPLIT = 256;    // smallest key split of a chunk-attention work item
constexpr int QBLOCK = PREFILL_QBLOCK;   // chunk rows per chunk-attention work item (the larger size)
constexpr int PARTS_ROWS = 512;   // split-K partials are sized for batches up to this many rows (larger
                                  // batches fill the GPU without splitting; with less room fewer splits run)

size_t esize(const sarathi_model_cfg* c) { return c->dtype == SARATHI_BF16 ? 2 : 4; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

int check_cfg(const sarathi_model_cfg* c) {
  if (!c) return fail(SARATHI_EINVAL, "cfg is NULL");
  if (c->dtype != SARATHI_F32 && c->dtype != SARATHI_BF16)
    return fail(SARATHI_EUNSUPPORTED, "dtype %d not supported (F32 or BF16)", c->dtype);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(SARATHI_EUNSUPPORTED, "head_dim %d not supported (64 or 128)", c->head_dim);
  if (c->hidden <= 0 || c->hidden % 8) return fail(SARATHI_EUNSUPPORTED, "hidden %d must be a positive multiple of 8", c->hidden);
  if (c->ffn <= 0 || c->ffn % 8) return fail(SARATHI_EUNSUPPORTED, "ffn %d must be a positive multiple of 8", c->ffn);
  // the norm kernels keep a row in registers: 12 x 256 x 8 (bf16) or x 4 (fp32) elements
  const int max_hidden = c->dtype == SARATHI_BF16 ? 24576 : 12288;
  if (c->hidden > max_hidden) return fail(SARATHI_EUNSUPPORTED, "hidden %d > %d", c->hidden, max_hidden);
  if (c->n_heads <= 0 || c->n_heads > 65535) return fail(SARATHI_EUNSUPPORTED, "n_heads %d out of range", c->n_heads);
  if (c->n_layers <= 0) return fail(SARATHI_EINVAL, "n_layers %d must be positive", c->n_layers);
  if (c->norm != SARATHI_NORM_RMS && c->norm != SARATHI_NORM_LAYER) return fail(SARATHI_EUNSUPPORTED, "norm %d", c->norm);
  if (c->act != SARATHI_ACT_SWIGLU && c->act != SARATHI_ACT_GELU) return fail(SARATHI_EUNSUPPORTED, "act %d", c->act);
  if (c->rope != 0 && c->rope != 1) return fail(SARATHI_EINVAL, "rope must be 0 or 1");
  if (c->rope && !(c->rope_base > 1.0f)) return fail(SARATHI_EINVAL, "rope_base must be > 1");
  if (!(c->eps > 0.0f)) return fail(SARATHI_EINVAL, "eps must be > 0");
  return SARATHI_OK;
}

bool same_cfg(const sarathi_model_cfg* a, const sarathi_model_cfg* b) {
  return a->hidden == b->hidden && a->n_heads == b->n_heads && a->head_dim == b->head_dim && a->ffn == b->ffn &&
         a->n_layers == b->n_layers && a->norm == b->norm && a->act == b->act && a->rope == b->rope &&
         a->rope_base == b->rope_base && a->eps == b->eps && a->dtype == b->dtype;
}

struct Layout {
  size_t a, qkv, o, hres, m, parts, part, meta, ping0, ping1, total;
};

// Workspace regions for batches of up to T rows in up to n_chunks prompt
// chunks (>= 1) with a KV of S positions per slot.
Layout make_layout(const sarathi_model_cfg* c, int T, int n_chunks, int S) {
  Layout L{};
  const size_t es = esize(c);
  const size_t H = c->hidden, F = c->ffn, QD = (size_t)c->n_heads * c->head_dim;
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t at = off; off = align256(off + bytes); return at; };
  if (n_chunks < 1) n_chunks = 1;
  L.a = take(T * H * es);
  L.qkv = take(T * 3 * QD * es);
  L.o = take(T * QD * es);
  L.hres = take(T * H * 4);
  L.m = take(T * F * es);
  L.parts = take((size_t)MAX_SPLIT * std::min(T, PARTS_ROWS) * H * 4);
  // query blocks of QBLOCK rows (each chunk starts a new block), at most one
  // key range per PRE_SPLIT keys each
  const size_t max_pre = ((size_t)(T + QBLOCK - 1) / QBLOCK + n_chunks - 1) * ((S + PRE_SPLIT - 1) / PRE_SPLIT);
  const size_t max_dec = (size_t)T * ((S + SPLIT_KEYS - 1) / SPLIT_KEYS);
  L.part = take((max_pre * QBLOCK + max_dec) * c->n_heads * (c->head_dim + PART_O) * 4);
  L.meta = take(((size_t)T * 5 + (size_t)n_chunks * 4 + max_pre * 4 + max_dec) * 4);
  L.ping0 = take(T * H * es);
  L.ping1 = take(T * H * es);
  L.total = off;
  return L;
}

// A batch of any number of prompt chunks plus decodes (the hybrid batch of
// the paper has at most one chunk).
struct ChunkDesc {
  int slot, offset, len;
};
struct BatchDesc {
  std::vector<ChunkDesc> chunks;
  int B = 0;
  const int* dslots = nullptr;
  const int* dctx = nullptr;
  int rows() const {
    int r = B;
    for (const ChunkDesc& c : chunks) r += c.len;
    return r;
  }
};

int from_hybrid(const sarathi_hybrid_batch* b, BatchDesc* out) {
  if (!b) return fail(SARATHI_EINVAL, "batch is NULL");
  if (b->chunk_len < 0) return fail(SARATHI_ERANGE, "chunk_len %d < 0", b->chunk_len);
  if (b->n_decodes < 0) return fail(SARATHI_EINVAL, "n_decodes %d < 0", b->n_decodes);
  out->chunks.clear();
  if (b->chunk_len > 0) out->chunks.push_back({b->prefill_slot, b->chunk_offset, b->chunk_len});
  out->B = b->n_decodes;
  out->dslots = b->decode_slots;
  out->dctx = b->decode_ctx_lens;
  return SARATHI_OK;
}

int from_mixed(const sarathi_mixed_batch* b, BatchDesc* out) {
  if (!b) return fail(SARATHI_EINVAL, "batch is NULL");
  if (b->n_chunks < 0 || b->n_chunks > (1 << 16)) return fail(SARATHI_EINVAL, "n_chunks %d out of range", b->n_chunks);
  if (b->n_decodes < 0) return fail(SARATHI_EINVAL, "n_decodes %d < 0", b->n_decodes);
  if (b->n_chunks > 0 && (!b->chunk_slots || !b->chunk_offsets || !b->chunk_lens))
    return fail(SARATHI_EINVAL, "chunk arrays are NULL");
  out->chunks.clear();
  for (int i = 0; i < b->n_chunks; ++i) {
    if (b->chunk_lens[i] < 1) return fail(SARATHI_ERANGE, "chunk_lens[%d] = %d < 1", i, b->chunk_lens[i]);
    out->chunks.push_back({b->chunk_slots[i], b->chunk_offsets[i], b->chunk_lens[i]});
  }
  out->B = b->n_decodes;
  out->dslots = b->decode_slots;
  out->dctx = b->decode_ctx_lens;
  return SARATHI_OK;
}

// Host-side description of the batch and its device metadata.
struct Plan {
  int C, B, T, row_base, n_pre, n_dec, n_chunks, pre_tiles;
  int qblock;      // chunk rows per chunk-attention q-block (PREFILL_QBLOCK or PREFILL_QBLOCK_SMALL)
  int pre_slots;   // partial q-block slots of the chunk items (items covering all keys of their rows write O)
  int comb_row0;   // first row whose attention output the combine pass writes
  // row_slot[T] row_pos[T] comb[3T] chunk table [n_chunks][slot, offset, len, first row]
  // pre_work[n_pre][chunk, q_block, partial slot, (first tile << 16) | end tile] dec_work[n_dec]
  std::vector<int> meta;
  size_t o_slot, o_pos, o_comb, o_chunks, o_pre, o_dec;   // int offsets into meta
};

int check_batch(const sarathi_model_cfg* cfg, const sarathi_kv* kv, const BatchDesc& b) {
  const int B = b.B, S = kv->max_seq_len;
  long rows = B;
  for (const ChunkDesc& c : b.chunks) rows += c.len;
  if (rows == 0) return fail(SARATHI_EINVAL, "empty batch (no chunk rows and no decodes)");
  if (rows > (1 << 19)) return fail(SARATHI_EINVAL, "batch of %ld rows too large", rows);
  std::vector<char> used(kv->n_slots, 0);
  for (size_t i = 0; i < b.chunks.size(); ++i) {
    const ChunkDesc& c = b.chunks[i];
    if (c.slot < 0 || c.slot >= kv->n_slots)
      return fail(SARATHI_EINVAL, "chunk %zu: slot %d outside [0, %d)", i, c.slot, kv->n_slots);
    if (used[c.slot]) return fail(SARATHI_EINVAL, "slot %d appears twice in the batch", c.slot);
    used[c.slot] = 1;
    if (c.offset < 0) return fail(SARATHI_ERANGE, "chunk %zu: offset %d < 0", i, c.offset);
    if ((long)c.offset + c.len > S)
      return fail(SARATHI_ERANGE, "chunk %zu: offset %d + length %d > max_seq_len %d", i, c.offset, c.len, S);
  }
  if (B > 0) {
    if (!b.dslots || !b.dctx) return fail(SARATHI_EINVAL, "decode arrays are NULL");
    for (int i = 0; i < B; ++i) {
      const int s = b.dslots[i], ctx = b.dctx[i];
      if (s < 0 || s >= kv->n_slots) return fail(SARATHI_EINVAL, "decode_slots[%d] = %d outside [0, %d)", i, s, kv->n_slots);
      if (used[s]) return fail(SARATHI_EINVAL, "slot %d appears twice in the batch", s);
      used[s] = 1;
      if (ctx < 0) return fail(SARATHI_ERANGE, "decode_ctx_lens[%d] = %d < 0", i, ctx);
      if ((long)ctx + 1 > S) return fail(SARATHI_ERANGE, "decode_ctx_lens[%d] + 1 = %d > max_seq_len %d", i, ctx + 1, S);
    }
  }
  (void)cfg;
  return SARATHI_OK;
}

Plan make_plan(const sarathi_model_cfg* cfg, const BatchDesc& b) {
  Plan p;
  p.B = b.B;
  p.C = b.rows() - b.B;
  p.T = p.C + p.B;
  p.n_chunks = (int)b.chunks.size();
  // bf16: chunk rows go to the MFMA chunk-attention kernel (work item = one
  // chunk's query block x key split), decodes to row attention (work
  // item = row x key split).  fp32: every row goes to row attention (a chunk
  // row at position p is attention over keys 0..p, like a decode with ctx = p).
  p.row_base = (cfg->dtype == SARATHI_BF16) ? p.C : 0;
  p.pre_tiles = PRE_SPLIT / 64;
  p.qblock = QBLOCK;
  p.pre_slots = 0;
  std::vector<int> slot(p.T), pos(p.T), comb(3 * p.T), tab, pre, dec;
  int r0 = 0;
  for (const ChunkDesc& c : b.chunks) {
    tab.insert(tab.end(), {c.slot, c.offset, c.len, r0});
    for (int r = 0; r < c.len; ++r) { slot[r0 + r] = c.slot; pos[r0 + r] = c.offset + r; }
    r0 += c.len;
  }
  for (int i = 0; i < p.B; ++i) { slot[p.C + i] = b.dslots[i]; pos[p.C + i] = b.dctx[i]; }
  if (p.row_base > 0) {
    // Partial slots run q-block by q-block (a row's splits are consecutive,
    // qblock partial rows apart); the work items run split by split so that
    // the query blocks that read the same keys are neighbours (and share an
    // XCD's L2, see the chunk-attention kernel).
    // Key ranges: each q-block's keys, in 64-key tiles, are cut into ns
    // near-equal ranges of at most tau tiles (tau >= PRE_SPLIT / 64).  tau
    // minimises rounds of blocks (one per CU) x (largest range + ~4 tiles of
    // fixed cost per block), fitted to measurements of the LLaMA-33B and
    // GPT-3 chunk shapes; ties go to the larger tau (fewer partials).
    // Two q-block sizes are priced the same way: a 128-row block (4 waves,
    // one per SIMD) takes ~0.82x the time of a 256-row block per key tile
    // (measured on the LLaMA-13B, LLaMA-33B and GPT-3 chunk shapes), and
    // wins when the chunk is short or the heads few (fewer idle waves and a
    // smaller set-up and output per block).
    std::vector<int> qtiles;   // tiles of every q-block, chunk by chunk
    int tau = PRE_SPLIT / 64;
    double best = 1e300;
    p.qblock = QBLOCK;
    for (const int qbs : {QBLOCK, PREFILL_QBLOCK_SMALL}) {
      const double per_tile = qbs == QBLOCK ? 1.0 : 0.82;
      std::vector<int> qt;
      int t_max = 1;
      for (const ChunkDesc& c : b.chunks)
        for (int qb = 0; qb * qbs < c.len; ++qb) {
          const int n_keys = c.offset + std::min((qb + 1) * qbs, c.len);
          qt.push_back((n_keys + 63) / 64);
          t_max = std::max(t_max, qt.back());
        }
      const int tau_min = PRE_SPLIT / 64;
      for (int cand = tau_min; cand <= std::max(t_max, tau_min); cand += std::max(1, cand / 4)) {
        long blocks = 0;
        int longest = 0;
        for (int t : qt) {
          const int ns = (t + cand - 1) / cand;
          blocks += ns;
          longest = std::max(longest, (t + ns - 1) / ns);
        }
        blocks *= cfg->n_heads;
        const double cost = (double)((blocks + 255) / 256) * (longest + 4) * per_tile;
        if (cost <= best) {
          best = cost;
          tau = cand;
          p.qblock = qbs;
          qtiles = qt;
        }
      }
    }
    p.pre_tiles = tau;
    r0 = 0;
    int slot_base = 0, qi = 0;
    // a q-block whose keys form one range is one item that writes its rows
    // of O directly (partial slot -1, no combine); split q-blocks get
    // consecutive partial slots
    for (int ci = 0; ci < p.n_chunks; ++ci) {
      const ChunkDesc& c = b.chunks[ci];
      const int qbs = p.qblock, nqb = (c.len + qbs - 1) / qbs;
      std::vector<int> ns(nqb), first(nqb), nt(nqb);
      int max_ns = 0;
      for (int qb = 0; qb < nqb; ++qb) {
        nt[qb] = qtiles[qi++];
        ns[qb] = (nt[qb] + tau - 1) / tau;
        first[qb] = ns[qb] > 1 ? slot_base : -1;
        if (ns[qb] > 1) slot_base += ns[qb];
        max_ns = std::max(max_ns, ns[qb]);
        for (int r = qb * qbs; r < std::min((qb + 1) * qbs, c.len); ++r) {
          comb[3 * (r0 + r)] = ns[qb] > 1 ? first[qb] * qbs + (r - qb * qbs) : 0;
          comb[3 * (r0 + r) + 1] = ns[qb] > 1 ? ns[qb] : 0;
          comb[3 * (r0 + r) + 2] = qbs;
        }
      }
      for (int s = 0; s < max_ns; ++s)
        for (int qb = 0; qb < nqb; ++qb)
          if (s < ns[qb]) {
            const int t0 = (int)((long)nt[qb] * s / ns[qb]), t1 = (int)((long)nt[qb] * (s + 1) / ns[qb]);
            pre.insert(pre.end(), {ci, qb, ns[qb] > 1 ? first[qb] + s : -1, (t0 << 16) | t1});
          }
      r0 += c.len;
    }
    p.pre_slots = slot_base;
  }
  const int pre_rows = p.pre_slots * p.qblock;
  // Row-attention items run in the order of the rows' KV slots (each row's
  // splits together), so the blocks in flight stream the cache in address
  // order (measured ~2% faster than a random slot order).
  std::vector<int> order;
  for (int r = p.row_base; r < p.T; ++r) order.push_back(r);
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return slot[x] < slot[y]; });
  for (int r : order) {
    const int ns = (pos[r] + 1 + SPLIT_KEYS - 1) / SPLIT_KEYS;
    comb[3 * r] = pre_rows + (int)dec.size();
    comb[3 * r + 1] = ns;
    comb[3 * r + 2] = 1;
    for (int s = 0; s < ns; ++s) dec.push_back(((r - p.row_base) << 12) | s);
  }
  p.n_pre = (int)pre.size() / 4;
  p.n_dec = (int)dec.size();
  p.comb_row0 = p.T;
  for (int r = 0; r < p.T; ++r)
    if (comb[3 * r + 1] > 0) {
      p.comb_row0 = r;
      break;
    }
  p.meta.reserve(5 * p.T + tab.size() + pre.size() + dec.size());
  p.o_slot = 0; p.meta.insert(p.meta.end(), slot.begin(), slot.end());
  p.o_pos = p.meta.size(); p.meta.insert(p.meta.end(), pos.begin(), pos.end());
  p.o_comb = p.meta.size(); p.meta.insert(p.meta.end(), comb.begin(), comb.end());
  p.o_chunks = p.meta.size(); p.meta.insert(p.meta.end(), tab.begin(), tab.end());
  p.o_pre = p.meta.size(); p.meta.insert(p.meta.end(), pre.begin(), pre.end());
  p.o_dec = p.meta.size(); p.meta.insert(p.meta.end(), dec.begin(), dec.end());
  return p;
}

int check_weights(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w, int layer) {
  if (!w) return fail(SARATHI_EINVAL, "weights are NULL");
  const void* need[] = {w->norm1_g, w->w_qkv, w->w_o, w->norm2_g, w->w_up, w->w_down};
  for (const void* p : need)
    if (!p) return fail(SARATHI_EINVAL, "layer %d: a weight pointer is NULL", layer);
  for (const void* p : need)
    if (!aligned16(p)) return fail(SARATHI_EINVAL, "layer %d: weights must be 16-byte aligned", layer);
  if (cfg->norm == SARATHI_NORM_LAYER) {
    if (!w->norm1_b || !w->norm2_b) return fail(SARATHI_EINVAL, "layer %d: LayerNorm biases are NULL", layer);
    if (!aligned16(w->norm1_b) || !aligned16(w->norm2_b))
      return fail(SARATHI_EINVAL, "layer %d: weights must be 16-byte aligned", layer);
  }
  return SARATHI_OK;
}

// ---- stage timing: a pool of HIP events recorded at stage boundaries.
constexpr int EV_PER_CALL = SARATHI_N_STAGES + 1;
struct Profiler {
  std::mutex mu;
  bool on = false;
  int max_calls = 0;
  int calls = 0;
  std::vector<hipEvent_t> pool;
};
Profiler g_prof;

// Events of the next layer call (nullptr when not recording).
hipEvent_t* prof_claim() {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (!g_prof.on || g_prof.calls >= g_prof.max_calls) return nullptr;
  return g_prof.pool.data() + EV_PER_CALL * (g_prof.calls++);
}

struct Ctx {
  const sarathi_model_cfg* cfg;
  sarathi_kv* kv;
  const Plan* plan;
  Layout L;
  char* ws;
  hipStream_t s;
};

// Metadata chunk `i` (META_CHUNK ints each).
void meta_chunk(const Plan& p, size_t i, MetaChunk* chunk) {
  const size_t at = i * META_CHUNK;
  chunk->count = (int)std::min<size_t>(META_CHUNK, p.meta.size() - at);
  std::memcpy(chunk->values, p.meta.data() + at, chunk->count * sizeof(int));
}

// Uploads every metadata chunk but the first, which the first norm_1 launch
// of the call carries (nothing the chunks feed runs before that norm ends).
int upload_meta_rest(const Ctx& c) {
  int* dst = reinterpret_cast<int*>(c.ws + c.L.meta);
  const size_t n = (c.plan->meta.size() + META_CHUNK - 1) / META_CHUNK;
  for (size_t i = 1; i < n; ++i) {
    MetaChunk chunk;
    meta_chunk(*c.plan, i, &chunk);
    hipError_t e = launch_meta_write(chunk, dst + i * META_CHUNK, c.s);
    if (e != hipSuccess) return hip_fail(e, "metadata upload");
  }
  return SARATHI_OK;
}

// One decoder layer; metadata already on the device.
// One layer on the planned batch.  norm1_ready: norm_1 of this layer already
// sits in the workspace (folded into the previous layer's last reduction);
// next: the layer after this one in a model step (null for the last layer or
// a single-layer call), whose norm_1 is folded into this layer's ffn_ln2
// split-K reduction when that op runs split (*next_norm1_done says so).
int layer_body(const Ctx& c, const sarathi_layer_weights* w, int layer, const void* x_in, void* x_out,
               bool carry_meta, bool norm1_ready = false, const sarathi_layer_weights* next = nullptr,
               bool* next_norm1_done = nullptr) {
  const sarathi_model_cfg* cfg = c.cfg;
  const Plan& P = *c.plan;
  const int T = P.T, H = cfg->hidden, nh = cfg->n_heads, hd = cfg->head_dim, F = cfg->ffn;
  const int QD = nh * hd;
  const int dt = cfg->dtype;
  const bool ln = cfg->norm == SARATHI_NORM_LAYER;
  char* ws = c.ws;
  const int* meta = reinterpret_cast<const int*>(ws + c.L.meta);
  float* hres = reinterpret_cast<float*>(ws + c.L.hres);
  float* parts = reinterpret_cast<float*>(ws + c.L.parts);
  const size_t parts_cap = (size_t)MAX_SPLIT * std::min(T, PARTS_ROWS) * H;
  char* kv_layer = static_cast<char*>(c.kv->mem) + (size_t)layer * c.kv->st.layer * esize(cfg);
  hipError_t e;
  hipEvent_t* ev = prof_claim();
  int stage = 0;
  auto mark = [&]() -> hipError_t { return ev ? hipEventRecord(ev[stage++], c.s) : hipSuccess; };
#define SARATHI_MARK()                                          \
  do {                                                          \
    hipError_t me = mark();                                     \
    if (me != hipSuccess) return hip_fail(me, "stage event");   \
  } while (0)

  // norm_1
  SARATHI_MARK();
  if (norm1_ready) {
    e = hipSuccess;
  } else if (carry_meta) {
    MetaChunk first;
    meta_chunk(P, 0, &first);
    e = launch_norm(dt, false, ln, x_in, w->norm1_g, w->norm1_b, ws + c.L.a, T, H, cfg->eps, c.s, &first,
                    reinterpret_cast<int*>(ws + c.L.meta));
  } else {
    e = launch_norm(dt, false, ln, x_in, w->norm1_g, w->norm1_b, ws + c.L.a, T, H, cfg->eps, c.s);
  }
  if (e != hipSuccess) return hip_fail(e, "norm_1");

  // preproj over all rows, with the rotary embedding and the in-place KV
  // append in its epilogue (bf16)
  SARATHI_MARK();
  RopeArgs ra{};
  ra.qkv = ws + c.L.qkv; ra.T = T; ra.nh = nh; ra.hd = hd; ra.rope = cfg->rope; ra.base = cfg->rope_base;
  ra.row_slot = meta + P.o_slot; ra.row_pos = meta + P.o_pos; ra.kv_layer = kv_layer; ra.st = c.kv->st;
  bool rope_done = false;
  LinearArgs q{};
  q.kind = LIN_PLAIN; q.M = T; q.N = 3 * QD; q.K = H; q.x = ws + c.L.a; q.w = w->w_qkv; q.out = ws + c.L.qkv;
  q.rope = &ra; q.rope_done = &rope_done;
  e = launch_linear(dt, q, c.s);
  if (e != hipSuccess) return hip_fail(e, "preproj");

  // rotary embedding + in-place KV append (unless fused above)
  SARATHI_MARK();
  if (!rope_done) {
    e = launch_rope_append(dt, ra, c.s);
    if (e != hipSuccess) return hip_fail(e, "rope/kv append");
  }

  // attention: the chunk and the decodes separately, then one combine pass
  SARATHI_MARK();
  float* part = reinterpret_cast<float*>(ws + c.L.part);   // attention partials
  if (P.n_pre > 0) {
    PrefillArgs pa{};
    pa.qkv = ws + c.L.qkv; pa.ld_qkv = 3 * QD; pa.kv_layer = kv_layer; pa.st = c.kv->st;
    pa.chunks = meta + P.o_chunks; pa.nh = nh; pa.hd = hd;
    pa.work = meta + P.o_pre; pa.n_work = P.n_pre; pa.qblock = P.qblock; pa.part = part;
    pa.out = ws + c.L.o; pa.ld_out = QD;
    e = launch_attn_prefill(dt, pa, c.s);
    if (e != hipSuccess) return hip_fail(e, "chunk attention");
  }
  SARATHI_MARK();
  if (P.n_dec > 0) {
    RowAttnArgs da{};
    da.qkv = ws + c.L.qkv; da.ld_qkv = 3 * QD; da.kv_layer = kv_layer; da.st = c.kv->st;
    da.row_slot = meta + P.o_slot; da.row_pos = meta + P.o_pos; da.work = meta + P.o_dec;
    da.row_base = P.row_base; da.n_work = P.n_dec; da.split_keys = SPLIT_KEYS; da.nh = nh; da.hd = hd;
    da.part = part; da.part_base = P.pre_slots * P.qblock;
    e = launch_attn_rows(dt, da, c.s);
    if (e != hipSuccess) return hip_fail(e, "decode attention");
  }
  SARATHI_MARK();
  CombineArgs ca{};
  ca.part = part; ca.comb = meta + P.o_comb; ca.row0 = P.comb_row0; ca.n_rows = T; ca.nh = nh; ca.hd = hd;
  ca.out = ws + c.L.o;
  ca.ld_out = QD;
  e = launch_attn_combine(dt, ca, c.s);
  if (e != hipSuccess) return hip_fail(e, "attention combine");

  // postproj + residual -> hres (fp32), with norm_2 folded into its split-K
  // reduction pass when it runs split over K
  SARATHI_MARK();
  NormArgs n2{w->norm2_g, w->norm2_b, ws + c.L.a, cfg->eps, ln};
  bool norm2_done = false;
  LinearArgs po{};
  po.kind = LIN_RESID; po.M = T; po.N = H; po.K = QD; po.x = ws + c.L.o; po.w = w->w_o; po.resid = x_in;
  po.out = hres; po.parts = parts; po.parts_cap = parts_cap;
  po.norm = &n2; po.norm_done = &norm2_done;
  e = launch_linear(dt, po, c.s);
  if (e != hipSuccess) return hip_fail(e, "postproj");

  // norm_2 (unless folded above)
  SARATHI_MARK();
  if (!norm2_done) {
    e = launch_norm(dt, true, ln, hres, w->norm2_g, w->norm2_b, ws + c.L.a, T, H, cfg->eps, c.s);
    if (e != hipSuccess) return hip_fail(e, "norm_2");
  }

  // ffn_ln1 + activation
  SARATHI_MARK();
  LinearArgs up{};
  up.kind = cfg->act == SARATHI_ACT_SWIGLU ? LIN_SWIGLU : LIN_GELU;
  up.M = T; up.N = F; up.K = H; up.x = ws + c.L.a; up.w = w->w_up; up.out = ws + c.L.m;
  e = launch_linear(dt, up, c.s);
  if (e != hipSuccess) return hip_fail(e, "ffn_ln1");

  // ffn_ln2 + residual -> x_out
  SARATHI_MARK();
  LinearArgs dn{};
  dn.kind = LIN_RESID_F32IN; dn.M = T; dn.N = H; dn.K = F; dn.x = ws + c.L.m; dn.w = w->w_down; dn.resid = hres;
  dn.out = x_out; dn.parts = parts; dn.parts_cap = parts_cap;
  NormArgs n1{};
  if (next != nullptr && next_norm1_done != nullptr) {
    n1 = NormArgs{next->norm1_g, next->norm1_b, ws + c.L.a, cfg->eps, ln};
    dn.norm = &n1; dn.norm_done = next_norm1_done;   // 'a' is free: ffn_ln1 has read it
  }
  e = launch_linear(dt, dn, c.s);
  if (e != hipSuccess) return hip_fail(e, "ffn_ln2");
  SARATHI_MARK();
#undef SARATHI_MARK
  return SARATHI_OK;
}

// Every check of a call that does not involve the workspace.
int check_call(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w, int n_w, const sarathi_kv* kv,
               const BatchDesc& batch, const void* x_in, const void* x_out) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!kv) return fail(SARATHI_EINVAL, "kv is NULL");
  if (!same_cfg(cfg, &kv->cfg)) return fail(SARATHI_EINVAL, "cfg differs from the cfg the KV cache was bound with");
  rc = check_batch(cfg, kv, batch);
  if (rc) return rc;
  for (int i = 0; i < n_w; ++i) {
    rc = check_weights(cfg, w + i, i);
    if (rc) return rc;
  }
  if (!x_in || !x_out) return fail(SARATHI_EINVAL, "x_in / x_out is NULL");
  if (x_in == x_out) return fail(SARATHI_EINVAL, "x_in and x_out alias");
  if (!aligned16(x_in) || !aligned16(x_out)) return fail(SARATHI_EINVAL, "x_in, x_out and ws must be 16-byte aligned");
  return SARATHI_OK;
}

int prepare(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w, int n_w, sarathi_kv* kv,
            const BatchDesc& batch, const void* x_in, void* x_out, void* ws, size_t ws_bytes,
            Plan* plan, Layout* L) {
  int rc = check_call(cfg, w, n_w, kv, batch, x_in, x_out);
  if (rc) return rc;
  if (!ws) return fail(SARATHI_EINVAL, "workspace is NULL");
  if (!aligned16(ws)) return fail(SARATHI_EINVAL, "x_in, x_out and ws must be 16-byte aligned");
  const int T = batch.rows();
  *L = make_layout(cfg, T, (int)batch.chunks.size(), kv->max_seq_len);
  if (ws_bytes < L->total)
    return fail(SARATHI_ENOSPC, "workspace of %zu bytes < %zu needed", ws_bytes, L->total);
  const char* wb = static_cast<const char*>(ws);
  const char* xi = static_cast<const char*>(x_in);
  const char* xo = static_cast<const char*>(x_out);
  const size_t xbytes = (size_t)T * cfg->hidden * esize(cfg);
  auto overlap = [](const char* a, size_t na, const char* b, size_t nb) { return a < b + nb && b < a + na; };
  if (overlap(xi, xbytes, wb, L->total) || overlap(xo, xbytes, wb, L->total) || overlap(xi, xbytes, xo, xbytes))
    return fail(SARATHI_EINVAL, "x_in, x_out and the workspace must not overlap");
  *plan = make_plan(cfg, batch);
  // the plan must fit the regions the layout sized for it (an internal
  // invariant: the bounds above hold for every batch check_batch accepts)
  const size_t part_rows = (L->meta - L->part) / ((size_t)cfg->n_heads * (cfg->head_dim + PART_O) * 4);
  if (plan->meta.size() * 4 > L->ping0 - L->meta || (size_t)plan->pre_slots * plan->qblock + plan->n_dec > part_rows)
    return fail(SARATHI_EINVAL, "internal: batch plan exceeds its workspace layout");
  return SARATHI_OK;
}

}  // namespace

int sarathi::hybrid_check_noalloc(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w, const sarathi_kv* kv,
                                  int layer, const sarathi_hybrid_batch* batch, const void* x_in, const void* x_out,
                                  size_t* need) {
  BatchDesc b;
  int rc = from_hybrid(batch, &b);
  if (rc) return rc;
  rc = check_call(cfg, w, 1, kv, b, x_in, x_out);
  if (rc) return rc;
  if (layer < 0 || layer >= cfg->n_layers) return fail(SARATHI_EINVAL, "layer %d outside [0, %d)", layer, cfg->n_layers);
  *need = make_layout(cfg, b.rows(), (int)b.chunks.size(), kv->max_seq_len).total;
  return SARATHI_OK;
}

// ============================================================================ C-ABI

extern "C" {

int sarathi_version(void) { return 1; }

const char* sarathi_last_error(void) { return g_err.c_str(); }

size_t sarathi_kv_bytes(const sarathi_model_cfg* cfg, int n_slots, int max_seq_len) {
  if (check_cfg(cfg) != SARATHI_OK || n_slots < 1 || max_seq_len < 1) return 0;
  return (size_t)cfg->n_layers * n_slots * 2 * cfg->n_heads * (size_t)max_seq_len * cfg->head_dim * esize(cfg);
}

int sarathi_kv_alloc(const sarathi_model_cfg* cfg, int n_slots, int max_seq_len, void* dev_mem, size_t dev_bytes,
                     sarathi_kv** out) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!out) return fail(SARATHI_EINVAL, "out is NULL");
  *out = nullptr;
  if (!dev_mem) return fail(SARATHI_EINVAL, "dev_mem is NULL");
  if (!aligned16(dev_mem)) return fail(SARATHI_EINVAL, "dev_mem must be 16-byte aligned");
  if (n_slots < 1 || n_slots > (1 << 20)) return fail(SARATHI_EINVAL, "n_slots %d out of range", n_slots);
  if (max_seq_len < 1 || max_seq_len > (1 << 20)) return fail(SARATHI_EINVAL, "max_seq_len %d out of range", max_seq_len);
  const size_t need = sarathi_kv_bytes(cfg, n_slots, max_seq_len);
  if (dev_bytes < need) return fail(SARATHI_ENOSPC, "KV memory of %zu bytes < %zu needed", dev_bytes, need);
  sarathi_kv* kv = new sarathi_kv;
  kv->cfg = *cfg;
  kv->n_slots = n_slots;
  kv->max_seq_len = max_seq_len;
  kv->mem = dev_mem;
  kv->bytes = dev_bytes;
  kv->st.pos = cfg->head_dim;
  kv->st.head = (size_t)max_seq_len * cfg->head_dim;
  kv->st.kv = kv->st.head * cfg->n_heads;
  kv->st.slot = kv->st.kv * 2;
  kv->st.layer = kv->st.slot * n_slots;
  *out = kv;
  return SARATHI_OK;
}

void sarathi_kv_free(sarathi_kv* kv) { delete kv; }

int sarathi_kv_get_strides(const sarathi_kv* kv, sarathi_kv_strides* out) {
  if (!kv || !out) return fail(SARATHI_EINVAL, "NULL argument");
  out->layer = kv->st.layer; out->slot = kv->st.slot; out->kv = kv->st.kv; out->head = kv->st.head; out->pos = kv->st.pos;
  return SARATHI_OK;
}

size_t sarathi_workspace_bytes(const sarathi_model_cfg* cfg, int max_tokens, int max_decodes, int max_seq_len) {
  if (check_cfg(cfg) != SARATHI_OK || max_tokens < 1 || max_decodes < 0 || max_seq_len < 1) return 0;
  (void)max_decodes;
  return make_layout(cfg, max_tokens, 1, max_seq_len).total;
}

size_t sarathi_mixed_workspace_bytes(const sarathi_model_cfg* cfg, int max_tokens, int max_chunks, int max_seq_len) {
  if (check_cfg(cfg) != SARATHI_OK || max_tokens < 1 || max_chunks < 0 || max_seq_len < 1) return 0;
  return make_layout(cfg, max_tokens, max_chunks, max_seq_len).total;
}

namespace {
int layout_out(const sarathi_model_cfg* cfg, int n_tokens, int n_chunks, int max_seq_len, sarathi_ws_layout* out) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!out) return fail(SARATHI_EINVAL, "out is NULL");
  if (n_tokens < 1 || n_chunks < 0 || max_seq_len < 1) return fail(SARATHI_EINVAL, "bad sizes");
  const Layout L = make_layout(cfg, n_tokens, n_chunks, max_seq_len);
  out->a = L.a; out->qkv = L.qkv; out->o = L.o; out->hres = L.hres; out->m = L.m;
  out->ping[0] = L.ping0; out->ping[1] = L.ping1; out->total = L.total;
  return SARATHI_OK;
}

int run_layer(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w, sarathi_kv* kv, int layer,
              const BatchDesc& b, const void* x_in, void* x_out, void* ws, size_t ws_bytes, void* hip_stream) {
  Plan plan;
  Layout L;
  int rc = prepare(cfg, w, 1, kv, b, x_in, x_out, ws, ws_bytes, &plan, &L);
  if (rc) return rc;
  if (layer < 0 || layer >= cfg->n_layers) return fail(SARATHI_EINVAL, "layer %d outside [0, %d)", layer, cfg->n_layers);
  Ctx c{cfg, kv, &plan, L, static_cast<char*>(ws), static_cast<hipStream_t>(hip_stream)};
  rc = upload_meta_rest(c);
  if (rc) return rc;
  return layer_body(c, w, layer, x_in, x_out, true);
}

int run_model(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w, sarathi_kv* kv, const BatchDesc& b,
              const void* x_in, void* x_out, void* ws, size_t ws_bytes, void* hip_stream) {
  Plan plan;
  Layout L;
  int rc = prepare(cfg, w, cfg->n_layers > 0 ? cfg->n_layers : 0, kv, b, x_in, x_out, ws, ws_bytes, &plan, &L);
  if (rc) return rc;
  Ctx c{cfg, kv, &plan, L, static_cast<char*>(ws), static_cast<hipStream_t>(hip_stream)};
  rc = upload_meta_rest(c);
  if (rc) return rc;
  char* ping[2] = {c.ws + L.ping0, c.ws + L.ping1};
  const int n = cfg->n_layers;
  bool norm1_ready = false;
  for (int l = 0; l < n; ++l) {
    const void* in = (l == 0) ? x_in : ping[l & 1];
    void* out = (l == n - 1) ? x_out : ping[(l + 1) & 1];
    bool next_ready = false;
    rc = layer_body(c, w + l, l, in, out, l == 0, norm1_ready, l + 1 < n ? w + l + 1 : nullptr, &next_ready);
    if (rc) return rc;
    norm1_ready = next_ready;
  }
  return SARATHI_OK;
}
}  // namespace

int sarathi_workspace_layout(const sarathi_model_cfg* cfg, int n_tokens, int n_decodes, int max_seq_len,
                             sarathi_ws_layout* out) {
  if (n_decodes < 0 || n_decodes > n_tokens) return fail(SARATHI_EINVAL, "bad sizes");
  return layout_out(cfg, n_tokens, 1, max_seq_len, out);
}

int sarathi_mixed_workspace_layout(const sarathi_model_cfg* cfg, int n_tokens, int n_chunks, int max_seq_len,
                                   sarathi_ws_layout* out) {
  return layout_out(cfg, n_tokens, n_chunks, max_seq_len, out);
}

int sarathi_hybrid_layer_forward(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w, sarathi_kv* kv,
                                 int layer, const sarathi_hybrid_batch* batch, const void* x_in, void* x_out,
                                 void* ws, size_t ws_bytes, void* hip_stream) {
  BatchDesc b;
  int rc = from_hybrid(batch, &b);
  if (rc) return rc;
  return run_layer(cfg, w, kv, layer, b, x_in, x_out, ws, ws_bytes, hip_stream);
}

int sarathi_model_step(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w, sarathi_kv* kv,
                       const sarathi_hybrid_batch* batch, const void* x_in, void* x_out, void* ws,
                       size_t ws_bytes, void* hip_stream) {
  if (!cfg) return fail(SARATHI_EINVAL, "cfg is NULL");
  BatchDesc b;
  int rc = from_hybrid(batch, &b);
  if (rc) return rc;
  return run_model(cfg, w, kv, b, x_in, x_out, ws, ws_bytes, hip_stream);
}

int sarathi_mixed_layer_forward(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w, sarathi_kv* kv,
                                int layer, const sarathi_mixed_batch* batch, const void* x_in, void* x_out,
                                void* ws, size_t ws_bytes, void* hip_stream) {
  BatchDesc b;
  int rc = from_mixed(batch, &b);
  if (rc) return rc;
  return run_layer(cfg, w, kv, layer, b, x_in, x_out, ws, ws_bytes, hip_stream);
}

int sarathi_mixed_model_step(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w, sarathi_kv* kv,
                             const sarathi_mixed_batch* batch, const void* x_in, void* x_out, void* ws,
                             size_t ws_bytes, void* hip_stream) {
  if (!cfg) return fail(SARATHI_EINVAL, "cfg is NULL");
  BatchDesc b;
  int rc = from_mixed(batch, &b);
  if (rc) return rc;
  return run_model(cfg, w, kv, b, x_in, x_out, ws, ws_bytes, hip_stream);
}

int sarathi_profile_begin(int max_calls) {
  if (max_calls < 1 || max_calls > (1 << 16)) return fail(SARATHI_EINVAL, "max_calls %d out of range", max_calls);
  std::lock_guard<std::mutex> lk(g_prof.mu);
  const size_t need = (size_t)EV_PER_CALL * max_calls;
  while (g_prof.pool.size() < need) {
    hipEvent_t e;
    hipError_t he = hipEventCreate(&e);
    if (he != hipSuccess) return hip_fail(he, "hipEventCreate");
    g_prof.pool.push_back(e);
  }
  g_prof.on = true;
  g_prof.max_calls = max_calls;
  g_prof.calls = 0;
  return SARATHI_OK;
}

int sarathi_profile_end(double* stage_ms, int* n_calls) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (!g_prof.on) return fail(SARATHI_EINVAL, "profiling was not started");
  if (!stage_ms || !n_calls) return fail(SARATHI_EINVAL, "NULL output");
  g_prof.on = false;
  for (int s = 0; s < SARATHI_N_STAGES; ++s) stage_ms[s] = 0.0;
  *n_calls = g_prof.calls;
  if (g_prof.calls == 0) return SARATHI_OK;
  hipError_t he = hipEventSynchronize(g_prof.pool[(size_t)EV_PER_CALL * g_prof.calls - 1]);
  if (he != hipSuccess) return hip_fail(he, "hipEventSynchronize");
  for (int c = 0; c < g_prof.calls; ++c) {
    hipEvent_t* ev = g_prof.pool.data() + (size_t)EV_PER_CALL * c;
    for (int s = 0; s < SARATHI_N_STAGES; ++s) {
      float ms = 0.f;
      he = hipEventElapsedTime(&ms, ev[s], ev[s + 1]);
      if (he != hipSuccess) return hip_fail(he, "hipEventElapsedTime");
      stage_ms[s] += ms;
    }
  }
  return SARATHI_OK;
}

size_t sarathi_linear_scratch_bytes(int M, int N) {
  if (M < 1 || N < 1) return 0;
  return (size_t)MAX_SPLIT * M * N * 4;
}

namespace {
int linear_common(int dtype, int kind, int M, int N, int K, const void* x, const void* w, const void* resid,
                  void* out, void* scratch, size_t scratch_bytes, void* hip_stream, int tile, int n_split) {
  if (dtype != SARATHI_F32 && dtype != SARATHI_BF16) return fail(SARATHI_EUNSUPPORTED, "dtype %d", dtype);
  if (kind < SARATHI_LINEAR_PLAIN || kind > SARATHI_LINEAR_GELU) return fail(SARATHI_EINVAL, "kind %d", kind);
  if (M < 1 || N < 1 || K < 1) return fail(SARATHI_EINVAL, "M, N, K must be positive");
  if (K % 8) return fail(SARATHI_EUNSUPPORTED, "K %d must be a multiple of 8", K);
  if (!x || !w || !out) return fail(SARATHI_EINVAL, "NULL pointer");
  const bool needs_resid = kind == SARATHI_LINEAR_RESID || kind == SARATHI_LINEAR_RESID_F32IN;
  if (needs_resid && !resid) return fail(SARATHI_EINVAL, "resid is NULL");
  if (!aligned16(x) || !aligned16(w)) return fail(SARATHI_EINVAL, "x and w must be 16-byte aligned");
  LinearArgs a{};
  a.kind = kind; a.M = M; a.N = N; a.K = K; a.x = x; a.w = w; a.resid = resid; a.out = out;
  if (needs_resid && scratch && aligned16(scratch)) {
    a.parts = static_cast<float*>(scratch);
    a.parts_cap = scratch_bytes / 4;
  }
  hipError_t e = launch_linear(dtype, a, static_cast<hipStream_t>(hip_stream), tile, n_split);
  if (e != hipSuccess) return hip_fail(e, "linear");
  return SARATHI_OK;
}
}  // namespace

int sarathi_linear(int dtype, int kind, int M, int N, int K, const void* x, const void* w, const void* resid,
                   void* out, void* scratch, size_t scratch_bytes, void* hip_stream) {
  return linear_common(dtype, kind, M, N, K, x, w, resid, out, scratch, scratch_bytes, hip_stream, -1, 0);
}

int sarathi_attention_plan(const sarathi_model_cfg* cfg, const sarathi_hybrid_batch* batch, sarathi_attn_plan* out) {
  if (!out) return fail(SARATHI_EINVAL, "out is NULL");
  int rc = check_cfg(cfg);
  if (rc) return rc;
  BatchDesc b;
  rc = from_hybrid(batch, &b);
  if (rc) return rc;
  if (b.rows() < 1) return fail(SARATHI_EINVAL, "empty batch (no chunk rows and no decodes)");
  if (b.B > 0 && (!b.dslots || !b.dctx)) return fail(SARATHI_EINVAL, "decode arrays are NULL");
  const Plan P = make_plan(cfg, b);
  const int* comb = P.meta.data() + P.o_comb;
  const int* pre = P.meta.data() + P.o_pre;
  const int* chunks = P.meta.data() + P.o_chunks;
  sarathi_attn_plan o{};
  o.chunk_items = P.n_pre;
  o.decode_items = P.n_dec;
  long written = P.n_dec;
  for (int i = 0; i < P.n_pre; ++i)
    if (pre[4 * i + 2] >= 0) {
      const int len = chunks[4 * pre[4 * i] + 2], q0 = pre[4 * i + 1] * P.qblock;
      written += std::min(P.qblock, len - q0);
    }
  o.partial_rows_written = written;
  for (int r = 0; r < P.T; ++r)
    if (comb[3 * r + 1] > 0) {
      o.partial_rows_read += comb[3 * r + 1];
      ++o.combine_rows;
    }
  *out = o;
  return SARATHI_OK;
}

int sarathi_linear_plan(int dtype, int kind, int M, int N, int K, size_t scratch_bytes, int* bm, int* bn,
                        int* n_split) {
  if (!bm || !bn || !n_split) return fail(SARATHI_EINVAL, "NULL pointer");
  if (dtype != SARATHI_F32 && dtype != SARATHI_BF16) return fail(SARATHI_EUNSUPPORTED, "dtype %d", dtype);
  if (kind < SARATHI_LINEAR_PLAIN || kind > SARATHI_LINEAR_GELU) return fail(SARATHI_EINVAL, "kind %d", kind);
  if (M < 1 || N < 1 || K < 1) return fail(SARATHI_EINVAL, "M, N, K must be positive");
  if (K % 8) return fail(SARATHI_EUNSUPPORTED, "K %d must be a multiple of 8", K);
  LinearArgs a{};
  a.kind = kind; a.M = M; a.N = N; a.K = K;
  static float dummy;   // plan only: the scratch is never touched
  if ((kind == SARATHI_LINEAR_RESID || kind == SARATHI_LINEAR_RESID_F32IN) && scratch_bytes >= 4) {
    a.parts = &dummy;
    a.parts_cap = scratch_bytes / 4;
  }
  LinearPlan pl{};
  if (launch_linear(dtype, a, nullptr, -1, 0, &pl) != hipSuccess) return fail(SARATHI_EINVAL, "no plan for this op");
  *bm = pl.bm; *bn = pl.bn; *n_split = pl.n_split;
  return SARATHI_OK;
}

size_t sarathi_layer_split_scratch_bytes(const sarathi_model_cfg* cfg, int n_tokens) {
  if (!cfg || n_tokens < 1) return 0;
  return (size_t)MAX_SPLIT * std::min(n_tokens, PARTS_ROWS) * cfg->hidden * 4;
}

int sarathi_linear_tile_count(void) { return linear_tile_count(); }

int sarathi_linear_tile_shape(int tile, int* bm, int* bn) {
  if (!bm || !bn) return fail(SARATHI_EINVAL, "NULL pointer");
  if (!linear_tile_shape(tile, bm, bn)) return fail(SARATHI_EINVAL, "tile %d outside [0, %d)", tile, linear_tile_count());
  return SARATHI_OK;
}

int sarathi_linear_tiled(int kind, int M, int N, int K, const void* x, const void* w, const void* resid, void* out,
                         void* scratch, size_t scratch_bytes, int tile, int n_split, void* hip_stream) {
  if (tile < 0 || tile >= linear_tile_count()) return fail(SARATHI_EINVAL, "tile %d outside [0, %d)", tile, linear_tile_count());
  if (n_split < 1) return fail(SARATHI_EINVAL, "n_split %d < 1", n_split);
  if (K % 64) return fail(SARATHI_EUNSUPPORTED, "K %d must be a multiple of 64 for a given tile", K);
  return linear_common(SARATHI_BF16, kind, M, N, K, x, w, resid, out, scratch, scratch_bytes, hip_stream, tile,
                       n_split);
}

}  // extern "C"
