// Host-side iteration scheduler: decode-maximal batching (Sec. 4.3), the
// prefill-only / decode-only baseline (Sec. 5.1) and Orca-style mixed
// batching (Sec. 5.2).  Pure host code; no GPU call.
#include <algorithm>
#include <deque>
#include <vector>

#include "host_error.h"
#include "sarathi_sched.h"

using sarathi::fail;

namespace {

enum State { PENDING = 0, PREFILL = 1, DECODE = 2, FINISHED = 3 };

struct Req {
  int P, D;
  int slot = -1;
  int done_prompt = 0;    // prompt tokens already in the cache
  int done_decodes = 0;
  State state = PENDING;
};

}  // namespace

struct sarathi_sched {
  sarathi_sched_cfg cfg;
  std::vector<Req> reqs;
  std::deque<int> pending;          // submitted, not admitted (submission order)
  std::vector<int> resident;        // admitted, not finished (admission order)
  std::vector<int> free_slots;      // stack, lowest slot on top
  bool have_step = false;
  std::vector<int> c_req, c_slot, c_off, c_len, d_req, d_slot, d_ctx;
  sarathi_sched_stats st{};
};

namespace {

void admit(sarathi_sched* s) {
  while ((int)s->resident.size() < s->cfg.max_batch && !s->pending.empty() && !s->free_slots.empty()) {
    const int id = s->pending.front();
    s->pending.pop_front();
    Req& r = s->reqs[id];
    r.slot = s->free_slots.back();
    s->free_slots.pop_back();
    r.state = PREFILL;
    s->resident.push_back(id);
    s->st.admitted++;
  }
}

void add_chunk(sarathi_sched* s, int id, int len) {
  const Req& r = s->reqs[id];
  s->c_req.push_back(id);
  s->c_slot.push_back(r.slot);
  s->c_off.push_back(r.done_prompt);
  s->c_len.push_back(len);
}

void build(sarathi_sched* s) {
  s->c_req.clear(); s->c_slot.clear(); s->c_off.clear(); s->c_len.clear();
  s->d_req.clear(); s->d_slot.clear(); s->d_ctx.clear();
  admit(s);
  const sarathi_sched_cfg& c = s->cfg;
  bool want_decodes = true;
  int decode_cap = c.max_batch;
  if (c.policy == SARATHI_POLICY_DECODE_MAXIMAL) {
    for (int id : s->resident) {
      const Req& r = s->reqs[id];
      if (r.state == PREFILL) {
        add_chunk(s, id, std::min(c.chunk, r.P - r.done_prompt));
        decode_cap = c.max_batch - 1;
        break;
      }
    }
  } else if (c.policy == SARATHI_POLICY_PREFILL_DECODE) {
    for (int id : s->resident) {
      const Req& r = s->reqs[id];
      if (r.state == PREFILL) {
        add_chunk(s, id, r.P - r.done_prompt);
        want_decodes = false;
        break;
      }
    }
  } else {   // MIXED
    int rows = 0;
    for (int id : s->resident) {
      const Req& r = s->reqs[id];
      if (r.state != PREFILL) continue;
      if ((int)s->c_req.size() >= c.max_chunks) break;
      const int len = r.P - r.done_prompt;
      if (!s->c_req.empty() && rows + len > c.max_tokens) break;
      add_chunk(s, id, len);
      rows += len;
    }
  }
  if (want_decodes) {
    for (int id : s->resident) {
      if ((int)s->d_req.size() >= decode_cap) break;
      const Req& r = s->reqs[id];
      if (r.state != DECODE) continue;
      s->d_req.push_back(id);
      s->d_slot.push_back(r.slot);
      s->d_ctx.push_back(r.P + r.done_decodes);
    }
  }
  s->have_step = true;
}

void retire(sarathi_sched* s, int id) {
  Req& r = s->reqs[id];
  r.state = FINISHED;
  s->free_slots.push_back(r.slot);
  // keep the lowest free slot on top so slot use is deterministic
  for (size_t i = s->free_slots.size() - 1; i > 0 && s->free_slots[i] > s->free_slots[i - 1]; --i)
    std::swap(s->free_slots[i], s->free_slots[i - 1]);
  s->st.finished++;
}

}  // namespace

extern "C" {

int sarathi_sched_create(const sarathi_sched_cfg* cfg, sarathi_sched** out) {
  if (!cfg || !out) return fail(SARATHI_EINVAL, "NULL argument");
  *out = nullptr;
  if (cfg->policy < SARATHI_POLICY_DECODE_MAXIMAL || cfg->policy > SARATHI_POLICY_MIXED)
    return fail(SARATHI_EINVAL, "unknown policy %d", cfg->policy);
  if (cfg->max_batch < 1) return fail(SARATHI_EINVAL, "max_batch %d < 1", cfg->max_batch);
  if (cfg->policy == SARATHI_POLICY_DECODE_MAXIMAL && cfg->chunk < 1)
    return fail(SARATHI_EINVAL, "chunk %d < 1", cfg->chunk);
  if (cfg->policy == SARATHI_POLICY_MIXED && (cfg->max_chunks < 1 || cfg->max_tokens < 1))
    return fail(SARATHI_EINVAL, "max_chunks and max_tokens must be >= 1");
  if (cfg->n_slots < cfg->max_batch) return fail(SARATHI_EINVAL, "n_slots %d < max_batch %d", cfg->n_slots, cfg->max_batch);
  if (cfg->max_seq_len < 1) return fail(SARATHI_EINVAL, "max_seq_len %d < 1", cfg->max_seq_len);
  sarathi_sched* s = new sarathi_sched;
  s->cfg = *cfg;
  for (int i = cfg->n_slots - 1; i >= 0; --i) s->free_slots.push_back(i);
  *out = s;
  return SARATHI_OK;
}

void sarathi_sched_destroy(sarathi_sched* s) { delete s; }

int sarathi_sched_submit(sarathi_sched* s, int prompt_len, int decode_len, int* request_id) {
  if (!s) return fail(SARATHI_EINVAL, "scheduler is NULL");
  if (prompt_len < 1 || decode_len < 0)
    return fail(SARATHI_ERANGE, "prompt_len %d must be >= 1 and decode_len %d >= 0", prompt_len, decode_len);
  if ((long long)prompt_len + decode_len > s->cfg.max_seq_len)
    return fail(SARATHI_ERANGE, "prompt_len + decode_len = %lld > max_seq_len %d",
                (long long)prompt_len + decode_len, s->cfg.max_seq_len);
  Req r;
  r.P = prompt_len;
  r.D = decode_len;
  s->reqs.push_back(r);
  const int id = (int)s->reqs.size() - 1;
  s->pending.push_back(id);
  s->st.submitted++;
  if (request_id) *request_id = id;
  return SARATHI_OK;
}

int sarathi_sched_next(sarathi_sched* s, sarathi_sched_step* out) {
  if (!s || !out) return fail(SARATHI_EINVAL, "NULL argument");
  // the described iteration stays fixed until commit; an empty one is
  // rebuilt so that requests submitted meanwhile are seen
  if (!s->have_step || (s->c_req.empty() && s->d_req.empty())) build(s);
  out->n_chunks = (int)s->c_req.size();
  out->chunk_request = s->c_req.data();
  out->chunk_slot = s->c_slot.data();
  out->chunk_offset = s->c_off.data();
  out->chunk_len = s->c_len.data();
  out->n_decodes = (int)s->d_req.size();
  out->decode_request = s->d_req.data();
  out->decode_slot = s->d_slot.data();
  out->decode_ctx = s->d_ctx.data();
  int rows = out->n_decodes;
  for (int l : s->c_len) rows += l;
  out->n_tokens = rows;
  return SARATHI_OK;
}

int sarathi_sched_commit(sarathi_sched* s) {
  if (!s) return fail(SARATHI_EINVAL, "scheduler is NULL");
  if (!s->have_step) return fail(SARATHI_ENOSPC, "no iteration to commit (call sarathi_sched_next first)");
  const bool chunks = !s->c_req.empty(), decodes = !s->d_req.empty();
  if (!chunks && !decodes) {   // idle: nothing to advance
    s->have_step = false;
    return SARATHI_OK;
  }
  std::vector<int> done;
  for (size_t i = 0; i < s->c_req.size(); ++i) {
    Req& r = s->reqs[s->c_req[i]];
    r.done_prompt += s->c_len[i];
    s->st.prefill_tokens += s->c_len[i];
    if (r.done_prompt == r.P) {
      r.state = DECODE;
      if (r.D == 0) done.push_back(s->c_req[i]);
    }
  }
  for (int id : s->d_req) {
    Req& r = s->reqs[id];
    r.done_decodes++;
    s->st.decode_tokens++;
    if (r.done_decodes == r.D) done.push_back(id);
  }
  for (int id : done) retire(s, id);
  if (!done.empty()) {
    std::vector<int> keep;
    for (int id : s->resident)
      if (s->reqs[id].state != FINISHED) keep.push_back(id);
    s->resident.swap(keep);
  }
  s->st.iterations++;
  if (chunks && decodes) s->st.hybrid_iterations++;
  else if (chunks) s->st.prefill_only_iterations++;
  else s->st.decode_only_iterations++;
  s->have_step = false;
  return SARATHI_OK;
}

int sarathi_sched_get_stats(const sarathi_sched* s, sarathi_sched_stats* out) {
  if (!s || !out) return fail(SARATHI_EINVAL, "NULL argument");
  *out = s->st;
  out->resident = (int)s->resident.size();
  return SARATHI_OK;
}

}  // extern "C"
