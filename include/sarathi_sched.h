/*
 * sarathi_sched.h -- host-side iteration scheduler of libsarathi.so.
 *
 * Forms the batch of every model iteration from a set of requests, each a
 * prompt of P tokens followed by D decode iterations, under one of three
 * policies:
 *
 *   SARATHI_POLICY_DECODE_MAXIMAL  (Sec. 4.3): every iteration carries at most
 *     one prefill chunk of up to `chunk` tokens (the next chunk of the oldest
 *     admitted request still in its prefill, Sec. 4.2) plus a decode for each
 *     admitted request in its decode phase -- at most max_batch - 1 decodes
 *     beside a chunk, max_batch without one;
 *   SARATHI_POLICY_PREFILL_DECODE  (the baseline of Sec. 5.1): prefill-only
 *     iterations, each the whole remaining prompt of one request, whenever an
 *     admitted request still has prompt left; otherwise one decode-only
 *     iteration over every admitted request in its decode phase;
 *   SARATHI_POLICY_MIXED  (the iteration-level "mixed batching" of Orca that
 *     Sec. 5.2 compares against): every iteration carries the whole remaining
 *     prompt of every admitted request still in prefill (up to `max_chunks`
 *     of them, oldest first, and while the rows stay within `max_tokens`)
 *     plus every decode.
 *
 * Requests are admitted in submission order while fewer than max_batch are
 * resident; an admitted request holds one KV slot (a pre-allocated slab of
 * max_seq_len positions, Sec. 4.5) until its last decode.  A request in its
 * decode phase with c tokens cached decodes at position c, so its decodes
 * run at context lengths P, P+1, ..., P+D-1; a request with D = 0 retires
 * when its prompt is done.  No decision depends on model outputs (no
 * sampling, no end-of-sequence), so a caller may enqueue iterations ahead of
 * the GPU.
 *
 * Use: sarathi_sched_next() describes the next iteration (the same one until
 * sarathi_sched_commit() is called, except that an empty description is
 * rebuilt, so requests submitted after it are seen); after enqueueing it,
 * commit advances every request in it.  Arrays in sarathi_sched_step are owned by the
 * scheduler and valid until the next call on it.  A scheduler is not
 * thread-safe.  Errors: SARATHI_EINVAL (null pointer, bad config value),
 * SARATHI_ERANGE (P + D > max_seq_len, P < 1, D < 0), SARATHI_ENOSPC (commit
 * with no iteration pending); message via sarathi_last_error().
 */
#ifndef SARATHI_SCHED_H
#define SARATHI_SCHED_H

#include "sarathi.h"

#ifdef __cplusplus
extern "C" {
#endif

#define SARATHI_POLICY_DECODE_MAXIMAL  0
#define SARATHI_POLICY_PREFILL_DECODE  1
#define SARATHI_POLICY_MIXED           2

typedef struct {
  int policy;
  int max_batch;    /* B: requests resident at once (>= 1) */
  int chunk;        /* C: prefill chunk length (DECODE_MAXIMAL; >= 1) */
  int max_chunks;   /* MIXED: prompts per iteration (>= 1) */
  int max_tokens;   /* MIXED: prompt rows per iteration (the oldest prompt is always taken whole) */
  int n_slots;      /* KV slots 0..n_slots-1 available (>= max_batch) */
  int max_seq_len;  /* positions per slot */
} sarathi_sched_cfg;

typedef struct sarathi_sched sarathi_sched;

typedef struct {
  int n_tokens;                 /* rows of the iteration: sum of chunk lengths + n_decodes */
  int n_chunks;                 /* 0 (decode-only), 1, or more (MIXED) */
  const int* chunk_request;     /* [n_chunks] request ids */
  const int* chunk_slot;        /* [n_chunks] KV slots */
  const int* chunk_offset;      /* [n_chunks] first position of each chunk */
  const int* chunk_len;         /* [n_chunks] */
  int n_decodes;
  const int* decode_request;    /* [n_decodes] request ids, in admission order */
  const int* decode_slot;       /* [n_decodes] */
  const int* decode_ctx;        /* [n_decodes] context length = position written */
} sarathi_sched_step;

typedef struct {
  long long iterations;         /* committed */
  long long prefill_tokens;
  long long decode_tokens;
  long long hybrid_iterations;  /* chunk(s) and decodes together */
  long long prefill_only_iterations;
  long long decode_only_iterations;
  int submitted, admitted, finished, resident;
} sarathi_sched_stats;

int sarathi_sched_create(const sarathi_sched_cfg* cfg, sarathi_sched** out);
void sarathi_sched_destroy(sarathi_sched* s);
/* Queue a request of prompt_len tokens and decode_len decode iterations; its id is the submission index. */
int sarathi_sched_submit(sarathi_sched* s, int prompt_len, int decode_len, int* request_id);
/* Describe the next iteration (n_tokens = 0 when every request is finished). */
int sarathi_sched_next(sarathi_sched* s, sarathi_sched_step* out);
/* Advance the requests of the iteration last returned by sarathi_sched_next. */
int sarathi_sched_commit(sarathi_sched* s);
int sarathi_sched_get_stats(const sarathi_sched* s, sarathi_sched_stats* out);

#ifdef __cplusplus
}
#endif

#endif /* SARATHI_SCHED_H */
