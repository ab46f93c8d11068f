/*
 * cp_sched.h — C ABI of the host-side chunked-prefill scheduler that builds
 * the batches cp_attn.h executes: Aging prefill ordering (Sec. 3.1, Eq. 1–4),
 * LPRS target-latency chunk selection (Sec. 3.2, Eq. 6–11, Algorithm 1) and
 * Active Prefill Control (Sec. 3.3, Eq. 12–14).  Plain C++17, no GPU calls.
 *
 * One scheduling round (the four-step online procedure of Sec. 3.2.2):
 *   1. the caller sets the GPU-memory features of the round
 *      (cps_set_memory_state, optional) and calls cps_schedule(now);
 *   2. every decoding request gets a one-token row first (decode-first
 *      admission, Sec. 3.1.3), while the token budget B_max lasts;
 *   3. waiting prefills are taken in priority order (max-heap on the ordering
 *      key K_i of Eq. 4 under CPS_POLICY_AGING, arrival order under
 *      CPS_POLICY_FCFS).  For each, h_i = min(r_i, B_max - U_t) (Eq. 6); the
 *      chunk is c = h_i under CPS_CHUNK_TOKEN_BUDGET (Eq. 7) or Algorithm 1's
 *      c* under CPS_CHUNK_LPRS; with APC on, Eq. 14 then accepts c*, replaces
 *      it by the warm-start chunk, or blocks it; once the round holds
 *      |P_t| > 0 prefill chunks and |P_t| >= C_t, Eq. 14 returns 0 for every
 *      later candidate, so the scan stops there.  A request gets at most one
 *      chunk per round; its remaining work drops by c (Eq. 2) and it goes back
 *      to the heap with its new key if prompt tokens remain;
 *   4. the batch comes back as cp_row_meta rows (decode rows first), ready
 *      for cp_kv_append / cp_attn_mixed.  After the step has run, the caller
 *      calls cps_complete(now): prefills that finished their prompt emit
 *      their first token and start decoding, decode rows emit one token each,
 *      and requests that reached their output length release their slot.
 *
 * Rows' req_id is a slot: a row index of the caller's block table
 * [max_seqs][ceil(max_seq_len / block_size)].  A request takes a free slot
 * when its first chunk is scheduled and keeps it until its last token.
 *
 * Ownership: a cps_sched is created and destroyed by the caller and is not
 * thread-safe.  Every array argument is a host array owned by the caller and
 * read or written only during the call.
 *
 * Errors: functions return CPS_OK (0) or a negative CPS_ERR_* code; a call
 * that fails changes no scheduler state, except CPS_ERR_NO_MEMORY from
 * cps_schedule, after which the scheduler may only be destroyed.  No C++
 * exception crosses the ABI.
 */
#ifndef CP_SCHED_H
#define CP_SCHED_H

#include <stdint.h>

#include "cp_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

#define CPS_OK 0
#define CPS_ERR_INVALID_ARG (-1) /* null pointer, value out of range          */
#define CPS_ERR_CAPACITY (-2)    /* output array too small, table full        */
#define CPS_ERR_NO_PREDICTOR (-3) /* LPRS selected but no predictor loaded    */
#define CPS_ERR_STATE (-4)       /* call out of order (complete before schedule,
                                    duplicate request id)                     */
#define CPS_ERR_NO_MEMORY (-5)   /* a host allocation failed                  */

#define CPS_POLICY_FCFS 0        /* prefills in arrival order                 */
#define CPS_POLICY_AGING 1       /* max-heap on K_i = -alpha*a_i + beta*r_i   */

#define CPS_CHUNK_TOKEN_BUDGET 0 /* c = h_i (static token budget, Eq. 7)      */
#define CPS_CHUNK_LPRS 1         /* Algorithm 1 against target_us             */

/* Number of predictor inputs: the 11 raw features of Table 1 followed by the
 * 5 derived features of Table 2, in this order:
 *   0 prefill_tokens            sum of chunk_len over prefill rows
 *   1 decode_tokens             number of decode rows (chunk_len == 1)
 *   2 batch_request_count       rows with chunk_len > 0
 *   3 sum_decode_context_len    sum of ctx_len over decode rows
 *   4 max_decode_context_len    max of ctx_len over decode rows (0 if none)
 *   5 prefill_processed_tokens  sum of chunk_start over prefill rows: the
 *                               prompt tokens already in the cache
 *   6 max_prefill_processed_tokens  max of chunk_start over prefill rows
 *   7 gpu_mem_used_mb  8 gpu_mem_free_mb  9 cuda_allocated_mb
 *  10 cuda_reserved_mb          the round's memory state (MB)
 *  11 bias = 1                  12 scheduled_tokens = decode + prefill tokens
 *  13 avg_decode_ctx = sum_decode_context_len / max(decode_tokens, 1)
 *  14 decode_ctx_interaction = decode_tokens * avg_decode_ctx
 *  15 prefill_interaction = prefill_tokens * prefill_processed_tokens
 * A row with chunk_len >= 2 is a prefill row, chunk_len == 1 a decode row,
 * the same split the attention kernels make. */
#define CPS_NUM_FEATURES 16

typedef struct {
  int32_t policy;        /* CPS_POLICY_*                                      */
  double alpha;          /* aging weight on waiting time (Eq. 1), > 0         */
  double beta;           /* weight on remaining prefill tokens (Eq. 1), < 0   */
  int32_t max_tokens;    /* B_max: scheduled tokens per round, >= 1           */
  int32_t max_seqs;      /* S_max: sequence slots, >= 1                       */
  int32_t max_seq_len;   /* prompt + output tokens of one request, >= 2       */
  int32_t chunking;      /* CPS_CHUNK_*                                       */
  double target_us;      /* T*: target step latency (predictor units)         */
  int32_t delta;         /* search granularity of Eq. 8, >= 1                 */
  double lambda_u;       /* underfill penalty of Eq. 10, >= 0                 */
  double lambda_o;       /* overflow penalty of Eq. 10, >= lambda_u           */
  int32_t apc;           /* 1: apply Eq. 12–14 to every prefill chunk         */
  int32_t max_active;    /* C_max of Eq. 12, >= 1                             */
  int32_t min_chunk;     /* L_min of Eq. 12–13, >= 1                          */
} cps_config;

/* Cumulative counters since cps_create. */
typedef struct {
  int64_t rounds;            /* cps_schedule calls                            */
  int64_t decode_rows;       /* decode rows scheduled                         */
  int64_t prefill_rows;      /* prefill chunks scheduled                      */
  int64_t prefill_tokens;    /* prompt tokens scheduled                       */
  int64_t lprs_calls;        /* Algorithm 1 evaluations                       */
  int64_t predictor_rows;    /* candidate feature vectors scored              */
  int64_t apc_blocked_cap;   /* Eq. 14 "otherwise": c* >= m_i but |P_t| >= C_t */
  int64_t apc_blocked_min;   /* Eq. 14 "otherwise": c* < m_i and |P_t| > 0     */
  int64_t apc_warm_starts;   /* Eq. 14 second case taken with c != c*          */
  int64_t skipped_no_slot;   /* candidates passed over: every slot taken      */
  int64_t apc_not_scored;    /* candidates left unscored: the round's active
                                set was full (|P_t| > 0 and |P_t| >= C_t, so
                                Eq. 14 gives 0 whatever c* is)                 */
  int64_t finished;          /* requests that emitted their last token        */
} cps_stats;

/* Per-request record, times in the caller's clock (the `now` arguments). */
typedef struct {
  double arrival;
  double first_token;        /* -1 until the prompt is done                   */
  double finish;             /* -1 until the last token                       */
  int32_t prompt_len, max_new_tokens, processed, generated, chunks, slot;
} cps_request_info;

/* Validates the configuration; returns NULL and *err < 0 on bad input. */
typedef struct cps_sched cps_sched;
cps_sched* cps_create(const cps_config* cfg, int* err);
void cps_destroy(cps_sched* s);

/* Loads the latency predictor f_theta (Sec. 3.2.1, Eq. 9): an MLP with
 * n_layers affine layers of sizes dims[0] = CPS_NUM_FEATURES, dims[1], ...,
 * dims[n_layers] = 1, ReLU between layers, applied to (x - x_mean) / x_std
 * and multiplied by y_scale.  weights holds W_l row-major [dims[l+1]][dims[l]]
 * back to back, biases the b_l back to back; the arrays are copied.  A
 * single layer (n_layers == 1) is a linear model. */
int cps_set_predictor(cps_sched* s, int32_t n_layers, const int32_t* dims,
                      const double* weights, const double* biases, const double* x_mean,
                      const double* x_std, double y_scale);

/* The four GPU-memory features (MB) used for every candidate until changed. */
int cps_set_memory_state(cps_sched* s, const double mem_mb[4]);

/* Registers a request that has arrived; id must be new and >= 0,
 * prompt_len >= 1, max_new_tokens >= 1, prompt_len + max_new_tokens <=
 * max_seq_len. */
int cps_add_request(cps_sched* s, int64_t id, double arrival, int32_t prompt_len,
                    int32_t max_new_tokens);

/* Builds the next batch (steps 2–4 above).  rows and ids (the request id of
 * each row) must hold `cap` entries; cap >= max_seqs always suffices.  Rows
 * come out decode rows first (*n_decode of them), then prefill chunks in
 * selection order.  *n_rows = 0 is a legal empty round.  The batch must be
 * completed before the next cps_schedule. */
int cps_schedule(cps_sched* s, double now, cp_row_meta* rows, int64_t* ids, int32_t cap,
                 int32_t* n_rows, int32_t* n_decode);

/* Records that the last scheduled batch has executed at time `now`. */
int cps_complete(cps_sched* s, double now);

int cps_get_stats(const cps_sched* s, cps_stats* out);
int cps_request(const cps_sched* s, int64_t id, cps_request_info* out);
/* Requests not yet finished (waiting, prefilling or decoding). */
int64_t cps_pending(const cps_sched* s);

/* ---- pieces of a round, exposed for callers that build batches themselves
 * ---- and for tests ------------------------------------------------------ */

/* Feature vector of one batch (definition above) into out[CPS_NUM_FEATURES]. */
int cps_batch_features(const cp_row_meta* rows, int32_t n_rows, const double mem_mb[4],
                       double* out);

/* Predictor outputs for n feature vectors x[n][CPS_NUM_FEATURES]. */
int cps_predict(const cps_sched* s, const double* x, int32_t n, double* out);

/* Algorithm 1 for one candidate: `committed` holds the rows already in the
 * round (U_t = sum of their chunk_len); the candidate would add the row
 * (slot, processed, c, processed + c).  Writes c* (0 if h_i <= 0) and, when
 * c* > 0, its predicted latency (else NaN).  Ties in score go to the larger
 * c; candidates whose score is NaN never win; the starvation rule returns 1
 * when nothing won, U_t == 0 and h_i >= 1. */
int cps_select_chunk(const cps_sched* s, const cp_row_meta* committed, int32_t n_committed,
                     int32_t slot, int32_t processed, int32_t remaining, int32_t* chunk,
                     double* predicted);

/* Eq. 12–14 for one candidate: with n_decode = |D_t|, n_active = |P_t| (the
 * prefill chunks already in the round), committed = U_t, h = h_i, remaining =
 * r_i and c_star the proposed chunk, writes the final chunk and the reason:
 * 0 accepted, 1 warm start, 2 blocked by the activity cap, 3 blocked by the
 * minimum effective chunk. */
int cps_apc_decide(const cps_config* cfg, int32_t c_star, int32_t h, int32_t remaining,
                   int32_t n_decode, int32_t n_active, int32_t committed, int32_t* chunk,
                   int32_t* reason);

#ifdef __cplusplus
}
#endif

#endif /* CP_SCHED_H */
