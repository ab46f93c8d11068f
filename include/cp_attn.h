/*
 * cp_attn.h — C ABI of the mixed prefill/decode paged-attention step of one
 * chunked-prefill scheduling iteration, for AMD Instinct MI355X (gfx950).
 *
 * The paper's scheduler (Aging ordering, LPRS target-time chunk selection,
 * APC activity control; Sec. 3) finalises a batch every round and submits it
 * to the backend (Sec. 3.2.2, the four-step online procedure).  A batch holds
 * every running decode request as a one-token row (decode-first admission,
 * Sec. 3.1.3) plus at most one prefill chunk per selected request (Sec. 3.1.3;
 * Algorithm 1 returns one chunk size per request).  This library executes the
 * attention part of that batch on the GPU:
 *
 *   cp_kv_append   writes the batch's new K/V rows into the paged cache;
 *   cp_attn_mixed  computes, for every scheduled query token, causal
 *                  attention over its request's cached keys.
 *
 * Scheduling never changes how chunks are executed or how the KV cache is
 * managed (Sec. 3.1.3), so this is a pure execution interface: the caller owns
 * every buffer and decides what goes in the batch.
 *
 * Definition computed (the paper names the operation but does not write it
 * out; this is standard scaled-dot-product attention with grouped KV heads):
 * for row r with metadata (req, start, len, ctx), query j < len sits at
 * absolute position p = start + j and q head h reads kv head g = h / (Hq/Hkv);
 *     out[t][h] = sum_{i<=p} softmax_i(sm_scale * q[t][h] . K_i) V_i
 * where K_i, V_i are the keys/values of request req at logical position i,
 * t = (sum of len over rows before r) + j.  Softmax is evaluated in fp32 with
 * bf16 inputs, products accumulated in fp32, and the output rounded to bf16.
 *
 * Layouts (all bf16 tensors are dense, row-major, 16-byte aligned):
 *   q, out        [T][Hq][D]        T = sum of chunk_len over rows, rows packed
 *                                   in the order of the rows array
 *   k_new, v_new  [T][Hkv][D]
 *   k_cache       [num_blocks][Hkv][B][D]   token-major inside a block
 *   v_cache       [num_blocks][Hkv][D][B]   feature-major inside a block
 *   block_tables  int32 [num_reqs_in_table][max_blocks_per_req]; entry
 *                 [req][i] is the physical block of logical block i
 *   rows          host array of cp_row_meta, read only during the call
 *
 * Ownership: every device buffer is allocated and owned by the caller.  The
 * library never allocates device memory in these calls; it keeps one pinned
 * host staging ring (allocated on first use, reused afterwards) for plan
 * uploads.  The workspace is caller-provided, device memory, at least
 * cp_workspace_bytes() bytes, 256-byte aligned; it must not be used by any
 * other call that is in flight at the same time.
 *
 * Errors: functions return CP_OK (0) or a negative CP_ERR_* code.  All
 * validation happens before anything is enqueued: a call that fails enqueues
 * no work and writes nothing.  No C++ exception crosses this interface.
 * Block-table entries live on the device and are normally not inspected on
 * the host; entries a batch reads must be in [0, num_blocks).  With the
 * environment variable CP_DEBUG=1, cp_kv_append and cp_attn_mixed first wait
 * for the stream, copy the entries the batch reads to the host, check them
 * (cp_check_block_tables) and return CP_ERR_BAD_META without enqueueing
 * anything if one is out of range; every launch is then followed by a stream
 * synchronisation so a kernel error surfaces at the call that caused it.
 *
 * Asynchrony: both compute calls are asynchronous on `stream` (a hipStream_t;
 * NULL is the legacy default stream).  cp_attn_mixed reads only the caches:
 * append the batch's K/V first, on the same stream.
 */
#ifndef CP_ATTN_H
#define CP_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CP_OK 0
#define CP_ERR_INVALID_ARG (-1) /* null pointer, bad size, misaligned buffer   */
#define CP_ERR_BAD_META (-2)    /* malformed row metadata                      */
#define CP_ERR_WORKSPACE (-3)   /* workspace smaller than cp_workspace_bytes() */
#define CP_ERR_UNSUPPORTED (-4) /* head_dim / block_size / group not supported */
#define CP_ERR_HIP (-5)         /* a HIP runtime call failed                   */

/* One scheduled row: a decode step (chunk_len == 1 at the end of a finished
 * prompt) or a prefill chunk.  Required: chunk_start >= 0, chunk_len >= 0,
 * ctx_len == chunk_start + chunk_len, ctx_len <= max_blocks_per_req *
 * block_size, 0 <= req_id < num_reqs_in_table, and no req_id twice in one
 * batch (one chunk per request per round, Sec. 3.1.3).  A row with
 * chunk_len == 0 is a legal no-op (Algorithm 1 and the APC rule of Eq. 14
 * may assign a zero chunk).  Rows may come in any order. */
typedef struct {
    int32_t req_id;
    int32_t chunk_start; /* tokens of this request already in the cache     */
    int32_t chunk_len;   /* new tokens processed in this iteration          */
    int32_t ctx_len;     /* keys visible to the row's last query            */
} cp_row_meta;

/* Geometry of the attention layer and of the paged pool.  Supported:
 * head_dim in {64, 128}; block_size in {16, 32}; num_q_heads / num_kv_heads
 * in {1, 2, 4, 8}; sm_scale finite and > 0 (1/sqrt(head_dim) is usual). */
typedef struct {
    int32_t num_q_heads;
    int32_t num_kv_heads;
    int32_t head_dim;
    int32_t block_size;
    int32_t num_blocks;
    int32_t max_blocks_per_req;
    int32_t num_reqs_in_table;
    float sm_scale;
} cp_attn_desc;

/* Library version as major*10000 + minor*100 + patch. */
int cp_version(void);

/* Static string for a CP_* code ("unknown error" for anything else). */
const char *cp_strerror(int code);

/* Host-only check of the block-table entries a batch reads: for every row,
 * entries [0, ceil(ctx_len / block_size)) of row req_id of block_tables_host
 * (a host copy of the int32 [num_reqs_in_table][max_blocks_per_req] table)
 * must lie in [0, num_blocks).  Returns CP_OK, the code cp_check_batch would
 * return for desc/rows, CP_ERR_INVALID_ARG for a null table, or
 * CP_ERR_BAD_META for an entry out of range.  Reads nothing else. */
int cp_check_block_tables(const cp_attn_desc *desc, const int32_t *block_tables_host,
                          const cp_row_meta *rows, int32_t n_rows);

/* Workspace bytes cp_attn_mixed and cp_kv_append need for this batch, or 0 if
 * desc/rows are invalid (call cp_check_batch for the reason).  Depends only
 * on desc and the rows' metadata, never on tensor contents. */
size_t cp_workspace_bytes(const cp_attn_desc *desc, const cp_row_meta *rows, int32_t n_rows);

/* Host-only validation of desc and rows; returns CP_OK or the code the
 * compute calls would return for them. */
int cp_check_batch(const cp_attn_desc *desc, const cp_row_meta *rows, int32_t n_rows);

/* Paged append: for every row and j < chunk_len, position p = chunk_start + j
 * of request req_id receives token t's K and V for every kv head:
 *   k_cache[bt[req][p / B]][h][p % B][:]  = k_new[t][h][:]
 *   v_cache[bt[req][p / B]][h][:][p % B]  = v_new[t][h][:]
 * A bit copy; every other cache slot is left untouched. */
int cp_kv_append(const cp_attn_desc *desc, const void *k_new, const void *v_new, void *k_cache,
                 void *v_cache, const int32_t *block_tables, const cp_row_meta *rows,
                 int32_t n_rows, void *ws, size_t ws_bytes, void *stream);

/* Mixed prefill/decode causal attention over the paged cache (definition in
 * the file header).  Writes out[T][Hq][D]; reads q, the caches and the
 * tables.  Rows with chunk_len >= L run on the bf16-MFMA chunk kernel, and
 * shorter rows on the split-K decode kernel, one query token at a time, each
 * over keys [0, its position]; L is 2 unless the environment variable
 * CP_PREFILL_MIN_LEN sets it (clamped to [2, 64], read on every call; every
 * value gives the same definition).  Long key ranges are split and merged by
 * a log-sum-exp pass.  When a step has both kinds of rows, the decode work
 * runs inside the prefill launch (workgroups streaming K/V beside the
 * workgroups on the matrix cores) unless CP_FUSE_DECODE=0 gives it a launch
 * of its own; CP_FUSE_DECODE 1 / 2 / 3 / 4 place those workgroups after /
 * before / spread among / merged longest first with the prefill tiles (4 is
 * the default); outputs are the same bits.  Workgroups sharing a K/V range
 * are dealt to one XCD unless that leaves the XCDs unbalanced (few kv heads),
 * when the planner cuts them into runs (CP_XCD_BALANCE_TOL, CP_XCD_PIECE_DIV;
 * placement only, outputs are the same bits). */
int cp_attn_mixed(const cp_attn_desc *desc, const void *q, const void *k_cache,
                  const void *v_cache, const int32_t *block_tables, const cp_row_meta *rows,
                  int32_t n_rows, void *out, void *ws, size_t ws_bytes, void *stream);

/* One step: cp_kv_append followed by cp_attn_mixed on the same rows, with
 * the same results bit for bit, in fewer launches: when the append's span
 * list fits the kernel arguments (at most 200 spans of one request and block),
 * the attention plan's copy into ws runs inside the append launch, so its
 * trip over PCIe overlaps the append; otherwise the two calls run in turn.
 * Arguments as for the two calls (one workspace for both, sized by
 * cp_workspace_bytes); same checks and codes, nothing enqueued on error. */
int cp_step_mixed(const cp_attn_desc *desc, const void *q, const void *k_new, const void *v_new,
                  void *k_cache, void *v_cache, const int32_t *block_tables,
                  const cp_row_meta *rows, int32_t n_rows, void *out, void *ws, size_t ws_bytes,
                  void *stream);

/* A batch's attention plan, made once and run several times: the layers of
 * one model iteration share rows, block tables and plan, and only q, the
 * caches and out change.  Plain data filled by cp_attn_prepare and owned by
 * the caller; the work lists it describes live in the workspace it was
 * prepared in, so it stays valid while nothing but cp_attn_run writes that
 * workspace (give cp_kv_append its own). */
typedef struct {
    cp_attn_desc desc;            /* the geometry it was made for             */
    int64_t tokens;               /* scheduled tokens T of the batch          */
    int64_t ws_bytes;             /* workspace bytes it occupies              */
    /* work records of the 128-row and 256-row prefill launches (one
     * workgroup each, idle padding included), decode items, merge groups */
    int32_t n_prefill_items, n_prefill_wide_items, n_decode, n_merge;
    int64_t off_prefill, off_prefill_wide, off_decode, off_merge;
    int64_t off_part_o, off_part_lse;  /* byte offsets in ws */
    int64_t partial_rows;         /* fp32 partial rows of split key ranges    */
    int32_t decode_in_prefill;    /* 0: decode items have their own launch;
                                   * 1 / 2: they run inside the 128-row / 256-row
                                   * prefill launch, whose record list then
                                   * names them                                */
    int32_t reserved;             /* 0                                         */
} cp_attn_plan;

/* Validates the batch, plans it and uploads the plan into ws (asynchronous on
 * stream); fills *plan.  Same checks and codes as cp_attn_mixed.  An empty
 * batch gives a plan whose runs do nothing. */
int cp_attn_prepare(const cp_attn_desc *desc, const cp_row_meta *rows, int32_t n_rows,
                    void *ws, size_t ws_bytes, void *stream, cp_attn_plan *plan);

/* cp_attn_mixed for a prepared batch: the same kernels on the same plan, so
 * the output equals cp_attn_mixed's bit for bit.  ws must be the workspace
 * the plan was prepared in (ws_bytes >= plan->ws_bytes); stream order must put
 * the prepare before the run.  Every list the plan names (its offset plus
 * its length times the item size) must lie inside plan->ws_bytes, else
 * CP_ERR_INVALID_ARG and nothing is enqueued; a decode block of a prefill
 * record list that names no decode unit of the plan does nothing.  It only
 * enqueues kernel launches (no copy, allocation or wait, unless CP_DEBUG or
 * the per-kernel profile is on), so a caller may capture it in a HIP graph
 * and replay it while the plan, the workspace and the buffers stay where they
 * were at capture. */
int cp_attn_run(const cp_attn_plan *plan, const void *q, const void *k_cache,
                const void *v_cache, const int32_t *block_tables, void *out, void *ws,
                size_t ws_bytes, void *stream);

/* Plan summary for diagnostics and tests (host only, enqueues nothing).
 * counts[0..5] receive: prefill work items, decode work items, merge groups,
 * partial rows, workspace bytes, decode blocks per split. */
int cp_plan_summary(const cp_attn_desc *desc, const cp_row_meta *rows, int32_t n_rows,
                    int64_t counts[6]);

/* Host-only copy of the plan's work items, for coverage tests.  Each item is
 * 8 int32: {kind (0 prefill, 1 decode), first token, tokens, first position,
 * req_id, kv head, key begin, key end}.  Writes min(cap, n) items to items
 * and returns n (the full count), or a negative CP_ERR_* code. */
int64_t cp_plan_items(const cp_attn_desc *desc, const cp_row_meta *rows, int32_t n_rows,
                      int32_t *items, int64_t cap);

/* Host-only copy of one prefill launch's record list in dispatch order
 * (which = 0: 128-row tiles, 1: 256-row tiles), for layout tests: workgroup i
 * runs record i, 8 int32 {first token, tokens, first position, req_id, key
 * begin, key end, first partial row or -1, kv head}.  tokens == 0 marks an
 * idle record; tokens == -1 a decode block, whose first token and first
 * position fields name the decode units of its waves 0-3 and 4-7 (-1: none;
 * unit u is decode item u / num_kv_heads for kv head u % num_kv_heads).
 * Writes min(cap, n) records and returns n, or a negative CP_ERR_* code. */
int64_t cp_plan_records(const cp_attn_desc *desc, const cp_row_meta *rows, int32_t n_rows,
                        int32_t which, int32_t *recs, int64_t cap);

/* ---- Allocation-free variant of cp_attn_mixed --------------------------
 *
 * For callers that cannot allocate device memory per call: code that must
 * not call hipMalloc (under HIP graph capture, in tight serving loops, in
 * harnesses that forbid it).  cp_attn_mixed_noalloc runs the same plan and
 * kernels as cp_attn_mixed (identical output), but takes no workspace: its
 * plan lists and split partials live in a static device array of
 * CP_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends, and its plan is staged through two pinned host
 * buffers of CP_NOALLOC_PLAN_BYTES set up once per device.
 *
 * cp_noalloc_init: the set-up.  Call it once per device, with that device
 * current, before the first cp_attn_mixed_noalloc there (further calls
 * return CP_OK at once).  It takes the device address of the scratch array
 * and allocates the two pinned staging buffers; CP_ERR_HIP if that fails.
 *
 * cp_attn_mixed_noalloc: cp_attn_mixed's arguments without ws / ws_bytes,
 * same validation and codes, plus CP_ERR_WORKSPACE (nothing enqueued) when
 * the batch's workspace would exceed CP_NOALLOC_SCRATCH_BYTES or its plan
 * lists CP_NOALLOC_PLAN_BYTES (cp_workspace_bytes gives the former; the five
 * synthetic mixes of this library's benchmark need at most 42 MB), and
 * CP_ERR_INVALID_ARG when cp_noalloc_init has not run on the current device.
 * It calls no device or pinned allocator: it waits for the staging buffer's
 * previous copy, writes the plan into it, enqueues one copy and the kernels.
 * The scratch needs no clearing (the plan is uploaded whole and every
 * partial row is written before it is read).  Every call on one GPU shares
 * that GPU's scratch: calls that overlap on one GPU (different streams, or
 * threads without ordering) race; calls on one stream are ordered. */
#define CP_NOALLOC_SCRATCH_BYTES (64u << 20)
#define CP_NOALLOC_PLAN_BYTES (1u << 20)

int cp_noalloc_init(void);

int cp_attn_mixed_noalloc(const cp_attn_desc *desc, const void *q, const void *k_cache,
                          const void *v_cache, const int32_t *block_tables,
                          const cp_row_meta *rows, int32_t n_rows, void *out, void *stream);

/* Diagnostics: per-kernel GPU time.  After cp_profile_begin(), every kernel
 * the compute calls launch is bracketed by a pair of HIP events recorded on
 * the call's stream.  cp_profile_end() waits for those events and writes,
 * per kernel kind (0 append, 1 prefill, 2 decode, 3 merge), the summed
 * milliseconds into ms[4] and the launch count into launches[4]; it then
 * stops recording.  Costs one event record per launch edge; not reentrant
 * across threads. */
int cp_profile_begin(void);
int cp_profile_end(double ms[4], int64_t launches[4]);

#ifdef __cplusplus
}
#endif

#endif /* CP_ATTN_H */
