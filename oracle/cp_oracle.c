/*
 * Plain fp64 CPU oracle for one chunked-prefill scheduling iteration's
 * attention step: the paged KV append and the mixed prefill/decode causal
 * attention over the scheduled batch.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header or table with the HIP path.
 *
 * What it follows from the paper:
 *  - a request's prompt is consumed in chunks; a chunk of c_i tokens starts
 *    where the previous chunk stopped (remaining-work update, Eq. 2 and the
 *    scheduling semantics of Sec. 3.1.3), so a chunk's history depth is the
 *    "prefill processed tokens" of Table 1 / prefill_interaction of Table 2;
 *  - chunks are interleaved with single-token decode rows in one batch
 *    (Sec. 2.1, Sec. 3.1.1);
 *  - the KV cache is paged (Sec. 2.1, paged attention).
 * The paper does not write the attention formula; this file is the plain
 * definition of causal scaled-dot-product attention with grouped KV heads,
 * evaluated independently for every (row, query token, q head):
 *
 *     p      = chunk_start + j            absolute position of query j
 *     g      = h / (Hq / Hkv)             kv head of q head h
 *     s_i    = scale * sum_d q[d] * K_i[d]        i = 0 .. p
 *     o      = sum_i exp(s_i - max s) V_i / sum_i exp(s_i - max s)
 *
 * Readings where the paper is silent: ctx_len = chunk_start + chunk_len;
 * bottom-right causal alignment (query j sees keys 0..chunk_start+j);
 * kv head = floor(h / G); scale is the float32 value passed in, widened.
 *
 * Data layouts (bf16 passed as raw uint16 words):
 *   rows    int32 [n_rows][4] = {req_id, chunk_start, chunk_len, ctx_len}
 *   q       [T][Hq][D]       T = sum chunk_len, rows packed in row order
 *   k_new   [T][Hkv][D]      v_new  [T][Hkv][D]
 *   k_cache [NB][Hkv][B][D]  v_cache [NB][Hkv][D][B]
 *   bt      int32 [R][MBR]   logical block -> physical block
 *   out     double [T][Hq][D]  (or [n_sel][D] when a selection is given)
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int Hq, Hkv, D, B, NB, R, MBR;
} geom_t;

static double bf16_value(uint16_t w)
{
    uint32_t bits = ((uint32_t)w) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static size_t k_slot(const geom_t *g, int64_t blk, int h, int slot, int d)
{
    return (((size_t)blk * g->Hkv + h) * g->B + slot) * g->D + d;
}

static size_t v_slot(const geom_t *g, int64_t blk, int h, int slot, int d)
{
    return (((size_t)blk * g->Hkv + h) * g->D + d) * g->B + slot;
}

/* physical block holding logical position pos of request req */
static int64_t block_of(const geom_t *g, const int32_t *bt, int req, int pos)
{
    return bt[(size_t)req * g->MBR + pos / g->B];
}

static int check_rows(const geom_t *g, const int32_t *rows, int n_rows)
{
    for (int r = 0; r < n_rows; ++r) {
        const int32_t *m = rows + 4 * r;
        if (m[0] < 0 || m[0] >= g->R || m[1] < 0 || m[2] < 0 || m[3] != m[1] + m[2])
            return -1;
        if (m[3] > g->MBR * g->B)
            return -1;
    }
    return 0;
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/*
 * Append: every new token t of row r lands at logical position
 * p = chunk_start + j, i.e. slot p mod B of physical block bt[req][p / B],
 * for every kv head.  A bit copy; every other slot is left as it was.
 */
int oracle_kv_append(int Hkv, int D, int B, int NB, int R, int MBR,
                     const uint16_t *k_new, const uint16_t *v_new,
                     uint16_t *k_cache, uint16_t *v_cache,
                     const int32_t *bt, const int32_t *rows, int n_rows)
{
    geom_t g = {Hkv, Hkv, D, B, NB, R, MBR};
    if (check_rows(&g, rows, n_rows))
        return -1;
    int64_t tok = 0;
    for (int r = 0; r < n_rows; ++r) {
        const int req = rows[4 * r], start = rows[4 * r + 1], len = rows[4 * r + 2];
        for (int j = 0; j < len; ++j, ++tok) {
            const int pos = start + j;
            const int64_t blk = block_of(&g, bt, req, pos);
            if (blk < 0 || blk >= NB)
                return -2;
            for (int h = 0; h < Hkv; ++h)
                for (int d = 0; d < D; ++d) {
                    const size_t src = ((size_t)tok * Hkv + h) * D + d;
                    k_cache[k_slot(&g, blk, h, pos % B, d)] = k_new[src];
                    v_cache[v_slot(&g, blk, h, pos % B, d)] = v_new[src];
                }
        }
    }
    return 0;
}

/* attention output of one (row, query j, q head h) into o[0..D) */
static void attend_one(const geom_t *g, double scale, const uint16_t *q_row,
                       const uint16_t *k_cache, const uint16_t *v_cache,
                       const int32_t *bt, int req, int pos, int h, double *s, double *o)
{
    const int kvh = h / (g->Hq / g->Hkv);
    const int n_keys = pos + 1;
    double smax = -INFINITY;
    for (int i = 0; i < n_keys; ++i) {
        const int64_t blk = block_of(g, bt, req, i);
        double dot = 0.0;
        for (int d = 0; d < g->D; ++d)
            dot += bf16_value(q_row[d]) * bf16_value(k_cache[k_slot(g, blk, kvh, i % g->B, d)]);
        s[i] = scale * dot;
        if (s[i] > smax)
            smax = s[i];
    }
    double denom = 0.0;
    for (int d = 0; d < g->D; ++d)
        o[d] = 0.0;
    for (int i = 0; i < n_keys; ++i) {
        const int64_t blk = block_of(g, bt, req, i);
        const double w = exp(s[i] - smax);
        denom += w;
        for (int d = 0; d < g->D; ++d)
            o[d] += w * bf16_value(v_cache[v_slot(g, blk, kvh, i % g->B, d)]);
    }
    for (int d = 0; d < g->D; ++d)
        o[d] /= denom;
}

/*
 * Attention over the batch.  sel == NULL: every (token, q head), out is
 * [T][Hq][D].  Otherwise sel holds n_sel flat indices t*Hq + h and out is
 * [n_sel][D].  Reads only the caches (the append must have run first).
 */
int oracle_attn(int Hq, int Hkv, int D, int B, int NB, int R, int MBR, float sm_scale,
                const uint16_t *q, const uint16_t *k_cache, const uint16_t *v_cache,
                const int32_t *bt, const int32_t *rows, int n_rows,
                const int64_t *sel, int64_t n_sel, double *out)
{
    geom_t g = {Hq, Hkv, D, B, NB, R, MBR};
    if (Hkv <= 0 || Hq % Hkv != 0 || check_rows(&g, rows, n_rows))
        return -1;
    int64_t T = 0;
    int max_ctx = 1;
    for (int r = 0; r < n_rows; ++r) {
        T += rows[4 * r + 2];
        if (rows[4 * r + 3] > max_ctx)
            max_ctx = rows[4 * r + 3];
    }
    /* token -> row map */
    int32_t *row_of = (int32_t *)malloc(sizeof(int32_t) * (size_t)(T > 0 ? T : 1));
    int64_t *off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n_rows + 1));
    if (!row_of || !off) {
        free(row_of);
        free(off);
        return -3;
    }
    off[0] = 0;
    for (int r = 0; r < n_rows; ++r) {
        off[r + 1] = off[r] + rows[4 * r + 2];
        for (int64_t t = off[r]; t < off[r + 1]; ++t)
            row_of[t] = r;
    }
    for (int r = 0; r < n_rows; ++r) {
        const int req = rows[4 * r];
        for (int i = 0; i < rows[4 * r + 3]; i += B) {
            const int64_t blk = block_of(&g, bt, req, i);
            if (blk < 0 || blk >= NB) {
                free(row_of);
                free(off);
                return -2;
            }
        }
    }
    const int64_t n_work = sel ? n_sel : T * Hq;
    for (int64_t w = 0; w < n_work; ++w) {
        const int64_t flat = sel ? sel[w] : w;
        if (flat < 0 || flat >= T * Hq) {
            free(row_of);
            free(off);
            return -4;
        }
    }
    const double scale = (double)sm_scale;
    int err = 0;
#pragma omp parallel
    {
        double *s = (double *)malloc(sizeof(double) * (size_t)max_ctx);
        if (!s) {
#pragma omp atomic write
            err = -3;
        }
#pragma omp for schedule(dynamic, 4)
        for (int64_t w = 0; w < n_work; ++w) {
            if (!s)
                continue;
            const int64_t flat = sel ? sel[w] : w;
            const int64_t t = flat / Hq;
            const int h = (int)(flat % Hq);
            const int r = row_of[t];
            const int pos = rows[4 * r + 1] + (int)(t - off[r]);
            attend_one(&g, scale, q + (size_t)flat * D, k_cache, v_cache, bt, rows[4 * r],
                       pos, h, s, out + (size_t)w * D);
        }
        free(s);
    }
    free(row_of);
    free(off);
    return err;
}
