/*
 * cp_layer.h — C ABI of the element-wise kernels that surround the
 * attention step in one decoder layer of a Qwen3 / Llama-style model, for
 * AMD Instinct MI355X (gfx950).  The paper's latency predictor and its
 * target T* are defined on the whole model iteration (Sec. 3.2.1; T* = 105 ms
 * for Qwen3-8B in Sec. 4.4), so measuring what the scheduler controls needs
 * the layer around cp_kv_append / cp_attn_mixed:
 *
 *   x -> RMSNorm -> QKV projection -> cpl_qkv_rope -> cp_kv_append,
 *        cp_attn_mixed -> O projection (+ x) -> RMSNorm -> gate/up
 *        projection -> cpl_swiglu -> down projection (+ residual)
 *
 * The projections are plain GEMMs: cpl_gemm (LDS-tiled MFMA) and, for
 * decode-sized batches, cpl_gemm_skinny, which streams the weights itself.  The paper does not describe the model; the layer
 * follows the published Qwen3 architecture (RMSNorm, per-head RMSNorm on
 * queries and keys before rotary embedding, SwiGLU feed-forward).
 *
 * Conventions: bf16 tensors are dense and row-major with 16-byte aligned
 * rows; arithmetic is fp32 (the rotation angle is formed in turns and
 * reduced to [-1/2, 1/2] turn in fp64 before the hardware's fp32 sine and
 * cosine) and results are rounded to bf16 (nearest even).  All pointers are device pointers owned by the
 * caller; nothing is allocated.  Calls are asynchronous on `stream`.  Return
 * CP_OK or CP_ERR_INVALID_ARG (null pointer, misaligned buffer, size out of
 * range), CP_ERR_UNSUPPORTED (head_dim), CP_ERR_HIP (launch failure);
 * a call that fails enqueues nothing.
 */
#ifndef CP_LAYER_H
#define CP_LAYER_H

#include <stddef.h>
#include <stdint.h>

#include "cp_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* RMSNorm over each row: out[r][i] = x[r][i] * w[i] / sqrt(mean_i(x[r][i]^2) + eps).
 * x, out [n_rows][width] (may alias), w [width]; 8 <= width <= 32768,
 * width % 8 == 0, n_rows >= 0, eps > 0. */
int cpl_rmsnorm(const void* x, const void* w, void* out, int32_t n_rows, int32_t width,
                float eps, void* stream);

/* Splits the fused projection qkv[T][(hq + 2*hkv) * head_dim] (q heads, then
 * k heads, then v heads) into q[T][hq][head_dim], k[T][hkv][head_dim] and
 * v[T][hkv][head_dim].  Every q head is RMS-normalised over head_dim with
 * q_norm_w[head_dim] and every k head with k_norm_w[head_dim] (eps as
 * above), then rotated to position positions[t] (int32, device, >= 0):
 * elements d and d + head_dim/2 form a pair turned by the angle
 * positions[t] * theta^(-2d/head_dim), d < head_dim/2.  v is copied.
 * head_dim in {64, 128}; theta > 1. */
int cpl_qkv_rope(const void* qkv, const void* q_norm_w, const void* k_norm_w,
                 const int32_t* positions, int32_t n_tokens, int32_t hq, int32_t hkv,
                 int32_t head_dim, double theta, float eps, void* q, void* k, void* v,
                 void* stream);

/* SwiGLU: out[t][i] = silu(gu[t][i]) * gu[t][inter + i], silu(g) = g / (1 + e^-g);
 * gu [T][2*inter], out [T][inter]; inter % 8 == 0. */
int cpl_swiglu(const void* gu, void* out, int32_t n_tokens, int32_t inter, void* stream);

/* Projection: c[M][N] = a[M][K] . w[N][K]^T (+ r[M][N]), bf16 in and out, fp32
 * accumulation on the matrix cores (v_mfma_f32_32x32x16_bf16), for batches of
 * any size (the layer runs its QKV and output projections on it above the
 * skinny kernel's batch sizes).  M >= 1, N % 128 == 0, K % 32 == 0; a, w, c,
 * r and ws 16-byte aligned; r may be NULL or equal to c (in-place residual
 * add); a and w must not alias c.  Output tiles of 64-256 x 128-256 with K
 * staged through LDS; when the tiles alone would leave CUs idle, K is split
 * into slices whose fp32 partial tiles go to ws (the caller's device
 * memory, at least cpl_gemm_workspace_bytes(m, n, k) bytes to split fully;
 * with less, or ws NULL, the split shrinks or is skipped: same definition,
 * fewer workgroups).  The environment variables CPL_GEMM_CFG (tile
 * configuration 0-7: 64x128, 128x128, 128x256, 256x128 with 32 k per stage,
 * 64x128, 128x128 with 64, 256x256 with 32 and 64) and CPL_GEMM_SPLIT
 * (slices) override the choice. */
int cpl_gemm(const void* a, const void* w, const void* r, void* c, int32_t m, int32_t n,
             int32_t k, void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes cpl_gemm uses for this shape (0: no split), or 0 if the
 * shape is unsupported. */
size_t cpl_gemm_workspace_bytes(int32_t m, int32_t n, int32_t k);

/* Projection of a small batch: c[M][N] = a[M][K] . w[N][K]^T (+ r[M][N]), bf16 in and
 * out, fp32 accumulation, for the decode-sized batches where a library GEMM
 * cannot stream the weights at memory speed.  1 <= M <= 128, N % 32 == 0,
 * K % 256 == 0; r may be NULL or equal to c (in-place residual add); a must
 * not alias c.  w is read once; a is re-read from cache by every 32-column
 * slice of the output (16-column slices when N <= 4096, M <= 32 and
 * K % 512 == 0, so that narrow projections occupy every CU). */
int cpl_gemm_skinny(const void* a, const void* w, const void* r, void* c, int32_t m, int32_t n,
                    int32_t k, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CP_LAYER_H */
