// Element-wise kernels around the attention step of one decoder layer
// (include/cp_layer.h): RMSNorm, the QKV split with per-head RMSNorm and
// rotary embedding, and SwiGLU.  All three are bound by HBM traffic: each
// reads its input once and writes its output once with 16-byte coalesced
// accesses.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "cp_layer.h"

namespace {

constexpr int kThreads = 256;

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ __forceinline__ uint16_t f32_to_bf16(float a) {
  return __builtin_bit_cast(uint16_t, (__bf16)a);  // nearest even
}

__device__ __forceinline__ float lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint32_t pack(float a, float b) {
  return (uint32_t)f32_to_bf16(a) | ((uint32_t)f32_to_bf16(b) << 16);
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

__device__ __forceinline__ float sumsq8(const uint4& a) {
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) s += lo(w[i]) * lo(w[i]) + hi(w[i]) * hi(w[i]);
  return s;
}

// One block per row.  x and out may alias: every element is read and then
// written by the same thread, after the block-wide reduction barrier.
__global__ __launch_bounds__(kThreads) void rmsnorm_kernel(const uint4* x, const uint4* w,
                                                           uint4* out, int width8,
                                                           float inv_width, float eps) {
  const size_t row = blockIdx.x;
  const uint4* xr = x + row * width8;
  uint4* orow = out + row * width8;
  float ss = 0.f;
  for (int v = threadIdx.x; v < width8; v += kThreads) ss += sumsq8(xr[v]);
  ss = wave_sum(ss);
  __shared__ float part[kThreads / 64];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  float total = 0.f;
#pragma unroll
  for (int i = 0; i < kThreads / 64; ++i) total += part[i];
  const float scale = 1.0f / sqrtf(total * inv_width + eps);
  for (int v = threadIdx.x; v < width8; v += kThreads) {
    const uint4 a = xr[v], g = w[v];
    const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, gw[4] = {g.x, g.y, g.z, g.w};
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      o[i] = pack(lo(aw[i]) * scale * lo(gw[i]), hi(aw[i]) * scale * hi(gw[i]));
    orow[v] = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// One wave per (token, group of 64 / (D/8) heads) of the fused projection.
// A head is D/8 consecutive lanes of 8 elements each (16-byte loads and
// stores); lane j < D/16 of a head holds elements of the first half and lane
// j + D/16 their rotation partners, and the two swap their raw words with
// one cross-lane exchange.  Heads [0, hq) are queries, [hq, hq + hkv) keys,
// the rest values.
template <int D>
__global__ __launch_bounds__(kThreads) void qkv_rope_kernel(
    const uint4* __restrict qkv, const uint4* __restrict qw, const uint4* __restrict kw,
    const int32_t* __restrict positions, int n_tokens, int hq, int hkv, double step,
    double step8, float eps, uint4* __restrict q, uint4* __restrict k, uint4* __restrict v) {
  constexpr int L = D / 8, HPW = 64 / L, HALF = L / 2;
  const int nh = hq + 2 * hkv;
  const int groups = (nh + HPW - 1) / HPW;
  const int64_t g = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (g >= (int64_t)n_tokens * groups) return;  // whole wave
  const int t = (int)(g / groups), h0 = (int)(g % groups) * HPW;
  const int lane = threadIdx.x & 63, sub = lane % L, hh = h0 + lane / L;
  const bool live = hh < nh;
  const uint4 a = live ? qkv[((size_t)t * nh + hh) * L + sub] : make_uint4(0, 0, 0, 0);
  if (h0 >= hq + hkv) {  // values only (wave-uniform)
    if (live) v[((size_t)t * hkv + (hh - hq - hkv)) * L + sub] = a;
    return;
  }
  uint4 b;  // the partner lane's raw words
  b.x = __shfl_xor(a.x, HALF, 64);
  b.y = __shfl_xor(a.y, HALF, 64);
  b.z = __shfl_xor(a.z, HALF, 64);
  b.w = __shfl_xor(a.w, HALF, 64);
  float ss = sumsq8(a);
#pragma unroll
  for (int m = 1; m < L; m <<= 1) ss += __shfl_xor(ss, m, 64);
  const float scale = 1.0f / sqrtf(ss / (float)D + eps);
  if (!live) return;
  if (hh >= hq + hkv) {
    v[((size_t)t * hkv + (hh - hq - hkv)) * L + sub] = a;
    return;
  }
  const bool is_q = hh < hq;
  const uint4* w = is_q ? qw : kw;
  const uint4 wo = w[sub], wp = w[sub ^ HALF];
  // frequency of element e in turns per position:
  // theta^(-2 (8 (sub mod D/16) + e) / D) / (2 pi) = step8^(sub mod D/16) * step^e / (2 pi),
  // by fp64 products; the angle is reduced to [-1/2, 1/2] turn in fp64 and its
  // sine and cosine taken by the hardware's turn-based instructions
  const int mlo = sub % HALF;
  double f = 0.15915494309189533576888376337251, p = step8;
#pragma unroll
  for (int bit = 0; bit < 3; ++bit) {
    if (mlo & (1 << bit)) f *= p;
    p *= p;
  }
  const double pos = (double)positions[t];
  const float sgn = sub < HALF ? -1.f : 1.f;
  const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, bw[4] = {b.x, b.y, b.z, b.w};
  const uint32_t wow[4] = {wo.x, wo.y, wo.z, wo.w}, wpw[4] = {wp.x, wp.y, wp.z, wp.w};
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float r2[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const double turns = pos * f;
      f *= step;
      const float r = (float)(turns - rint(turns));
      const float sn = __builtin_amdgcn_sinf(r), cs = __builtin_amdgcn_cosf(r);
      const float xo = (h ? hi(aw[i]) : lo(aw[i])) * scale * (h ? hi(wow[i]) : lo(wow[i]));
      const float xp = (h ? hi(bw[i]) : lo(bw[i])) * scale * (h ? hi(wpw[i]) : lo(wpw[i]));
      r2[h] = xo * cs + sgn * (xp * sn);
    }
    o[i] = pack(r2[0], r2[1]);
  }
  const uint4 out = make_uint4(o[0], o[1], o[2], o[3]);
  if (is_q)
    q[((size_t)t * hq + hh) * L + sub] = out;
  else
    k[((size_t)t * hkv + (hh - hq)) * L + sub] = out;
}

__global__ __launch_bounds__(kThreads) void swiglu_kernel(const uint4* __restrict gu,
                                                          uint4* __restrict out, int inter8,
                                                          int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= n) return;
  const int64_t t = i / inter8, c = i % inter8;
  const uint4 g = gu[t * 2 * inter8 + c], u = gu[t * 2 * inter8 + inter8 + c];
  const uint32_t gw[4] = {g.x, g.y, g.z, g.w}, uw[4] = {u.x, u.y, u.z, u.w};
  uint32_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float g0 = lo(gw[j]), g1 = hi(gw[j]);
    o[j] = pack(g0 / (1.0f + __expf(-g0)) * lo(uw[j]), g1 / (1.0f + __expf(-g1)) * hi(uw[j]));
  }
  out[i] = make_uint4(o[0], o[1], o[2], o[3]);
}


// Skinny GEMM C[M][N] = A[M][K] * W[N][K]^T (+ R), M <= 32 * MB: every weight
// byte is streamed from HBM once while the activations stay in L2.  A
// workgroup owns 32 output columns; its four waves take a quarter of K
// each, with v_mfma_f32_32x32x16_bf16 on W rows (the 32 "m" rows) against
// activation rows (the 32 "n" columns), then add their partial sums through
// LDS.
//
// The matrix core wants lane l to hold 16 bytes of W row l % 32, so loading
// its operands straight from memory touches 32 rows with 32-byte pieces per
// instruction.  Instead each wave reads a batch of U k-steps as whole
// 32U-byte row segments (2U lanes per row, 32 / U rows per instruction) with
// non-temporal loads, parks them in its own slice of LDS and reads its MFMA
// operands from there: the weight stream then moves in whole 128-byte
// (U = 4) or 256-byte (U = 8) runs per row, which is what lets it approach
// the HBM rate.  Only the
// wave that writes a slice reads it, so no barrier is needed until the final
// reduction.  Activations are read directly (they are small and cached).
template <int MB, int U>
__global__ __launch_bounds__(256) void gemm_skinny_kernel(const uint4* __restrict__ A,
                                                          const uint4* __restrict__ W,
                                                          const uint16_t* R, uint16_t* C, int M,
                                                          int N, int K) {
  typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
  typedef float f32x16_t __attribute__((ext_vector_type(16)));
  constexpr int kRowPad = 33;           // floats per reduction row (bank spread)
  constexpr int kPitch = 2 * U + 1;     // uint4 per staged row (bank spread)
  constexpr int kLanesPerRow = 2 * U, kRowsPerLoad = 64 / kLanesPerRow;
  constexpr int kStage = 4 * 32 * kPitch * 16, kRed = 4 * 32 * MB * kRowPad * 4;
  __shared__ __align__(16) char smem[kStage > kRed ? kStage : kRed];
  uint4* stage = reinterpret_cast<uint4*>(smem) + (threadIdx.x >> 6) * 32 * kPitch;
  auto red = reinterpret_cast<float(*)[32 * MB][kRowPad]>(smem);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * 32;
  const int kq = K / 4, kb = wave * kq;
  const int K8 = K / 8;  // uint4 per row
  const int lr = lane & 31, lg = lane >> 5;
  const int rin = lane / kLanesPerRow, col = lane % kLanesPerRow;
  const u32x4_t* wsrc =
      reinterpret_cast<const u32x4_t*>(W + (int64_t)(n0 + rin) * K8 + (kb >> 3) + col);
  const uint4* arow[MB];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
    arow[rb] = A + (int64_t)min(rb * 32 + lr, M - 1) * K8 + (kb >> 3) + lg;
  f32x16_t acc[MB];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[rb][r] = 0.f;
  u32x4_t wr[U];  // the next batch, rows rin + kRowsPerLoad * i
  auto load = [&](int b) {
#pragma unroll
    for (int i = 0; i < U; ++i)
      wr[i] = __builtin_nontemporal_load(wsrc + (int64_t)kRowsPerLoad * i * K8 + b * 2 * U);
  };
  const int batches = kq / (16 * U);
  load(0);
  for (int b = 0; b < batches; ++b) {
#pragma unroll
    for (int i = 0; i < U; ++i)
      stage[(kRowsPerLoad * i + rin) * kPitch + col] = make_uint4(wr[i][0], wr[i][1], wr[i][2], wr[i][3]);
    uint4 wc[U], ac[U][MB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      wc[u] = stage[lr * kPitch + 2 * u + lg];
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) ac[u][rb] = arow[rb][b * 2 * U + 2 * u];
    }
    if (b + 1 < batches) load(b + 1);
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int rb = 0; rb < MB; ++rb)
        acc[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, wc[u]), __builtin_bit_cast(bf16x8_t, ac[u][rb]),
            acc[rb], 0, 0, 0);
  }
  __syncthreads();  // every wave is done with its staging slice
  // D[i][j] = sum_k W[n0 + i][k] A[32 rb + j][k]: lane holds j = lane % 32,
  // register r holds i = 8 (r / 4) + 4 (lane / 32) + r % 4
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      red[wave][rb * 32 + lr][8 * (r >> 2) + 4 * lg + (r & 3)] = acc[rb][r];
  __syncthreads();
  for (int idx = threadIdx.x; idx < 32 * MB * 32; idx += 256) {
    const int j = idx >> 5, i = idx & 31;
    if (j >= M) break;  // rows are visited in increasing order
    float v = red[0][j][i] + red[1][j][i] + red[2][j][i] + red[3][j][i];
    const int64_t o = (int64_t)j * N + n0 + i;
    if (R) v += bf16_to_f32(R[o]);
    C[o] = f32_to_bf16(v);
  }
}

// The same product with 16 output columns per workgroup
// (v_mfma_f32_16x16x32_bf16), for projections whose N / 32 column slices
// would leave CUs idle; M <= 16 * MB.  A wave's batch is 4 k-steps of 32: 16
// rows of 256 bytes (4 rows per load instruction), staged in its LDS slice
// as above.  Lane l holds W row l % 16, k-chunk l / 16 of each step, and
// activation row l % 16 of the same chunk.
template <int MB>
__global__ __launch_bounds__(256) void gemm_skinny16_kernel(const uint4* __restrict__ A,
                                                            const uint4* __restrict__ W,
                                                            const uint16_t* R, uint16_t* C, int M,
                                                            int N, int K) {
  typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
  typedef float f32x4_t __attribute__((ext_vector_type(4)));
  constexpr int U = 4;                 // k-steps of 32 per batch
  constexpr int kPitch = 4 * U + 1;    // uint4 per staged row (256 bytes + pad)
  constexpr int kRowPad = 17;          // floats per reduction row
  constexpr int kStage = 4 * 16 * kPitch * 16, kRed = 4 * 16 * MB * kRowPad * 4;
  __shared__ __align__(16) char smem[kStage > kRed ? kStage : kRed];
  uint4* stage = reinterpret_cast<uint4*>(smem) + (threadIdx.x >> 6) * 16 * kPitch;
  auto red = reinterpret_cast<float(*)[16 * MB][kRowPad]>(smem);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * 16;
  const int kq = K / 4, kb = wave * kq;
  const int K8 = K / 8;
  const int lr = lane & 15, lg = lane >> 4;        // MFMA row, k-chunk
  const int rin = lane >> 4, col = lane & 15;      // staging: row within a load, 16-byte column
  const u32x4_t* wsrc =
      reinterpret_cast<const u32x4_t*>(W + (int64_t)(n0 + rin) * K8 + (kb >> 3) + col);
  const uint4* arow[MB];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
    arow[rb] = A + (int64_t)min(rb * 16 + lr, M - 1) * K8 + (kb >> 3) + lg;
  f32x4_t acc[MB];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[rb][r] = 0.f;
  u32x4_t wr[4];  // the next batch, rows rin + 4 i
  auto load = [&](int b) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      wr[i] = __builtin_nontemporal_load(wsrc + (int64_t)4 * i * K8 + b * 4 * U);
  };
  const int batches = kq / (32 * U);
  load(0);
  for (int b = 0; b < batches; ++b) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      stage[(4 * i + rin) * kPitch + col] = make_uint4(wr[i][0], wr[i][1], wr[i][2], wr[i][3]);
    uint4 wc[U], ac[U][MB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      wc[u] = stage[lr * kPitch + 4 * u + lg];
#pragma unroll
      for (int rb = 0; rb < MB; ++rb) ac[u][rb] = arow[rb][b * 4 * U + 4 * u];
    }
    if (b + 1 < batches) load(b + 1);
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int rb = 0; rb < MB; ++rb)
        acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8_t, wc[u]), __builtin_bit_cast(bf16x8_t, ac[u][rb]),
            acc[rb], 0, 0, 0);
  }
  __syncthreads();  // every wave is done with its staging slice
  // D[i][j] = sum_k W[n0 + i][k] A[16 rb + j][k]: lane holds j = lane % 16,
  // register r holds i = 4 (lane / 16) + r
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int r = 0; r < 4; ++r) red[wave][rb * 16 + lr][4 * lg + r] = acc[rb][r];
  __syncthreads();
  for (int idx = threadIdx.x; idx < 16 * MB * 16; idx += 256) {
    const int j = idx >> 4, i = idx & 15;
    if (j >= M) break;  // rows are visited in increasing order
    float v = red[0][j][i] + red[1][j][i] + red[2][j][i] + red[3][j][i];
    const int64_t o = (int64_t)j * N + n0 + i;
    if (R) v += bf16_to_f32(R[o]);
    C[o] = f32_to_bf16(v);
  }
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

int launched() { return hipGetLastError() == hipSuccess ? CP_OK : CP_ERR_HIP; }

}  // namespace

extern "C" {

int cpl_rmsnorm(const void* x, const void* w, void* out, int32_t n_rows, int32_t width,
                float eps, void* stream) {
  if (n_rows < 0 || width < 8 || width > 32768 || width % 8 != 0 || !(eps > 0.f))
    return CP_ERR_INVALID_ARG;
  if (n_rows == 0) return CP_OK;
  if (!x || !w || !out || !aligned16(x) || !aligned16(w) || !aligned16(out))
    return CP_ERR_INVALID_ARG;
  (void)hipGetLastError();
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(n_rows), dim3(kThreads), 0, (hipStream_t)stream,
                     (const uint4*)x, (const uint4*)w, (uint4*)out, width / 8, 1.0f / width, eps);
  return launched();
}

int cpl_qkv_rope(const void* qkv, const void* q_norm_w, const void* k_norm_w,
                 const int32_t* positions, int32_t n_tokens, int32_t hq, int32_t hkv,
                 int32_t head_dim, double theta, float eps, void* q, void* k, void* v,
                 void* stream) {
  if (head_dim != 64 && head_dim != 128) return CP_ERR_UNSUPPORTED;
  if (n_tokens < 0 || hq < 1 || hkv < 1 || hq > 1024 || hkv > 1024 || !(theta > 1.0) ||
      !(eps > 0.f))
    return CP_ERR_INVALID_ARG;
  if (n_tokens == 0) return CP_OK;
  if (!qkv || !q_norm_w || !k_norm_w || !positions || !q || !k || !v) return CP_ERR_INVALID_ARG;
  if (!aligned16(qkv) || !aligned16(q_norm_w) || !aligned16(k_norm_w) || !aligned16(q) ||
      !aligned16(k) || !aligned16(v))
    return CP_ERR_INVALID_ARG;
  const int64_t hpw = 64 / (head_dim / 8);
  const int64_t groups = (hq + 2 * hkv + hpw - 1) / hpw;
  const int64_t waves = (int64_t)n_tokens * groups;
  const int64_t blocks = (waves + kThreads / 64 - 1) / (kThreads / 64);
  if (blocks > 0x7fffffff) return CP_ERR_INVALID_ARG;
  // ratio of consecutive frequencies theta^(-2/D), and its eighth power
  const double step = exp2(-2.0 / head_dim * log2(theta));
  const double step8 = exp2(-16.0 / head_dim * log2(theta));
  (void)hipGetLastError();
  auto kern = head_dim == 128 ? qkv_rope_kernel<128> : qkv_rope_kernel<64>;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kThreads), 0, (hipStream_t)stream,
                     (const uint4*)qkv, (const uint4*)q_norm_w, (const uint4*)k_norm_w, positions,
                     n_tokens, hq, hkv, step, step8, eps, (uint4*)q, (uint4*)k, (uint4*)v);
  return launched();
}

int cpl_swiglu(const void* gu, void* out, int32_t n_tokens, int32_t inter, void* stream) {
  if (n_tokens < 0 || inter < 8 || inter % 8 != 0) return CP_ERR_INVALID_ARG;
  if (n_tokens == 0) return CP_OK;
  if (!gu || !out || !aligned16(gu) || !aligned16(out)) return CP_ERR_INVALID_ARG;
  const int64_t n = (int64_t)n_tokens * (inter / 8);
  const int64_t blocks = (n + kThreads - 1) / kThreads;
  if (blocks > 0x7fffffff) return CP_ERR_INVALID_ARG;
  (void)hipGetLastError();
  hipLaunchKernelGGL(swiglu_kernel, dim3((unsigned)blocks), dim3(kThreads), 0,
                     (hipStream_t)stream, (const uint4*)gu, (uint4*)out, inter / 8, n);
  return launched();
}

int cpl_gemm_skinny(const void* a, const void* w, const void* r, void* c, int32_t m, int32_t n,
                    int32_t k, void* stream) {
  if (m < 1 || m > 128 || n < 32 || n % 32 != 0 || k < 256 || k % 256 != 0 || k > (1 << 20))
    return CP_ERR_INVALID_ARG;
  if (!a || !w || !c || !aligned16(a) || !aligned16(w) || a == c) return CP_ERR_INVALID_ARG;
  (void)hipGetLastError();
  const dim3 grid(n / 32), block(256);
  hipStream_t s = (hipStream_t)stream;
  const uint4* A = (const uint4*)a;
  const uint4* W = (const uint4*)w;
  const uint16_t* R = (const uint16_t*)r;
  uint16_t* C = (uint16_t*)c;
  // batches of 8 k-steps (256-byte row segments) where each wave's quarter
  // of K holds whole batches, else of 4
  const bool u8 = k % 512 == 0;
  using Kernel = void (*)(const uint4*, const uint4*, const uint16_t*, uint16_t*, int, int, int);
  Kernel kern;
  // narrow projections (32-column slices would leave half the CUs idle):
  // 16-column slices, so that every CU gets one
  if (m <= 32 && u8 && n / 32 <= 128) {
    kern = m <= 16 ? gemm_skinny16_kernel<1> : gemm_skinny16_kernel<2>;
    hipLaunchKernelGGL(kern, dim3(n / 16), block, 0, s, A, W, R, C, m, n, k);
    return launched();
  }
  if (m <= 32)
    kern = u8 ? gemm_skinny_kernel<1, 8> : gemm_skinny_kernel<1, 4>;
  else if (m <= 64)
    kern = u8 ? gemm_skinny_kernel<2, 8> : gemm_skinny_kernel<2, 4>;
  else
    kern = u8 ? gemm_skinny_kernel<4, 8> : gemm_skinny_kernel<4, 4>;
  hipLaunchKernelGGL(kern, grid, block, 0, s, A, W, R, C, m, n, k);
  return launched();
}

}  // extern "C"
