// Tiled bf16 GEMM for the projections of the decoder layer around the
// attention step (include/cp_layer.h, cpl_gemm):
//     C[M][N] = A[M][K] . W[N][K]^T (+ R[M][N]),   fp32 accumulation, bf16 out.
// Both operands are K-contiguous rows, which is exactly how the matrix cores
// take their operands: with v_mfma_f32_32x32x16_bf16 every lane holds 16
// bytes (8 consecutive k) of one row of each operand.
//
// A workgroup of 4 (2 x 2) or 8 (2 x 4) waves computes a BM x BN tile of C,
// each wave a (BM/2) x (BN/2 or BN/4) part of it as blocks of 32 x 32.  The
// products are formed transposed, D^T (32 n x 32 m) = W_blk . A_blk^T, so a
// lane's accumulators hold 4 consecutive n of one m: the epilogue writes 8
// contiguous bytes per lane and row.
//
// K is walked in stages of BK.  A stage's A and W tiles are copied from
// global memory straight into LDS (global_load_lds_dwordx4: 16 bytes per
// lane, no register staging) into a ring of STAGES buffers, issued
// STAGES - 1 stages ahead of their use; one barrier per stage, after an
// explicit wait for exactly that stage's copies.  A tile row holds BK / 8
// chunks of 16 bytes; chunk c of row r is stored at chunk c ^ swz(r), so the
// 16 lanes of every phase of an operand read (rows r..r+15, one logical
// chunk) hit 16 distinct 16-byte bank groups.
//
// Split over K: with a workspace, a grid too small to fill the GPU is
// multiplied by S slices of K; slice s writes its fp32 partial tile to
// ws[s][M][N] and a second kernel adds the S partials (and R) and rounds.
//
// Workgroup order: workgroup g runs on XCD g mod 8; each XCD takes whole
// column blocks of W and walks them in row groups of up to 8 row blocks, so
// that the workgroups resident on an XCD share both A and W panels in its
// L2 (with row blocks innermost across all of M, a 4096-row A would stream
// from the last-level cache once per pair of column blocks).

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>

#include <type_traits>

#include "cp_layer.h"

namespace {

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kXcds = 8;
constexpr int kMinSliceK = 256;  // shortest K slice of a split

__device__ __forceinline__ f32x16_t mfma(uint4 a, uint4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// 16 bytes per lane from global memory into LDS at lds + 16 * lane
// (`lds` wave-uniform).  The address-space cast exists only in the device pass.
__device__ __forceinline__ void copy16_to_lds(const void* src, uint8_t* lds) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_global_load_lds(src, (lds_ptr_t)lds, 16, 0, 0);
#endif
}

// s_waitcnt with vmcnt <= N, the other counters unconstrained (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}

// waits until at most `later` stages' copies (LOADS each) are pending
template <int LOADS, int MAXLATER>
__device__ __forceinline__ void wait_stages(int later) {
  if constexpr (MAXLATER >= 3) {
    if (later >= 3) { wait_vmcnt<3 * LOADS>(); return; }
  }
  if constexpr (MAXLATER >= 2) {
    if (later >= 2) { wait_vmcnt<2 * LOADS>(); return; }
  }
  if (later >= 1) { wait_vmcnt<LOADS>(); return; }
  wait_vmcnt<0>();
}

// Compile-time loop: f(std::integral_constant<int, I>) for I in [I0, N).
template <int I0, int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I0 < N) {
    f(std::integral_constant<int, I0>());
    static_for<I0 + 1, N>(f);
  }
}

// Workgroup barrier without the memory fence of __syncthreads, which would
// also wait for the copies of later stages (the waits above are explicit).
__device__ __forceinline__ void barrier() { asm volatile("s_barrier" ::: "memory"); }

__device__ __forceinline__ uint16_t to_bf16(float a) {
  return __builtin_bit_cast(uint16_t, (__bf16)a);  // nearest even
}
__device__ __forceinline__ uint32_t pack(float a, float b) {
  return (uint32_t)to_bf16(a) | ((uint32_t)to_bf16(b) << 16);
}
__device__ __forceinline__ float lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <int BM, int BN, int BK, int STAGES, int WGM = 2, int WGN = 2>
struct GemmGeom {
  static constexpr int NW = WGM * WGN;               // waves
  static constexpr int WTM = BM / WGM, WTN = BN / WGN;  // wave tile
  static constexpr int TM = WTM / 32, TN = WTN / 32;    // 32 x 32 blocks per wave
  static constexpr int ROW = BK * 2;                 // bytes per tile row
  static constexpr int CPR = ROW / 16;               // 16-byte chunks per row
  static constexpr int RPP = 1024 / ROW;             // rows per 1 KiB copy
  static constexpr int KS = BK / 16;                 // MFMA k-steps per stage
  static constexpr int A_BYTES = BM * ROW, W_BYTES = BN * ROW;
  static constexpr int STAGE_BYTES = A_BYTES + W_BYTES;
  static constexpr int A_PW = A_BYTES / 1024 / NW, W_PW = W_BYTES / 1024 / NW;  // copies per wave
  static constexpr int LOADS = A_PW + W_PW;
  static_assert(BK == 32 || BK == 64, "BK");
  static_assert(A_PW * 1024 * NW == A_BYTES && W_PW * 1024 * NW == W_BYTES, "copies per wave");
  static_assert(LOADS * (STAGES - 1) < 64 && STAGES <= 4, "vmcnt range");
  // stored chunk of logical chunk c in row r: 16 consecutive rows (one
  // 16-lane phase of an operand read) land in 16 distinct 16-byte groups of
  // the 256-byte bank width
  __device__ static int swz(int r, int c) {
    return CPR == 8 ? c ^ ((r >> 1) & 7) : c ^ ((r >> 2) & 3);
  }
};

template <int BM, int BN, int BK, int STAGES, int WGM, int WGN>
__global__ __launch_bounds__(64 * WGM * WGN, 8 / (WGM * WGN)) void gemm_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ W, const uint16_t* R,
    uint16_t* C, float* __restrict__ part, int M, int N, int K, int S) {
  using G = GemmGeom<BM, BN, BK, STAGES, WGM, WGN>;
  constexpr int TM = G::TM, TN = G::TN, ROW = G::ROW;
  // one array per ring buffer, every access naming its array at compile
  // time: the compiler then tells the copies in flight into one buffer from
  // the operand reads of another, and waits only where they meet
  constexpr int SB = G::STAGE_BYTES;
  __shared__ __attribute__((aligned(1024))) uint8_t sb0[SB];
  __shared__ __attribute__((aligned(1024))) uint8_t sb1[SB];
  __shared__ __attribute__((aligned(1024))) uint8_t sb2[STAGES > 2 ? SB : 1024];
  __shared__ __attribute__((aligned(1024))) uint8_t sb3[STAGES > 3 ? SB : 1024];
  auto buf = [&](auto i_c) -> uint8_t* {
    constexpr int i = decltype(i_c)::value % STAGES;
    if constexpr (i == 0) return sb0;
    else if constexpr (i == 1) return sb1;
    else if constexpr (i == 2) return sb2;
    else return sb3;
  };

  // ---- tile and K slice of this workgroup.  XCD x = g mod 8 owns column
  // blocks x, x + 8, ...; its workgroups run row groups of GM row blocks
  // against all its column blocks in turn (row block fastest), so the
  // workgroups resident on an XCD at once share GM row panels of A and a
  // few column panels of W in its L2
  const int MB = (M + BM - 1) / BM, NB = N / BN;
  const int NBX = (NB + kXcds - 1) / kXcds;
  const int GM = MB % 8 == 0 ? 8 : MB % 4 == 0 ? 4 : MB;
  const int g = blockIdx.x;
  int t = g / kXcds;
  const int m_in = t % GM;
  t /= GM;
  const int sl = t % S;
  t /= S;
  const int nb = (t % NBX) * kXcds + g % kXcds;
  const int mb = (t / NBX) * GM + m_in;
  if (nb >= NB) return;
  const int m0 = mb * BM, n0 = nb * BN;
  const int kslice = K / S;  // a multiple of BK
  const int kbeg = sl * kslice;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;

  // ---- copy geometry: piece p of a tile = rows [RPP p, RPP (p + 1)); lane l
  // writes row RPP p + l / CPR at stored chunk l % CPR
  const int crow = lane / G::CPR;
  const uint16_t* a_src[G::A_PW];
  const uint16_t* w_src[G::W_PW];
#pragma unroll
  for (int i = 0; i < G::A_PW; ++i) {
    const int r = (wave * G::A_PW + i) * G::RPP + crow;
    const int c = G::swz(r, lane % G::CPR);  // the swizzle is an involution
    const int m = min(m0 + r, M - 1);        // rows past M read row M-1 (results discarded)
    a_src[i] = A + (int64_t)m * K + kbeg + c * 8;
  }
#pragma unroll
  for (int i = 0; i < G::W_PW; ++i) {
    const int r = (wave * G::W_PW + i) * G::RPP + crow;
    const int c = G::swz(r, lane % G::CPR);
    w_src[i] = W + (int64_t)(n0 + r) * K + kbeg + c * 8;
  }
  auto issue = [&](int st, uint8_t* base) {
    const int k0 = st * BK;
#pragma unroll
    for (int i = 0; i < G::A_PW; ++i)
      copy16_to_lds(a_src[i] + k0, base + (wave * G::A_PW + i) * 1024);
#pragma unroll
    for (int i = 0; i < G::W_PW; ++i)
      copy16_to_lds(w_src[i] + k0, base + G::A_BYTES + (wave * G::W_PW + i) * 1024);
  };

  // ---- operand reads: k-step ks of a stage, 32-row block: lane l reads
  // row l % 32 of the block, logical chunk 2 ks + l / 32 (block offsets are
  // multiples of 32 rows, which leave the swizzle unchanged)
  uint32_t ofs[G::KS];
#pragma unroll
  for (int ks = 0; ks < G::KS; ++ks) {
    const int r = lane & 31;
    ofs[ks] = (uint32_t)(r * ROW + G::swz(r, 2 * ks + (lane >> 5)) * 16);
  }

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int jn = 0; jn < TN; ++jn)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][jn][r] = 0.f;

  const int nk = kslice / BK;
  static_for<0, STAGES - 1>([&](auto s_c) {
    if (decltype(s_c)::value < nk) issue(decltype(s_c)::value, buf(s_c));
  });

  // stages in groups of GROUP (a multiple of STAGES), so that every buffer
  // index is a constant; the compiler drains the copies once per group (at
  // the loop head it no longer knows which buffer each pending copy fills)
  constexpr int GROUP = STAGES * (8 / STAGES);
  for (int kb0 = 0; kb0 < nk; kb0 += GROUP) {
    static_for<0, GROUP>([&](auto i_c) {
      constexpr int i = decltype(i_c)::value;
      const int kb = kb0 + i;
      if (kb >= nk) return;
      // stage kb has landed once at most the later stages' copies are pending
      wait_stages<G::LOADS, STAGES - 2>(min(STAGES - 2, nk - 1 - kb));
      barrier();  // every wave's copies of stage kb are in; stage kb-1's buffer is free
      if (kb + STAGES - 1 < nk)
        issue(kb + STAGES - 1, buf(std::integral_constant<int, i + STAGES - 1>()));
      const uint8_t* base = buf(i_c);
      const uint8_t* as = base + wm * G::WTM * ROW;
      const uint8_t* ws = base + G::A_BYTES + wn * G::WTN * ROW;
#pragma unroll
      for (int ks = 0; ks < G::KS; ++ks) {
        uint4 av[TM], wv[TN];
#pragma unroll
        for (int ii = 0; ii < TM; ++ii)
          av[ii] = *reinterpret_cast<const uint4*>(as + ii * 32 * ROW + ofs[ks]);
#pragma unroll
        for (int jn = 0; jn < TN; ++jn)
          wv[jn] = *reinterpret_cast<const uint4*>(ws + jn * 32 * ROW + ofs[ks]);
#pragma unroll
        for (int ii = 0; ii < TM; ++ii)
#pragma unroll
          for (int jn = 0; jn < TN; ++jn) acc[ii][jn] = mfma(wv[jn], av[ii], acc[ii][jn]);
      }
    });
  }

  // ---- epilogue: acc[i][jn] register 4q + e holds
  //   m = m0 + wm*WTM + 32i + lane%32,   n = n0 + wn*WTN + 32jn + 8q + 4(lane/32) + e
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = m0 + wm * G::WTM + 32 * i + (lane & 31);
    if (m >= M) continue;
#pragma unroll
    for (int jn = 0; jn < TN; ++jn)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = n0 + wn * G::WTN + 32 * jn + 8 * q + 4 * (lane >> 5);
        const int64_t off = (int64_t)m * N + n;
        float v0 = acc[i][jn][4 * q], v1 = acc[i][jn][4 * q + 1];
        float v2 = acc[i][jn][4 * q + 2], v3 = acc[i][jn][4 * q + 3];
        if (part) {  // fp32 partial of slice sl
          *reinterpret_cast<float4*>(part + (int64_t)sl * M * N + off) =
              make_float4(v0, v1, v2, v3);
          continue;
        }
        if (R) {
          const uint2 r = *reinterpret_cast<const uint2*>(R + off);
          v0 += lo(r.x), v1 += hi(r.x), v2 += lo(r.y), v3 += hi(r.y);
        }
        *reinterpret_cast<uint2*>(C + off) = make_uint2(pack(v0, v1), pack(v2, v3));
      }
  }
}

// C = sum over S slices of part (+ R), 4 elements per thread
__global__ __launch_bounds__(256) void split_sum_kernel(const float* __restrict__ part,
                                                        const uint16_t* R, uint16_t* C,
                                                        int64_t mn4, int S) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= mn4) return;
  float4 v = reinterpret_cast<const float4*>(part)[i];
  for (int s = 1; s < S; ++s) {
    const float4 p = reinterpret_cast<const float4*>(part + (int64_t)s * mn4 * 4)[i];
    v.x += p.x, v.y += p.y, v.z += p.z, v.w += p.w;
  }
  if (R) {
    const uint2 r = reinterpret_cast<const uint2*>(R)[i];
    v.x += lo(r.x), v.y += hi(r.x), v.z += lo(r.y), v.w += hi(r.y);
  }
  reinterpret_cast<uint2*>(C)[i] = make_uint2(pack(v.x, v.y), pack(v.z, v.w));
}

template <int BM, int BN, int BK, int STAGES, int WGM = 2, int WGN = 2>
hipError_t launch(const uint16_t* A, const uint16_t* W, const uint16_t* R, uint16_t* C,
                  float* part, int M, int N, int K, int S, hipStream_t s) {
  const int MB = (M + BM - 1) / BM, NB = N / BN;
  const int NBX = (NB + kXcds - 1) / kXcds * kXcds;  // column blocks rounded up to the XCDs
  hipLaunchKernelGGL((gemm_kernel<BM, BN, BK, STAGES, WGM, WGN>), dim3(MB * NBX * S),
                     dim3(64 * WGM * WGN), 0, s, A, W, R, C, part, M, N, K, S);
  return hipGetLastError();
}

// Tile configurations (M x N tile, k per stage; 4 waves in 2 x 2, or 8 in
// 2 x 4 for the 256 x 256 tiles).  The default choice is measured; the others
// stay selectable (CPL_GEMM_CFG) for comparison on other shapes.
struct Cfg {
  int bm, bn, bk;
};
constexpr int kNumCfgs = 8;
constexpr Cfg kCfgs[kNumCfgs] = {{64, 128, 32},  {128, 128, 32}, {128, 256, 32}, {256, 128, 32},
                                 {64, 128, 64},  {128, 128, 64}, {256, 256, 32}, {256, 256, 64}};

hipError_t launch_cfg(int cfg, const uint16_t* A, const uint16_t* W, const uint16_t* R,
                      uint16_t* C, float* part, int M, int N, int K, int S, hipStream_t s) {
  switch (cfg) {
    case 0: return launch<64, 128, 32, 4>(A, W, R, C, part, M, N, K, S, s);
    case 1: return launch<128, 128, 32, 4>(A, W, R, C, part, M, N, K, S, s);
    case 2: return launch<128, 256, 32, 3>(A, W, R, C, part, M, N, K, S, s);
    case 3: return launch<256, 128, 32, 3>(A, W, R, C, part, M, N, K, S, s);
    case 4: return launch<64, 128, 64, 3>(A, W, R, C, part, M, N, K, S, s);
    case 5: return launch<128, 128, 64, 2>(A, W, R, C, part, M, N, K, S, s);
    case 6: return launch<256, 256, 32, 3, 2, 4>(A, W, R, C, part, M, N, K, S, s);
    case 7: return launch<256, 256, 64, 2, 2, 4>(A, W, R, C, part, M, N, K, S, s);
  }
  return hipErrorInvalidValue;
}

// the configuration with the same tile and 32 k per stage
int with_bk32(int cfg) { return cfg == 4 ? 0 : cfg == 5 ? 1 : cfg == 7 ? 6 : cfg; }

int env_int(const char* name, int dflt) {
  const char* s = getenv(name);
  return s ? atoi(s) : dflt;
}

// Tile configuration and K split for a shape: the largest tile that still
// gives every CU work, then a split over K while the grid is below two
// workgroups per CU (each slice at least kMinSliceK long).
void choose(int M, int N, int K, size_t ws_floats, int* cfg, int* S) {
  const int forced = env_int("CPL_GEMM_CFG", -1);
  int c = forced;
  // measured on the layer's projections (N 4096-6144, K 4096): 64 x 128
  // tiles with 64 k per stage up to 64 rows, 128 x 128 with 64 k above
  if (c < 0 || c >= kNumCfgs) c = M <= 64 ? 4 : 5;
  if (kCfgs[c].bn > 128 && N % kCfgs[c].bn != 0) c = 1;
  const Cfg& f = kCfgs[c];
  const int64_t tiles = (int64_t)((M + f.bm - 1) / f.bm) * (N / f.bn);
  int s = 1;
  const int forced_s = env_int("CPL_GEMM_SPLIT", 0);
  if (forced_s > 0) {
    s = forced_s;
  } else {
    while (tiles * s * 2 <= 512 && K % (2 * s * f.bk) == 0 && K / (2 * s) >= kMinSliceK) s *= 2;
  }
  while (s > 1 && (K % (s * f.bk) != 0 || (size_t)s * M * N > ws_floats)) s /= 2;
  *cfg = c;
  *S = s;
}

}  // namespace

extern "C" {

size_t cpl_gemm_workspace_bytes(int32_t m, int32_t n, int32_t k) {
  if (m < 1 || n < 128 || n % 128 != 0 || k < 32 || k % 32 != 0) return 0;
  int cfg, s;
  choose(m, n, k, (size_t)-1 / 8, &cfg, &s);
  return s > 1 ? (size_t)s * m * n * sizeof(float) : 0;
}

int cpl_gemm(const void* a, const void* w, const void* r, void* c, int32_t m, int32_t n,
             int32_t k, void* ws, size_t ws_bytes, void* stream) {
  if (m < 1 || n < 128 || n % 128 != 0 || k < 32 || k % 32 != 0) return CP_ERR_INVALID_ARG;
  if (!a || !w || !c || a == c || w == c) return CP_ERR_INVALID_ARG;
  auto al16 = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  if (!al16(a) || !al16(w) || !al16(c) || (r && !al16(r)) || (ws && !al16(ws)))
    return CP_ERR_INVALID_ARG;
  if ((int64_t)m * k >= ((int64_t)1 << 40) || (int64_t)n * k >= ((int64_t)1 << 40) ||
      (int64_t)m * n >= ((int64_t)1 << 40))
    return CP_ERR_INVALID_ARG;
  int cfg, S;
  choose(m, n, k, ws ? ws_bytes / sizeof(float) : 0, &cfg, &S);
  if (k % kCfgs[cfg].bk != 0) cfg = with_bk32(cfg);  // k per stage must divide K
  (void)hipGetLastError();
  hipStream_t s = (hipStream_t)stream;
  const uint16_t* A = (const uint16_t*)a;
  const uint16_t* W = (const uint16_t*)w;
  const uint16_t* R = (const uint16_t*)r;
  uint16_t* C = (uint16_t*)c;
  float* part = S > 1 ? (float*)ws : nullptr;
  hipError_t e = launch_cfg(cfg, A, W, R, C, part, m, n, k, S, s);
  if (e == hipSuccess && S > 1) {
    const int64_t mn4 = (int64_t)m * n / 4;
    hipLaunchKernelGGL(split_sum_kernel, dim3((unsigned)((mn4 + 255) / 256)), dim3(256), 0, s,
                       part, R, C, mn4, S);
    e = hipGetLastError();
  }
  return e == hipSuccess ? CP_OK : CP_ERR_HIP;
}

}  // extern "C"
