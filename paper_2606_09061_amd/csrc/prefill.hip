// Prefill-chunk attention on bf16 MFMA (v_mfma_f32_32x32x16_bf16).
//
// Prefill is compute bound (Sec. 1 and 2.1 of the paper): a chunk of c
// queries over s prior keys costs ~c*s + c^2/2 query-key pairs per head (the
// prefill_interaction feature of Table 2 tracks exactly that product).
//
// Work item: a tile of up to 32*NW query rows of one chunk, where a row is a
// (token, q head) pair of the G q heads that share one kv head, so K and V
// are gathered once for all G heads (GQA sharing); plus a key range.  Each
// of the NW waves owns 32 rows.  Per 64-key step the workgroup gathers the K
// rows and the feature-major V blocks of the step through the block table
// into an LDS tile; each wave then computes
//     S^T (64 keys x 32 queries) = K . Q^T      MFMA, fp32 accumulators
//     online softmax down each query column     fp32, base 2
//     O^T (D x 32 queries)     += V^T . P^T     MFMA, P rounded to bf16
// Computing the transposed products keeps one query per lane column, so the
// softmax is lane-local except for one exchange between the two lane halves.
// The rows of the K operand are loaded in a permuted key order (sigma) that
// makes the score registers of a lane exactly the B operand of the P.V step,
// so probabilities never leave registers.  Only steps that cross the causal
// diagonal or the end of the range apply a mask.
//
// The query operand Q^T stays in registers for the whole item.  Pipeline:
// one register set stages the gather into one of two LDS tiles while the
// other is computed.
// Each load instruction reads 1 KiB of one block, so its block id is
// wave-uniform and the block base lives in scalar registers.
// LDS rows are XOR-swizzled in 16-byte units instead of padded so that the
// MFMA operand reads of 16 consecutive lanes hit distinct banks.
#include "device.hpp"
#include "kernels.hpp"
#include "prefill_common.hpp"

namespace cpattn {

template <int D, int B, int G, int NW>
__global__ __launch_bounds__(NW * 64, 8 / NW) void prefill_kernel(
    const PrefillItem* __restrict__ items, const int32_t* __restrict__ slots,
    const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ k_cache, const uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ bt, uint16_t* __restrict__ out, float* __restrict__ part_o,
    float* __restrict__ part_lse, int hq, int hkv, int mbr, float scale_log2) {
  using L = PrefillLayout<D, B>;
  constexpr int NKS = D / 16;                   // k-steps of S^T
  constexpr int NDT = D / 32;                   // 32-feature tiles of O^T
  constexpr int KCH = L::KCH;
  constexpr int VPB = D * B / 8;                // 16-byte chunks per V block (one kv head)
  constexpr int LOG2B = B == 16 ? 4 : 5;
  static_assert(B == 16 || B == 32, "block size");
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  const int slot = slots[blockIdx.x];
  if (slot < 0) return;  // idle slot of the XCD-interleaved order
  const int item = slot / hkv;
  const int kvh = slot - item * hkv;
  const PrefillItem it = items[item];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int col = lane & 31;
  const int g = lane >> 5;
  const int row = wave * 32 + col;  // query row of the tile
  const int tl = row / G;
  const int hh = row % G;
  const bool row_valid = tl < it.n_tok;
  const int qpos = it.pos0 + tl;
  const int32_t* bt_row = bt + (int64_t)it.req * mbr;
  const int64_t blk_elems = (int64_t)hkv * B * D;
  const uint16_t* kbase = k_cache + (int64_t)kvh * B * D;
  const uint16_t* vbase = v_cache + (int64_t)kvh * B * D;

  // Q^T operand: lane holds features [16 ks + 8 g, +8) of its query row
  uint4 qreg[NKS];
  {
    const uint16_t* qp =
        q + ((int64_t)(it.tok0 + (row_valid ? tl : 0)) * hq + kvh * G + hh) * D + g * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qreg[ks] = row_valid ? ld_global16(qp + ks * 16) : make_uint4(0, 0, 0, 0);
  }

  // ---- gather: a step is BN keys of K (token-major rows) and BN / B V
  // blocks (feature-major).  The first half of the waves load the K rows,
  // the second half the V blocks, each wave a contiguous run of 1 KiB pieces
  // (64 lanes x 16 bytes).  K and V address alike: chunk x of the step lies
  // in block x / VPB at element (x % VPB) * 8.  No piece straddles a block,
  // so every load instruction needs one wave-uniform block-table entry.
  // Every load is issued: a piece past the range re-reads the step's first
  // block (a valid entry, since k0 < kv_end).  Scores of keys past the range
  // are masked, so such K rows may hold anything; V past the range is zeroed.
  constexpr int HALF = NW / 2;                  // waves loading K
  constexpr int CPL = BN * KCH / (HALF * 64);   // 16-byte chunks per lane per step
  static_assert(CPL >= 1 && VPB % 64 == 0 && VPB == B * KCH, "gather geometry");
  struct Regs {
    uint4 c[CPL];
  };
  const bool vwave = wave >= HALF;
  const int wbase = (vwave ? wave - HALF : wave) * CPL * 64;  // first chunk of this wave
  const uint16_t* gbase = vwave ? vbase : kbase;
  auto gload = [&](Regs& r, int k0) {
    const int b0 = k0 >> LOG2B;
    const bool full = k0 + BN <= it.kv_end;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int p = wbase + i * 64;  // first chunk of the piece
      const int bi = p / VPB;
      const bool live = full || (k0 + (vwave ? bi * B : p / KCH) < it.kv_end);
      const uint16_t* bp = gbase + (int64_t)bt_row[b0 + (live ? bi : 0)] * blk_elems;
      uint4 val = ld_global16(bp + ((p + lane) % VPB) * 8);
      if (vwave && !full) {  // zero values of keys past the range
        const int vpos = k0 + bi * B + (((p + lane) % VPB) % L::VSLOTS) * 8;
        uint32_t* wv = reinterpret_cast<uint32_t*>(&val);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t lo = (vpos + 2 * e) < it.kv_end ? 0x0000ffffu : 0u;
          const uint32_t hi = (vpos + 2 * e + 1) < it.kv_end ? 0xffff0000u : 0u;
          wv[e] &= (lo | hi);
        }
      }
      r.c[i] = val;
    }
  };
  // LDS destination of chunk i of this lane (fixed for the whole item)
  auto soff = [&](int i) {
    const int x = wbase + i * 64 + lane;
    const int w = x % VPB;
    return vwave ? L::v_off(x / VPB, w / L::VSLOTS, w % L::VSLOTS) : L::k_off(x / KCH, x % KCH);
  };
  auto sstore = [&](const Regs& r, int buf) {
    uint8_t* base = smem + buf * L::BUF;
#pragma unroll
    for (int i = 0; i < CPL; ++i) *reinterpret_cast<uint4*>(base + soff(i)) = r.c[i];
  };

  f32x16_t oacc[NDT];
#pragma unroll
  for (int i = 0; i < NDT; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
  float m_run = -INFINITY;  // running max of the scaled (base-2) scores
  float l_run = 0.f;
  const int krow0 = sigma(col);

  // MFMA loops: operand reads run kRing MFMAs ahead through a register ring;
  // scheduling fences keep that order (left alone, the scheduler trades the
  // ring for registers and waits on every read).
  constexpr int kRing = 4;
  // ---- S^T = K . Q^T of the step in buffer `buf`: MFMA i uses k-step i / 2
  // and 32-key sub-tile i % 2
  auto qk = [&](int buf, f32x16_t* sacc) {
    const uint8_t* base = smem + buf * L::BUF;
    constexpr int NQK = 2 * NKS;
    auto kop = [&](int i) {
      return *reinterpret_cast<const uint4*>(base + L::k_off((i & 1) * 32 + krow0, 2 * (i >> 1) + g));
    };
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kt][r] = 0.f;
    uint4 ring[kRing];
#pragma unroll
    for (int i = 0; i < kRing; ++i) ring[i] = kop(i);
#pragma unroll
    for (int i = 0; i < NQK; ++i) {
      const uint4 a = ring[i % kRing];
      if (i + kRing < NQK) ring[i % kRing] = kop(i + kRing);
      sacc[i & 1] = mfma32x32x16(a, qreg[i >> 1], sacc[i & 1]);
      __builtin_amdgcn_sched_barrier(0);  // keep reads kRing MFMAs ahead
    }
  };
  // ---- online softmax on raw scores (the scale is folded into exp2); the
  // bf16 weights come out as the P^T operand of the next product
  auto softmax = [&](f32x16_t* sacc, int k0, uint4 (&pk)[2][2]) {
    const bool edge = (k0 + BN - 1 > it.pos0) || (k0 + BN > it.kv_end);
    if (edge) {
      // keys [k0, k0 + lim) are visible; register r of half g holds key
      // kt*32 + acc_key(r, 0) + 8*g, so compare against lim - 8*g
      const int limg = min(qpos + 1, it.kv_end) - k0 - 8 * g;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (kt * 32 + acc_key(r, 0) >= limg) sacc[kt][r] = -INFINITY;
    }
    float mt = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; r += 2) mt = fmaxf(fmaxf(mt, sacc[kt][r]), sacc[kt][r + 1]);
    mt = fmaxf(mt, shfl_xor_f(mt, 32)) * scale_log2;
    if (__builtin_amdgcn_ballot_w64(mt > m_run + kRescaleThreshold)) {
      const float mnew = fmaxf(m_run, mt);
      const float alpha = (m_run == -INFINITY) ? 0.f : exp2f(m_run - mnew);
      m_run = mnew;
      l_run *= alpha;
#pragma unroll
      for (int i = 0; i < NDT; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[i][r] *= alpha;
    }
    const float neg_m = m_run == -INFINITY ? 0.f : -m_run;
    const uint32_t ones = 0x3f803f80u;  // bf16 pair (1, 1)
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 =
              __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kt][8 * h2 + 2 * e], scale_log2, neg_m));
          const float p1 = __builtin_amdgcn_exp2f(
              __builtin_fmaf(sacc[kt][8 * h2 + 2 * e + 1], scale_log2, neg_m));
          w[e] = pack_bf16x2(p0, p1);
          l_run = dot2_bf16(w[e], ones, l_run);  // sum of the rounded weights
        }
        pk[kt][h2] = make_uint4(w[0], w[1], w[2], w[3]);
      }
  };
  // ---- O^T += V^T . P^T with the step in buffer `buf` (values of keys past
  // the range were zeroed by the gather): MFMA i uses key step i / NDT and
  // feature tile i % NDT
  auto pv = [&](int buf, const uint4 (&pk)[2][2]) {
    const uint8_t* base = smem + buf * L::BUF;
    constexpr int NPV = 4 * NDT;
    auto vop = [&](int i) {
      const int ks2 = i / NDT, dt = i % NDT;
      return *reinterpret_cast<const uint4*>(
          base + L::v_off((ks2 * 16) / B, dt * 32 + col, ((ks2 * 16) % B) / 8 + g));
    };
    uint4 ring[kRing];
#pragma unroll
    for (int i = 0; i < kRing; ++i) ring[i] = vop(i);
#pragma unroll
    for (int i = 0; i < NPV; ++i) {
      const uint4 a = ring[i % kRing];
      if (i + kRing < NPV) ring[i % kRing] = vop(i + kRing);
      const int ks2 = i / NDT;
      oacc[i % NDT] = mfma32x32x16(a, pk[ks2 >> 1][ks2 & 1], oacc[i % NDT]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  const int n_step = (it.kv_end - it.kv_begin + BN - 1) / BN;
  auto step = [&](int buf, int k0) {
    f32x16_t sacc[2];
    uint4 pk[2][2];
    qk(buf, sacc);
    softmax(sacc, k0, pk);
    pv(buf, pk);
  };
  // Two LDS buffers, step s in buffer s % 2: the loads of step s+1 are
  // issued before step s is computed and written to the other buffer after
  // it, so every gather has one step of MFMA work to arrive.
  Regs ra;
  gload(ra, it.kv_begin);
  sstore(ra, 0);
  __syncthreads();
  for (int st = 0; st < n_step; ++st) {
    const int k0 = it.kv_begin + st * BN;
    const bool has_next = st + 1 < n_step;
    if (has_next) gload(ra, k0 + BN);
    step(st & 1, k0);
    if (has_next) sstore(ra, (st & 1) ^ 1);
    __syncthreads();
  }

  // ---- finish: the two lane halves hold disjoint keys of the same query
  const float l_tot = l_run + shfl_xor_f(l_run, 32);
  if (!row_valid) return;
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (it.part < 0) {
    uint16_t* op = out + ((int64_t)(it.tok0 + tl) * hq + kvh * G + hh) * D + 4 * g;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d0 = dt * 32 + 8 * i;
        uint2 w;
        w.x = pack_bf16x2(oacc[dt][4 * i + 0] * inv, oacc[dt][4 * i + 1] * inv);
        w.y = pack_bf16x2(oacc[dt][4 * i + 2] * inv, oacc[dt][4 * i + 3] * inv);
        *reinterpret_cast<uint2*>(op + d0) = w;
      }
  } else {
    const int prow = it.part + kvh * it.part_kvh_stride + row;
    float* pp = part_o + (int64_t)prow * D + 4 * g;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d0 = dt * 32 + 8 * i;
        *reinterpret_cast<float4*>(pp + d0) =
            make_float4(oacc[dt][4 * i + 0] * inv, oacc[dt][4 * i + 1] * inv,
                        oacc[dt][4 * i + 2] * inv, oacc[dt][4 * i + 3] * inv);
      }
    if (g == 0) part_lse[prow] = l_tot > 0.f ? m_run + __log2f(l_tot) : -INFINITY;
  }
}

template <int D, int B, int G, int NW>
static hipError_t launch_prefill_t(const PrefillItem* items, const int32_t* slots, int n,
                                   const AttnArgs& a, hipStream_t s) {
  constexpr int smem = 2 * PrefillLayout<D, B>::BUF;
  static const hipError_t attr =
      hipFuncSetAttribute(reinterpret_cast<const void*>(&prefill_kernel<D, B, G, NW>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, smem);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((prefill_kernel<D, B, G, NW>), dim3(n), dim3(NW * 64), smem, s, items, slots,
                     a.q,
                     a.k_cache, a.v_cache, a.bt, a.out, a.part_o, a.part_lse, a.hq, a.hkv, a.mbr,
                     a.scale_log2);
  return hipGetLastError();
}

template <int D, int B, int NW>
static hipError_t launch_prefill_g(int G, const PrefillItem* items, const int32_t* slots, int n,
                                   const AttnArgs& a, hipStream_t s) {
  switch (G) {
    case 1: return launch_prefill_t<D, B, 1, NW>(items, slots, n, a, s);
    case 2: return launch_prefill_t<D, B, 2, NW>(items, slots, n, a, s);
    case 4: return launch_prefill_t<D, B, 4, NW>(items, slots, n, a, s);
    case 8: return launch_prefill_t<D, B, 8, NW>(items, slots, n, a, s);
  }
  return hipErrorInvalidValue;
}

template <int NW>
static hipError_t launch_prefill_w(int D, int G, const PrefillItem* items, const int32_t* slots,
                                   int n, const AttnArgs& a, hipStream_t s) {
  if (D == 128 && a.block_size == 16) return launch_prefill_g<128, 16, NW>(G, items, slots, n, a, s);
  if (D == 128 && a.block_size == 32) return launch_prefill_g<128, 32, NW>(G, items, slots, n, a, s);
  if (D == 64 && a.block_size == 16) return launch_prefill_g<64, 16, NW>(G, items, slots, n, a, s);
  if (D == 64 && a.block_size == 32) return launch_prefill_g<64, 32, NW>(G, items, slots, n, a, s);
  return hipErrorInvalidValue;
}

hipError_t launch_prefill(int D, int G, const AttnArgs& a, hipStream_t s) {
  hipError_t e = hipSuccess;
  if (a.n_prefill_wide_slots > 0)
    e = launch_prefill_w<8>(D, G, a.prefill_wide, a.prefill_wide_slots, a.n_prefill_wide_slots, a,
                            s);
  if (e == hipSuccess && a.n_prefill_slots > 0)
    e = launch_prefill_w<4>(D, G, a.prefill, a.prefill_slots, a.n_prefill_slots, a, s);
  return e;
}

}  // namespace cpattn
