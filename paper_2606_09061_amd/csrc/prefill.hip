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
// Pipeline: two LDS tiles and two register sets.  The global loads of step
// s+2 are issued at the start of step s and written to LDS at the end of
// step s+1, so every gather has two steps of MFMA work to arrive.  Block ids
// are wave-uniform for every load instruction (a wave's 64 lanes read one
// block), so the block base is computed once per wave in scalar registers.
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
  // Wide (8-wave) tiles keep the query operand in LDS and double the
  // register staging of the gather (two steps in flight); 4-wave tiles keep
  // the query operand in registers with one step in flight.
  constexpr bool kWide = NW == 8;
  constexpr int NT = NW * 64;                   // threads
  constexpr int NKS = D / 16;                   // k-steps of S^T
  constexpr int NDT = D / 32;                   // 32-feature tiles of O^T
  constexpr int KCH = L::KCH;
  constexpr int CK = BN * KCH / NT;             // K chunks per thread per step
  constexpr int VPB = D * B / 8;                // 16-byte chunks per V block (one kv head)
  constexpr int CV = BN * D / 8 / NT;           // V chunks per thread per step
  constexpr int LOG2B = B == 16 ? 4 : 5;
  static_assert(B == 16 || B == 32, "block size");
  static_assert(CK >= 1 && CV >= 1, "tile geometry");
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  const int slot = slots[blockIdx.x];
  if (slot < 0) return;  // idle slot of the XCD-interleaved order
  const int item = slot / hkv;
  const int kvh = slot - item * hkv;
  const PrefillItem it = items[item];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
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
  uint4 qreg[kWide ? 1 : NKS];
  if constexpr (kWide) {
    // stage the tile's query rows in LDS: chunk x -> row x / KCH, chunk x % KCH
#pragma unroll
    for (int i = 0; i < NW * 32 * KCH / NT; ++i) {
      const int x = i * NT + tid;
      const int r = x / KCH;
      const int t = r / G;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (t < it.n_tok)
        v = ld_global16(q + ((int64_t)(it.tok0 + t) * hq + kvh * G + r % G) * D + (x % KCH) * 8);
      *reinterpret_cast<uint4*>(smem + L::q_off(r, x % KCH)) = v;
    }
  } else {
    const uint16_t* qp =
        q + ((int64_t)(it.tok0 + (row_valid ? tl : 0)) * hq + kvh * G + hh) * D + g * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qreg[ks] = row_valid ? ld_global16(qp + ks * 16) : make_uint4(0, 0, 0, 0);
  }
  auto qop = [&](int ks) -> uint4 {
    if constexpr (kWide)
      return *reinterpret_cast<const uint4*>(smem + L::q_off(row, 2 * ks + g));
    else
      return qreg[ks];
  };

  // ---- gather geometry: K chunk i of this thread is x = i*NT + tid
  // (key x / KCH, chunk x % KCH); V chunk i is x = i*NT + tid (step-block
  // x / VPB, feature row, 8-key slot).  All of a wave's lanes read one block.
  struct Regs {
    uint4 k[CK], v[CV];
  };
  auto gload = [&](Regs& r, int k0) {
    const int b0 = k0 >> LOG2B;
    const bool full = k0 + BN <= it.kv_end;
#pragma unroll
    for (int i = 0; i < CK; ++i) {
      const int x = i * NT + tid;
      const int key = x / KCH;
      const int kb = uniform(key) >> LOG2B;       // block of this wave's keys
      const bool live = full || (k0 + uniform(key) < it.kv_end);
      uint4 val = make_uint4(0, 0, 0, 0);
      if (live) {
        const int64_t blk = bt_row[b0 + kb];
        val = ld_global16(kbase + blk * blk_elems + (key & (B - 1)) * D + (x % KCH) * 8);
      }
      r.k[i] = val;
    }
#pragma unroll
    for (int i = 0; i < CV; ++i) {
      const int x = i * NT + tid;
      const int bi = uniform(x / VPB);
      const int w = x % VPB;
      const int d = w / L::VSLOTS;
      const int s = w % L::VSLOTS;
      const int vpos = k0 + bi * B + s * 8;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (full || k0 + bi * B < it.kv_end) {
        const int64_t blk = bt_row[b0 + bi];
        val = ld_global16(vbase + blk * blk_elems + d * B + s * 8);
        if (!full && vpos + 8 > it.kv_end) {  // zero values of keys past the range
          uint32_t* wv = reinterpret_cast<uint32_t*>(&val);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t lo = (vpos + 2 * e) < it.kv_end ? 0x0000ffffu : 0u;
            const uint32_t hi = (vpos + 2 * e + 1) < it.kv_end ? 0xffff0000u : 0u;
            wv[e] &= (lo | hi);
          }
        }
      }
      r.v[i] = val;
    }
  };
  auto sstore = [&](const Regs& r, int buf) {
    uint8_t* base = smem + buf * L::BUF;
#pragma unroll
    for (int i = 0; i < CK; ++i) {
      const int x = i * NT + tid;
      *reinterpret_cast<uint4*>(base + L::k_off(x / KCH, x % KCH)) = r.k[i];
    }
#pragma unroll
    for (int i = 0; i < CV; ++i) {
      const int x = i * NT + tid;
      const int w = x % VPB;
      *reinterpret_cast<uint4*>(base + L::v_off(x / VPB, w / L::VSLOTS, w % L::VSLOTS)) = r.v[i];
    }
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
  auto compute = [&](int buf, int k0) {
    const uint8_t* base = smem + buf * L::BUF;
    // ---- S^T = K . Q^T: MFMA i uses k-step i / 2 and 32-key sub-tile i % 2
    constexpr int NQK = 2 * NKS;
    auto kop = [&](int i) {
      return *reinterpret_cast<const uint4*>(base + L::k_off((i & 1) * 32 + krow0, 2 * (i >> 1) + g));
    };
    f32x16_t sacc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kt][r] = 0.f;
    {
      uint4 ring[kRing];
#pragma unroll
      for (int i = 0; i < kRing; ++i) ring[i] = kop(i);
#pragma unroll
      for (int i = 0; i < NQK; ++i) {
        const uint4 a = ring[i % kRing];
        if (i + kRing < NQK) ring[i % kRing] = kop(i + kRing);
        sacc[i & 1] = mfma32x32x16(a, qop(i >> 1), sacc[i & 1]);
        __builtin_amdgcn_sched_barrier(0);  // keep reads kRing MFMAs ahead
      }
    }
    // ---- online softmax on raw scores (the scale is folded into exp2)
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
    uint4 pk[2][2];
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
    // values of keys past the range were zeroed by the gather
    // ---- O^T += V^T . P^T: MFMA i uses key step i / NDT and feature tile i % NDT
    constexpr int NPV = 4 * NDT;
    auto vop = [&](int i) {
      const int ks2 = i / NDT, dt = i % NDT;
      return *reinterpret_cast<const uint4*>(
          base + L::v_off((ks2 * 16) / B, dt * 32 + col, ((ks2 * 16) % B) / 8 + g));
    };
    {
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
    }
  };

  const int n_step = (it.kv_end - it.kv_begin + BN - 1) / BN;
  if constexpr (kWide) {
    Regs ra, rb;
    gload(ra, it.kv_begin);
    sstore(ra, 0);
    if (n_step > 1) gload(rb, it.kv_begin + BN);
    __syncthreads();
    for (int st = 0; st < n_step; st += 2) {
      const int k0 = it.kv_begin + st * BN;
      // even step: LDS 0 holds step st, rb carries step st+1
      if (st + 2 < n_step) gload(ra, k0 + 2 * BN);
      compute(0, k0);
      if (st + 1 < n_step) sstore(rb, 1);
      __syncthreads();
      if (st + 1 >= n_step) break;
      // odd step: LDS 1 holds step st+1, ra carries step st+2
      if (st + 3 < n_step) gload(rb, k0 + 3 * BN);
      compute(1, k0 + BN);
      if (st + 2 < n_step) sstore(ra, 0);
      __syncthreads();
    }
  } else {
    Regs ra;
    gload(ra, it.kv_begin);
    sstore(ra, 0);
    __syncthreads();
    for (int st = 0; st < n_step; ++st) {
      const int k0 = it.kv_begin + st * BN;
      const bool has_next = st + 1 < n_step;
      if (has_next) gload(ra, k0 + BN);
      compute(st & 1, k0);
      if (has_next) sstore(ra, (st & 1) ^ 1);
      __syncthreads();
    }
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
  constexpr int smem = PrefillLayout<D, B>::KV_TOTAL + (NW == 8 ? NW * 32 * D * 2 : 0);
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
