// Prefill-chunk attention on bf16 MFMA (v_mfma_f32_32x32x16_bf16).
//
// Prefill is compute bound (Sec. 1 and 2.1 of the paper): a chunk of c
// queries over s prior keys costs ~c*s + c^2/2 query-key pairs per head (the
// prefill_interaction feature of Table 2 tracks exactly that product).
//
// Work item: a tile of up to 128 query rows of one chunk, where a row is a
// (token, q head) pair of the G q heads that share one kv head, so K and V
// are loaded once for all G heads (GQA sharing); plus a key range.  Four
// waves own 32 rows each.  Per 64-key step the workgroup gathers the K rows
// and the feature-major V blocks of the step through the block table into
// a double-buffered LDS tile (the next step's global loads are in flight
// while the current one is multiplied), then each wave computes
//     S^T (64 keys x 32 queries) = K . Q^T      MFMA, fp32 accumulators
//     online softmax down each query column     fp32, base 2
//     O^T (D x 32 queries)     += V^T . P^T     MFMA, P rounded to bf16
// Computing the transposed products keeps one query per lane column, so the
// softmax is lane-local except for one exchange between the two lane halves.
// The rows of the K operand are loaded in a permuted key order (sigma) that
// makes the score registers of a lane exactly the B operand of the P.V step,
// so probabilities never leave registers.  Only steps that cross the causal
// diagonal or the end of the range apply a mask.
#include "device.hpp"
#include "kernels.hpp"

namespace cpattn {

namespace {

constexpr int BN = kPrefillKeys;  // keys per step

// key row loaded into MFMA row c of a 32-key sub-tile: swaps bits 2 and 3
__device__ __forceinline__ int sigma(int c) {
  return (c & ~12) | ((c & 4) << 1) | ((c & 8) >> 1);
}

// key (within a 32-key sub-tile) of accumulator register r of lane half g:
// sigma of the accumulator row 8*(r/4) + 4*g + r%4
__device__ __forceinline__ int acc_key(int r, int g) {
  return 16 * ((r >> 3) & 1) + 8 * g + 4 * ((r >> 2) & 1) + (r & 3);
}

}  // namespace

template <int D>
struct PrefillSmem {
  static constexpr int KS = D * 2 + 16;   // bytes per K row (padded)
  static constexpr int VS = BN * 2 + 16;  // bytes per V^T feature row (padded)
  static constexpr int K_BYTES = BN * KS;
  static constexpr int V_BYTES = D * VS;
  static constexpr int BUF = K_BYTES + V_BYTES;
  static constexpr int TOTAL = 2 * BUF;
};

template <int D, int B, int G>
__global__ __launch_bounds__(256, 2) void prefill_kernel(
    const PrefillItem* __restrict__ items, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ k_cache, const uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ bt, uint16_t* __restrict__ out, float* __restrict__ part_o,
    float* __restrict__ part_lse, int hq, int hkv, int mbr, float scale_log2) {
  using SM = PrefillSmem<D>;
  constexpr int NKS = D / 16;                   // k-steps of S^T
  constexpr int NDT = D / 32;                   // 32-feature tiles of O^T
  constexpr int CH = BN * D * 2 / (256 * 16);   // 16-byte chunks per thread per K (and V) step
  constexpr int KCH = D / 8;                    // 16-byte chunks per K row
  constexpr int VPB = D * B / 8;                // 16-byte chunks per V block (one kv head)
  constexpr int LOG2B = B == 16 ? 4 : 5;
  static_assert(B == 16 || B == 32, "block size");
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  const PrefillItem it = items[blockIdx.x];
  if (it.n_tok == 0) return;  // padding slot of the XCD-interleaved order
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
  const uint16_t* kbase = k_cache + (int64_t)it.kvh * B * D;
  const uint16_t* vbase = v_cache + (int64_t)it.kvh * B * D;

  // Q^T operand: lane holds features [16 ks + 8 g, +8) of its query row
  uint4 qreg[NKS];
  {
    const uint16_t* qp =
        q + ((int64_t)(it.tok0 + (row_valid ? tl : 0)) * hq + it.kvh * G + hh) * D + g * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qreg[ks] = row_valid ? ld_global16(qp + ks * 16) : make_uint4(0, 0, 0, 0);
  }

  // ---- gather geometry of 16-byte chunk c of this thread (shifts and masks
  // only: every divisor below is a compile-time power of two)
  //   K chunk: key kkey(c) of the step, feature chunk x % KCH
  //   V chunk: block x / VPB of the step, feature row d, 8 keys from slot s0
  auto kkey = [&](int c) { return (c * 256 + tid) / KCH; };
  auto kgoff = [&](int c) { return (kkey(c) & (B - 1)) * D + ((c * 256 + tid) % KCH) * 8; };
  auto klds = [&](int c) { return kkey(c) * SM::KS + ((c * 256 + tid) % KCH) * 16; };
  auto vblk = [&](int c) { return (c * 256 + tid) / VPB; };
  auto vd = [&](int c) { return ((c * 256 + tid) % VPB) / (B / 8); };
  auto vs0 = [&](int c) { return (((c * 256 + tid) % VPB) % (B / 8)) * 8; };
  auto vkey = [&](int c) { return vblk(c) * B + vs0(c); };
  auto vgoff = [&](int c) { return vd(c) * B + vs0(c); };
  auto vlds = [&](int c) { return vd(c) * SM::VS + vkey(c) * 2; };

  uint4 kreg[CH], vreg[CH];
  auto gload = [&](int k0) {
    const int b0 = k0 >> LOG2B;
    if (k0 + BN <= it.kv_end) {
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        const int64_t kb = bt_row[b0 + (kkey(c) >> LOG2B)];
        kreg[c] = ld_global16(kbase + kb * blk_elems + kgoff(c));
        const int64_t vb = bt_row[b0 + vblk(c)];
        vreg[c] = ld_global16(vbase + vb * blk_elems + vgoff(c));
      }
    } else {  // last step of the range: keys at or past kv_end are zero
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        uint4 kv = make_uint4(0, 0, 0, 0);
        if (k0 + kkey(c) < it.kv_end) {
          const int64_t kb = bt_row[b0 + (kkey(c) >> LOG2B)];
          kv = ld_global16(kbase + kb * blk_elems + kgoff(c));
        }
        kreg[c] = kv;
        uint4 vv = make_uint4(0, 0, 0, 0);
        const int vpos = k0 + vkey(c);
        if (vpos < it.kv_end) {
          const int64_t vb = bt_row[b0 + vblk(c)];
          vv = ld_global16(vbase + vb * blk_elems + vgoff(c));
          if (vpos + 8 > it.kv_end) {
            uint32_t* w = reinterpret_cast<uint32_t*>(&vv);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const uint32_t lo = (vpos + 2 * e) < it.kv_end ? 0x0000ffffu : 0u;
              const uint32_t hi = (vpos + 2 * e + 1) < it.kv_end ? 0xffff0000u : 0u;
              w[e] &= (lo | hi);
            }
          }
        }
        vreg[c] = vv;
      }
    }
  };
  auto sstore = [&](int buf) {
    uint8_t* kb = smem + buf * SM::BUF;
    uint8_t* vb = kb + SM::K_BYTES;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      *reinterpret_cast<uint4*>(kb + klds(c)) = kreg[c];
      *reinterpret_cast<uint4*>(vb + vlds(c)) = vreg[c];
    }
  };

  f32x16_t oacc[NDT];
#pragma unroll
  for (int i = 0; i < NDT; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
  float m_run = -INFINITY;  // running max of the scaled (base-2) scores
  float l_run = 0.f;

  const int n_step = (it.kv_end - it.kv_begin + BN - 1) / BN;
  gload(it.kv_begin);
  sstore(0);
  __syncthreads();

  const int krow0 = sigma(col);
  for (int st = 0; st < n_step; ++st) {
    const int cur = st & 1;
    const int k0 = it.kv_begin + st * BN;
    const bool has_next = st + 1 < n_step;
    if (has_next) gload(k0 + BN);

    const uint8_t* kb = smem + cur * SM::BUF;
    const uint8_t* vb = kb + SM::K_BYTES;

    // ---- S^T = K . Q^T for two 32-key sub-tiles
    f32x16_t sacc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kt][r] = 0.f;
      const uint8_t* ka = kb + (kt * 32 + krow0) * SM::KS + g * 16;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const uint4 a = *reinterpret_cast<const uint4*>(ka + ks * 32);
        sacc[kt] = mfma32x32x16(a, qreg[ks], sacc[kt]);
      }
    }

    // ---- online softmax down this lane's query column (raw scores; the
    // scale is folded into the exponent)
    if ((k0 + BN - 1 > it.pos0) || (k0 + BN > it.kv_end)) {
      const int lim = min(qpos + 1, it.kv_end) - k0;  // keys [k0, k0 + lim) are visible
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (kt * 32 + acc_key(r, g) >= lim) sacc[kt][r] = -INFINITY;
    }
    float mt = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mt = fmaxf(mt, sacc[kt][r]);
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
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        float p[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          p[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kt][8 * h2 + e], scale_log2, neg_m));
          l_run += p[e];
        }
        pk[kt][h2] = make_uint4(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                                pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7]));
      }

    // ---- O^T += V^T . P^T
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const uint8_t* va = vb + (dt * 32 + col) * SM::VS + g * 16;
#pragma unroll
      for (int ks2 = 0; ks2 < 4; ++ks2) {
        const uint4 a = *reinterpret_cast<const uint4*>(va + ks2 * 32);
        oacc[dt] = mfma32x32x16(a, pk[ks2 >> 1][ks2 & 1], oacc[dt]);
      }
    }

    if (has_next) sstore(cur ^ 1);
    __syncthreads();
  }

  // ---- finish: the two lane halves hold disjoint keys of the same query
  const float l_tot = l_run + shfl_xor_f(l_run, 32);
  if (!row_valid) return;
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (it.part < 0) {
    uint16_t* op = out + ((int64_t)(it.tok0 + tl) * hq + it.kvh * G + hh) * D + 4 * g;
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
    const int prow = it.part + row;
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

template <int D, int B, int G>
static hipError_t launch_prefill_t(const AttnArgs& a, hipStream_t s) {
  constexpr int smem = PrefillSmem<D>::TOTAL;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&prefill_kernel<D, B, G>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, smem);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((prefill_kernel<D, B, G>), dim3(a.n_prefill), dim3(256), smem, s, a.prefill,
                     a.q, a.k_cache, a.v_cache, a.bt, a.out, a.part_o, a.part_lse, a.hq, a.hkv,
                     a.mbr, a.scale_log2);
  return hipGetLastError();
}

template <int D, int B>
static hipError_t launch_prefill_g(int G, const AttnArgs& a, hipStream_t s) {
  switch (G) {
    case 1: return launch_prefill_t<D, B, 1>(a, s);
    case 2: return launch_prefill_t<D, B, 2>(a, s);
    case 4: return launch_prefill_t<D, B, 4>(a, s);
    case 8: return launch_prefill_t<D, B, 8>(a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_prefill(int D, int G, const AttnArgs& a, hipStream_t s) {
  if (D == 128 && a.block_size == 16) return launch_prefill_g<128, 16>(G, a, s);
  if (D == 128 && a.block_size == 32) return launch_prefill_g<128, 32>(G, a, s);
  if (D == 64 && a.block_size == 16) return launch_prefill_g<64, 16>(G, a, s);
  if (D == 64 && a.block_size == 32) return launch_prefill_g<64, 32>(G, a, s);
  return hipErrorInvalidValue;
}

}  // namespace cpattn
