// Prefill-chunk attention on bf16 MFMA (v_mfma_f32_32x32x16_bf16).
//
// Prefill is compute bound (Sec. 1 and 2.1 of the paper): a chunk of c
// queries over s prior keys costs ~c*s + c^2/2 query-key pairs per head (the
// prefill_interaction feature of Table 2 tracks exactly that product).
//
// Work item: a tile of up to 32*RG*NW query rows of one chunk, where a row is
// a (token, q head) pair of the G q heads that share one kv head, so K and V
// are gathered once for all G heads (GQA sharing); plus a key range.  Each
// wave owns RG groups of 32 rows that share every K and V operand read.  The
// build uses RG = 1 (RG = 2 needs more registers than a wave can hold without
// spilling the scores), NW = 4 or 8, and two workgroups per CU, so two waves
// share each SIMD.  Per 64-key step and row group a wave computes
//     S^T (64 keys x 32 queries) = K . Q^T      MFMA, fp32 accumulators
//     online softmax down each query column     fp32, base 2
//     O^T (D x 32 queries)     += V^T . P^T     MFMA, P rounded to bf16
// Computing the transposed products keeps one query per lane column, so the
// softmax is lane-local except for one exchange between the two lane halves.
// The rows of the K operand are loaded in a permuted key order (sigma) that
// makes the score registers of a lane exactly the B operand of the P.V step,
// so probabilities never leave registers.  Q^T stays in registers.
//
// Software pipeline inside each wave.  Iteration j has two phases:
//   phase K: S_{j+1} = K_{j+1} . Q^T   interleaved with   P_j = exp2(T_j)
//   phase V: O += V_j . P_j^T          interleaved with   the row sums of P_j,
//            the running max of S_{j+1} and T_{j+1} = S_{j+1} * scale - max
// so the MFMA pipe always has independent VALU work beside it.  The running
// max moves lazily (only when a score exceeds it by 2^8), and the rescale of
// O it then needs is a uniform branch after phase V.
//
// Gather.  K and V tiles are copied from the paged pools straight into LDS
// with global_load_lds_dwordx4 (16 bytes per lane, no VGPR staging), each
// wave a few 1 KiB pieces of one or two blocks per step, with wave-uniform
// block-table entries.  Per-lane source addresses are permuted so the LDS
// tiles land XOR-swizzled (conflict-free MFMA operand reads).  K and V each
// have two LDS buffers, separate arrays so that every access names its buffer
// at compile time.  The copy of a tile is issued 1.5 iterations before it is
// read; every phase starts with a wait on the copies it needs (the only
// waits on them: see copy16_to_lds) and one barrier.
//
// Output.  A lane's accumulators hold half the features of one row, in runs of four;
// stored directly, every store instruction would touch 32 rows.  Instead each
// wave writes its normalised rows into a private slice of the (then idle) K/V
// buffers and stores them back as whole rows, consecutive lanes taking
// consecutive 16-byte pieces of a row.
#include "decode_body.hpp"
#include "device.hpp"
#include "kernels.hpp"
#include "prefill_common.hpp"

#include <type_traits>

namespace cpattn {

namespace prefill_impl {

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Compile-time loop: f(std::integral_constant<int, I>) for I in [I0, N).  Every
// index into a register array stays a constant, so the arrays never spill to
// scratch however large the unrolled body gets.
template <int I0, int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I0 < N) {
    f(std::integral_constant<int, I0>());
    static_for<I0 + 1, N>(f);
  }
}

// Marks x as used here (no instruction), so the optimiser cannot sink its
// computation past this point into a later phase.
// (The "v" register constraint exists only for the device pass.)
__device__ __forceinline__ void keep(uint32_t x) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("" ::"v"(x));
#endif
}
__device__ __forceinline__ void keep(float x) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("" ::"v"(x));
#endif
}

// hides the known bits of x from the optimiser (no instruction)
__device__ __forceinline__ uint32_t opaque(uint32_t x) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("" : "+v"(x));
#endif
  return x;
}

__device__ __forceinline__ void set_word(uint4& v, int e, uint32_t w) {
  if (e == 0) v.x = w;
  else if (e == 1) v.y = w;
  else if (e == 2) v.z = w;
  else v.w = w;
}
__device__ __forceinline__ uint32_t get_word(const uint4& v, int e) {
  return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w;
}

// 16 bytes per lane from global memory (uniform base + this lane's byte
// offset) straight into LDS at lds + 16 * lane (`lds` wave-uniform, in M0),
// written as the instruction itself.  Built from the compiler's intrinsic,
// the copies were tracked by its wait insertion, which cannot tell which of
// the four LDS tiles a copy in flight fills: it waited for every copy,
// including the K tile issued 1.5 iterations ahead, before the V operand
// reads of every other iteration.  Untracked, the copies are awaited only by
// the explicit vmcnt waits below (no other vector-memory loads run in the
// loop, so the counts are exact; the compiler's own waits for the Q loads
// issued before them only ever wait longer).  The s_nop is the wait state a
// copy needs after M0 is written, which the compiler inserts only for its own.
__device__ __forceinline__ void copy16_to_lds(const uint16_t* base, uint32_t byte_off,
                                              uint8_t* lds) {
#if defined(__HIP_DEVICE_COMPILE__)
  const uint32_t dst = (uint32_t)(uintptr_t)(lds_ptr_t)lds;
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(byte_off), "s"(base),
               "{m0}"(dst)
               : "memory");
#endif
}

// s_waitcnt with vmcnt <= N, the other counters unconstrained (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ void barrier() { asm volatile("s_barrier" ::: "memory"); }

// max and sum of a value over the two 32-lane halves (v_permlane32_swap)
__device__ __forceinline__ float halves_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __builtin_fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int D, int B, int NW>
struct PrefillGeom {
  static constexpr int NKS = D / 16;               // k-steps of S^T (MFMAs per 32-key half)
  static constexpr int NDT = D / 32;               // 32-feature tiles of O^T
  static constexpr int NQK = 2 * NKS;              // K operand reads per step
  static constexpr int NPV = 4 * NDT;              // V operand reads per step
  static constexpr int KCH = D / 8;                // 16-byte chunks per K row
  static constexpr int TILE_BYTES = BN * D * 2;    // one step of K (or of V)
  static constexpr int PIECES = TILE_BYTES / 1024; // 1 KiB copies per step and tensor
  static constexpr int PW = PIECES / NW;           // ... per wave
  static constexpr int KPP = 1024 / (2 * D);       // keys per K piece
  static constexpr int PPB = D * B * 2 / 1024;     // pieces per block (K or V)
  static constexpr int NBW = PW > PPB ? PW / PPB : 1;  // blocks a wave copies per step
  static constexpr int V_ROWS = 1024 / (B * 2);    // V feature rows per piece
  static constexpr int V_LPR = B / 8;              // lanes per V feature row
  static constexpr int LOG2B = B == 16 ? 4 : 5;
  static constexpr int kRing = 3;                  // operand reads ahead of their MFMAs
  static_assert(PW >= 1 && PIECES % NW == 0, "gather geometry");
  static_assert(PW % NBW == 0 && (PW <= PPB ? PPB % PW == 0 : PW % PPB == 0), "piece split");
};

// row groups (32 query rows each) per wave
#ifndef CP_PREFILL_RG
#define CP_PREFILL_RG 1
#endif
constexpr int kPrefillRG = CP_PREFILL_RG;

}  // namespace prefill_impl

using namespace prefill_impl;

template <int D, int B, int G, int NW, int RG>
__global__ __launch_bounds__(NW * 64, RG == 1 ? 2 : 1) void prefill_kernel(
    const PrefillRec* __restrict__ recs, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ k_cache, const uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ bt, uint16_t* __restrict__ out, float* __restrict__ part_o,
    float* __restrict__ part_lse, int hq, int hkv, int mbr, float scale_log2,
    const DecodeItem* __restrict__ dec, int n_units) {
  using C = PrefillGeom<D, B, NW>;
  using L = PrefillLayout<D, B>;
  constexpr int NKS = C::NKS, NDT = C::NDT, NQK = C::NQK, NPV = C::NPV, PW = C::PW;
  constexpr int KCH = C::KCH, NBW = C::NBW, kRing = C::kRing;
  constexpr int NP = 16 * RG;  // weight pairs per lane and step
  using T_ = std::true_type;
  using F_ = std::false_type;
  __shared__ __attribute__((aligned(1024))) uint8_t kb0[C::TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t kb1[C::TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t vb0[C::TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t vb1[C::TILE_BYTES];

  // this workgroup's record (the grid is the record list, in the planner's
  // XCD-interleaved order); records with no tokens are idle padding
  const PrefillRec it = recs[blockIdx.x];
  if (it.n_tok == kDecodeBlock) {
    // NW / 4 decode units, one per group of four waves, each on LDS buffers
    // of its own (a decode block copies no tiles); the decode rows' K/V
    // stream from HBM while the tiles' workgroups keep the matrix cores busy
    using DL = decode_impl::DecodeLds<D, G>;
    static_assert(DL::O_BYTES <= C::TILE_BYTES && DL::SMALL_BYTES <= C::TILE_BYTES, "decode LDS");
    static_assert(NW == 4 || NW == 8, "decode groups");
    const int grp = uniform((int)threadIdx.x >> 8);
    const int u = grp == 0 ? it.tok0 : it.pos0;
    const bool active = u >= 0 && u < n_units;
    DecodeItem di{0, 0, 0, 0, -1, 0, 0, 0};
    if (active) di = dec[u / hkv];
    decode_unit<D, B, G>(di, active ? u % hkv : 0, active, (int)threadIdx.x & 255, q, k_cache,
                         v_cache, bt, out, part_o, part_lse, hq, hkv, mbr, scale_log2,
                         decode_impl::DecodeLdsPtrs{reinterpret_cast<float*>(grp == 0 ? kb0 : kb1),
                                                    grp == 0 ? vb0 : vb1});
    return;
  }
  if (it.n_tok <= 0) return;
  const int kvh = it.kvh;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = uniform(tid >> 6);
  const int col = lane & 31;
  const int g = lane >> 5;
  const int32_t* bt_row = bt + (int64_t)it.req * mbr;
  const int64_t blk_elems = (int64_t)hkv * B * D;
  const uint16_t* kbase = k_cache + (int64_t)kvh * B * D;
  const uint16_t* vbase = v_cache + (int64_t)kvh * B * D;
  const int n_step = (it.kv_end - it.kv_begin + BN - 1) / BN;

  // row groups: rows 32*RG*wave + 32*rg + col of the tile
  int tl[RG], qpos[RG];
  bool row_valid[RG];
  uint4 qreg[RG][NKS];  // Q^T operand: lane holds features [16 ks + 8 g, +8) of its row
  static_for<0, RG>([&](auto rg_c) {
    constexpr int rg = decltype(rg_c)::value;
    const int row = (wave * RG + rg) * 32 + col;
    tl[rg] = row / G;
    row_valid[rg] = tl[rg] < it.n_tok;
    qpos[rg] = it.pos0 + tl[rg];
    const uint16_t* qp = q + ((int64_t)(it.tok0 + (row_valid[rg] ? tl[rg] : 0)) * hq + kvh * G +
                              row % G) * D + g * 8;
    static_for<0, NKS>([&](auto ks_c) {
      constexpr int ks = decltype(ks_c)::value;
      qreg[rg][ks] = row_valid[rg] ? ld_global16(qp + ks * 16) : make_uint4(0, 0, 0, 0);
    });
  });

  // ---- gather geometry: wave w copies pieces [w*PW, (w+1)*PW) of every K
  // and V step; piece p lies in block p / PPB of the step, the same for K
  // and V.  Lane offsets (elements inside a block) are fixed for the item.
  const int lb_first = it.kv_begin >> C::LOG2B;
  const int lb_last = (it.kv_end - 1) >> C::LOG2B;
  uint32_t koff[PW], voff[PW];
  static_for<0, PW>([&](auto i_c) {
    constexpr int i = decltype(i_c)::value;
    const int p = wave * PW + i;
    const int key = p * C::KPP + lane / KCH;  // key of the step
    const int c = (lane % KCH) ^ (sigma(key & 15) & (KCH - 1));
    koff[i] = (uint32_t)((key & (B - 1)) * D + c * 8);
    const int d = (p % C::PPB) * C::V_ROWS + lane / C::V_LPR;
    const int h = B == 16 ? (((d >> 2) ^ (d >> 3)) & 1) : ((d >> 2) & 3);
    const int s = (lane % C::V_LPR) ^ h;
    voff[i] = (uint32_t)(d * B + s * 8);
  });
  // table entries of step st for this wave's blocks (clamped to the last
  // valid block: pieces past the range read valid memory and are masked)
  struct Blocks {
    int b[NBW];
  };
  auto blocks_of = [&](int st) {
    Blocks r;
    static_for<0, NBW>([&](auto j_c) {
      constexpr int j = decltype(j_c)::value;
      const int lb = min(lb_first + st * (BN / B) + (wave * PW) / C::PPB + j, lb_last);
      r.b[j] = uniform(bt_row[lb]);
    });
    return r;
  };
  auto issue = [&](const uint16_t* base, const uint32_t (&off)[PW], const Blocks& blk,
                   uint8_t* buf) {
    static_for<0, NBW>([&](auto j_c) {
      constexpr int j = decltype(j_c)::value;
      const uint16_t* src = base + (int64_t)blk.b[j] * blk_elems;
      static_for<j * (PW / NBW), (j + 1) * (PW / NBW)>([&](auto i_c) {
        constexpr int i = decltype(i_c)::value;
        copy16_to_lds(src, off[i] * 2u, buf + (wave * PW + i) * 1024);
      });
    });
  };
  // wait until at most `groups` of this wave's copy groups are in flight
  auto wait_groups = [&](int groups) {
    if (groups >= 2) wait_vmcnt<2 * PW>();
    else if (groups == 1) wait_vmcnt<PW>();
    else wait_vmcnt<0>();
  };

  f32x16_t oacc[RG][NDT];
  // scores of two consecutive steps; iteration st (parity p) reads sbuf[p]
  // (its step) and writes sbuf[p ^ 1] (the next step), so no copies
  f32x16_t sbuf[2][RG][2];  // [buffer][row group][32-key half]
  uint4 pk[RG][2][2];  // P^T operands of the current step: [row group][key half][16-key slice]
  static_for<0, RG>([&](auto rg_c) {
    constexpr int rg = decltype(rg_c)::value;
    static_for<0, NDT>([&](auto i_c) {
      constexpr int i = decltype(i_c)::value;
      static_for<0, 16>([&](auto r_c) { oacc[rg][i][decltype(r_c)::value] = 0.f; });
    });
    static_for<0, 2>([&](auto kt_c) {
      constexpr int kt = decltype(kt_c)::value;
      static_for<0, 16>([&](auto r_c) {
        sbuf[0][rg][kt][decltype(r_c)::value] = 0.f;
        sbuf[1][rg][kt][decltype(r_c)::value] = 0.f;
      });
    });
  });
  float m_run[RG], l_run[RG];  // running max of the scaled (base-2) scores; this half's sum
  static_for<0, RG>([&](auto rg_c) {
    m_run[decltype(rg_c)::value] = -INFINITY;
    l_run[decltype(rg_c)::value] = 0.f;
  });
  const int krow0 = sigma(col);

  // MFMA operand addresses inside a tile.  K read i: key half i / NKS, k-step
  // i % NKS, so each half's k-steps run back to back (one accumulator's chain
  // at a time keeps the matrix pipe fuller, with two waves per SIMD, than
  // alternating two accumulators).  Its swizzled chunk differs per k-step, so
  // one lane offset per k-step, the key half being a constant (the swizzle
  // repeats every 16 keys).
  // V read i: 16-key slice i / NDT, feature tile i % NDT; the swizzle depends
  // on the lane and, for 32-key blocks, on the slice parity.  The offsets are
  // made opaque so the compiler adds buffer and tile offsets as immediates
  // instead of building one address register per buffer.
  uint32_t kofs[NKS], vofs[B == 16 ? 1 : 2];
  static_for<0, NKS>([&](auto ks_c) {
    constexpr int ks = decltype(ks_c)::value;
    kofs[ks] = opaque((uint32_t)L::k_off(krow0, 2 * ks + g));
  });
  static_for<0, (B == 16 ? 1 : 2)>([&](auto p_c) {
    constexpr int par = decltype(p_c)::value;
    vofs[par] = opaque((uint32_t)(L::v_off(0, col, par * 2 + g) - L::K_BYTES));
  });
  auto kop = [&](const uint8_t* kb, auto i_c) {
    constexpr int i = decltype(i_c)::value;
    return *reinterpret_cast<const uint4*>(kb + kofs[i % NKS] + (i / NKS) * 32 * D * 2);
  };
  auto vop = [&](const uint8_t* vb, auto i_c) {
    constexpr int i = decltype(i_c)::value;
    constexpr int ks2 = i / NDT, dt = i % NDT;
    // block ks2*16/B, feature row dt*32 + col, slot ((ks2*16) % B)/8 + g
    constexpr int imm = (ks2 * 16 / B) * D * B * 2 + dt * 32 * B * 2;
    return *reinterpret_cast<const uint4*>(vb + vofs[B == 16 ? 0 : (ks2 & 1)] + imm);
  };
  // keys of step st that a row sees: [k0, k0 + lim); register r of half g
  // holds key kt*32 + acc_key(r, 0) + 8g
  auto mask_scores = [&](f32x16_t (&sc)[RG][2], int st) {
    const int k0 = it.kv_begin + st * BN;
    static_for<0, RG>([&](auto rg_c) {
      constexpr int rg = decltype(rg_c)::value;
      const int limg = min(qpos[rg] + 1, it.kv_end) - k0 - 8 * g;
      static_for<0, 2>([&](auto kt_c) {
        constexpr int kt = decltype(kt_c)::value;
        static_for<0, 16>([&](auto r_c) {
          constexpr int r = decltype(r_c)::value;
          if (kt * 32 + acc_key(r, 0) >= limg) sc[rg][kt][r] = -INFINITY;
        });
      });
    });
  };

  // Weight pair j (0 .. 16*RG-1) of a step: row group j >> 4, scores 2(j&7), +1 of
  // key half (j >> 3) & 1, packed into word j & 3 of pk[rg][kt][(j >> 2) & 1].
  auto exp_pair = [&](auto par_c, auto j_c, float& p0, float& p1) {
    constexpr int P = decltype(par_c)::value, j = decltype(j_c)::value;
    constexpr int rg = j >> 4, kt = (j >> 3) & 1, r = 2 * (j & 7);
    p0 = __builtin_amdgcn_exp2f(sbuf[P][rg][kt][r]);
    p1 = __builtin_amdgcn_exp2f(sbuf[P][rg][kt][r + 1]);
  };
  auto put_pair = [&](auto j_c, float p0, float p1) {
    constexpr int j = decltype(j_c)::value;
    set_word(pk[j >> 4][(j >> 3) & 1][(j >> 2) & 1], j & 3, pack_bf16x2(p0, p1));
  };

  auto keep_pk = [&]() {
    static_for<0, RG>([&](auto rg_c) {
      static_for<0, 4>([&](auto w_c) {
        constexpr int rg = decltype(rg_c)::value, w = decltype(w_c)::value;
        keep(get_word(pk[rg][w >> 1][w & 1], 0));
        keep(get_word(pk[rg][w >> 1][w & 1], 1));
        keep(get_word(pk[rg][w >> 1][w & 1], 2));
        keep(get_word(pk[rg][w >> 1][w & 1], 3));
      });
    });
  };
  auto keep_sbuf = [&](auto buf_c) {
    static_for<0, RG>([&](auto rg_c) {
      static_for<0, 2>([&](auto kt_c) {
        static_for<0, 16>([&](auto r_c) {
          keep(sbuf[decltype(buf_c)::value][decltype(rg_c)::value][decltype(kt_c)::value]
                   [decltype(r_c)::value]);
        });
      });
    });
  };

  // ---- phase K: snext = K . Q^T from kb, interleaved with P = exp2(scur).
  // Read i carries the exponentials of pairs [i*NP/NQK, (i+1)*NP/NQK) and
  // the packing of the pair before each (no packing waits on its own exps).
  auto phase_k = [&](const uint8_t* kb, auto par_c, auto with_exp_c) {
    constexpr bool WITH_EXP = decltype(with_exp_c)::value;
    constexpr int P = decltype(par_c)::value;
    auto& snext = sbuf[P ^ 1];
    static_for<0, RG>([&](auto rg_c) {
      static_for<0, 2>([&](auto kt_c) {
        static_for<0, 16>([&](auto r_c) {
          snext[decltype(rg_c)::value][decltype(kt_c)::value][decltype(r_c)::value] = 0.f;
        });
      });
    });
    uint4 ring[kRing];
    static_for<0, kRing>([&](auto i_c) {
      constexpr int i = decltype(i_c)::value;
      ring[i] = kop(kb, i_c);
    });
    float pa = 0.f, pb = 0.f;
    static_for<0, NQK>([&](auto i_c) {
      constexpr int i = decltype(i_c)::value;
      const uint4 a = ring[i % kRing];
      if constexpr (i + kRing < NQK) ring[i % kRing] = kop(kb, std::integral_constant<int, i + kRing>());
      static_for<0, RG>([&](auto rg_c) {
        constexpr int rg = decltype(rg_c)::value;
        snext[rg][i / NKS] = mfma32x32x16(a, qreg[rg][i % NKS], snext[rg][i / NKS]);
      });
      if constexpr (WITH_EXP) {
        static_for<i * NP / NQK, (i + 1) * NP / NQK>([&](auto j_c) {
          constexpr int j = decltype(j_c)::value;
          float p0, p1;
          exp_pair(par_c, j_c, p0, p1);
          if constexpr (j > 0) put_pair(std::integral_constant<int, j - 1>(), pa, pb);
          pa = p0, pb = p1;
        });
      }
      __builtin_amdgcn_sched_barrier(0);
    });
    if constexpr (WITH_EXP) {
      put_pair(std::integral_constant<int, NP - 1>(), pa, pb);
      keep_pk();
    }
  };
  // phase K of the last step: only the exponentials
  auto exp_only = [&](auto par_c) {
    static_for<0, NP>([&](auto j_c) {
      float p0, p1;
      exp_pair(par_c, j_c, p0, p1);
      put_pair(j_c, p0, p1);
    });
    keep_pk();
  };

  // ---- phase V: O += V^T . P^T from vb.  With a next step, interleaved with
  // the row sums of P and the row max of snext (first half of the reads), the
  // lazy max update (middle read) and snext -> snext * scale - max (second
  // half).  VMASK zeroes the values of keys past the range (partial last
  // step).  Returns whether any lane moved its max (O must then be scaled).
  auto phase_v = [&](const uint8_t* vb, auto par_c, auto has_next_c, float (&alpha)[RG]) -> bool {
    constexpr int P = decltype(par_c)::value;
    auto& snext = sbuf[P ^ 1];
    constexpr bool HAS_NEXT = decltype(has_next_c)::value;
    constexpr uint32_t ones = 0x3f803f80u;  // bf16 pair (1, 1)
    constexpr int H = NPV / 2;              // read that carries the max update
    auto vload = [&](auto i_c) { return vop(vb, i_c); };
    uint4 ring[kRing];
    static_for<0, kRing>([&](auto i_c) { ring[decltype(i_c)::value] = vload(i_c); });
    float mt[RG], neg_m[RG];
    bool need[RG];
    static_for<0, RG>([&](auto rg_c) {
      constexpr int rg = decltype(rg_c)::value;
      mt[rg] = -INFINITY, neg_m[rg] = 0.f, need[rg] = false, alpha[rg] = 1.f;
    });
    static_for<0, NPV>([&](auto i_c) {
      constexpr int i = decltype(i_c)::value;
      const uint4 a = ring[i % kRing];
      if constexpr (i + kRing < NPV) ring[i % kRing] = vload(std::integral_constant<int, i + kRing>());
      constexpr int ks2 = i / NDT;
      static_for<0, RG>([&](auto rg_c) {
        constexpr int rg = decltype(rg_c)::value;
        oacc[rg][i % NDT] = mfma32x32x16(a, pk[rg][ks2 >> 1][ks2 & 1], oacc[rg][i % NDT]);
      });
      if constexpr (i < H) {
        static_for<i * NP / H, (i + 1) * NP / H>([&](auto j_c) {
          constexpr int j = decltype(j_c)::value;
          l_run[j >> 4] = dot2_bf16(get_word(pk[j >> 4][(j >> 3) & 1][(j >> 2) & 1], j & 3), ones,
                                    l_run[j >> 4]);
          if constexpr (HAS_NEXT) {
            constexpr int rg = j >> 4, kt = (j >> 3) & 1, r = 2 * (j & 7);
            mt[rg] = __builtin_fmaxf(__builtin_fmaxf(mt[rg], snext[rg][kt][r]),
                                     snext[rg][kt][r + 1]);
          }
        });
      } else if constexpr (i == H) {
        if constexpr (HAS_NEXT) {
          static_for<0, RG>([&](auto rg_c) {
            constexpr int rg = decltype(rg_c)::value;
            const float m = halves_max(mt[rg]) * scale_log2;
            need[rg] = m > m_run[rg] + kRescaleThreshold;
            alpha[rg] = need[rg] ? __builtin_amdgcn_exp2f(m_run[rg] - m) : 1.f;  // -inf: 0
            m_run[rg] = need[rg] ? m : m_run[rg];
            neg_m[rg] = m_run[rg] == -INFINITY ? 0.f : -m_run[rg];
          });
        }
      } else {
        if constexpr (HAS_NEXT) {
          constexpr int R = NPV - H - 1;
          static_for<(i - H - 1) * 32 * RG / R, (i - H) * 32 * RG / R>([&](auto j_c) {
            constexpr int j = decltype(j_c)::value;
            constexpr int rg = j >> 5, kt = (j >> 4) & 1, r = j & 15;
            snext[rg][kt][r] = __builtin_fmaf(snext[rg][kt][r], scale_log2, neg_m[rg]);
          });
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    });
    if constexpr (HAS_NEXT) keep_sbuf(std::integral_constant<int, P ^ 1>());
    bool any = false;
    static_for<0, RG>([&](auto rg_c) { any = any || need[decltype(rg_c)::value]; });
    return HAS_NEXT && __builtin_amdgcn_ballot_w64(any) != 0;
  };
  auto rescale = [&](const float (&alpha)[RG]) {
    static_for<0, RG>([&](auto rg_c) {
      constexpr int rg = decltype(rg_c)::value;
      static_for<0, NDT>([&](auto i_c) {
        constexpr int i = decltype(i_c)::value;
        static_for<0, 16>([&](auto r_c) { oacc[rg][i][decltype(r_c)::value] *= alpha[rg]; });
      });
    });
  };
  // prologue version of the max update: O and l are still zero
  auto first_max = [&]() {
    static_for<0, RG>([&](auto rg_c) {
      constexpr int rg = decltype(rg_c)::value;
      float mt = -INFINITY;
      static_for<0, 16>([&](auto j_c) {
        constexpr int j = decltype(j_c)::value;
        mt = __builtin_fmaxf(__builtin_fmaxf(mt, sbuf[0][rg][j >> 3][2 * (j & 7)]),
                             sbuf[0][rg][j >> 3][2 * (j & 7) + 1]);
      });
      m_run[rg] = halves_max(mt) * scale_log2;
      const float neg_m = m_run[rg] == -INFINITY ? 0.f : -m_run[rg];
      static_for<0, 2>([&](auto kt_c) {
        constexpr int kt = decltype(kt_c)::value;
        static_for<0, 16>([&](auto r_c) {
          constexpr int r = decltype(r_c)::value;
          sbuf[0][rg][kt][r] = __builtin_fmaf(sbuf[0][rg][kt][r], scale_log2, neg_m);
        });
      });
    });
  };
  // Zeroes the values of keys [vlim, BN) of the V tile vb: the 16-byte slot
  // (block bi, feature d, 8 keys) of step keys [8x, 8x + 8), x = bi*B/8 + s.
  const bool partial = (it.kv_end - it.kv_begin) % BN != 0;
  auto zero_tail = [&](uint8_t* vb, int vlim) {
    constexpr int SLOTS = BN / 8;  // 16-byte slots per feature row of a step
    for (int x = tid; x < SLOTS * D; x += NW * 64) {
      const int sl = x % SLOTS, d = x / SLOTS;
      const int first = sl * 8;
      if (first + 8 <= vlim) continue;
      uint4* p = reinterpret_cast<uint4*>(
          vb + (L::v_off(sl / (B / 8), d, sl % (B / 8)) - L::K_BYTES));
      uint4 v = make_uint4(0, 0, 0, 0);
      if (first < vlim) {  // keep keys below vlim
        v = *p;
        static_for<0, 4>([&](auto e_c) {
          constexpr int e = decltype(e_c)::value;
          const uint32_t lo = first + 2 * e < vlim ? 0x0000ffffu : 0u;
          const uint32_t hi = first + 2 * e + 1 < vlim ? 0xffff0000u : 0u;
          set_word(v, e, get_word(v, e) & (lo | hi));
        });
      }
      *p = v;
    }
  };

  // first edge step: steps >= e_step cross the causal diagonal or the range end
  const int lim = min(it.pos0 + 1, it.kv_end) - BN;
  const int e_step = it.kv_begin > lim ? 0 : (lim - it.kv_begin) / BN + 1;

  // ---- prologue: copies K0 -> kb0, K1 -> kb1, V0 -> vb0; S_0 = K0 . Q^T
  {
    const Blocks b0 = blocks_of(0);
    issue(kbase, koff, b0, kb0);
    if (n_step > 1) issue(kbase, koff, blocks_of(1), kb1);
    issue(vbase, voff, b0, vb0);
  }
  wait_groups(n_step > 1 ? 2 : 1);
  barrier();
  phase_k(kb0, std::integral_constant<int, 1>(), F_());  // writes sbuf[0]
  if (e_step == 0) mask_scores(sbuf[0], 0);
  first_max();

  // ---- main loop.  Iteration st (parity p = st & 1): phase K reads K_{st+1}
  // from kb[1-p], phase V reads V_st from vb[p].  Copies: V_{st+1} into vb[1-p]
  // after the phase-K barrier (phase V of st-1 read it last); K_{st+3} into
  // kb[1-p] after the phase-V barrier (phase K of st read it last); K_2 into
  // kb0 at st = 0, before V_1.  Buffers are chosen at compile time so every
  // LDS access names its array.
  Blocks blk_k = n_step > 2 ? blocks_of(2) : Blocks{};  // entries of the next K copy
  Blocks blk_v = n_step > 1 ? blocks_of(1) : Blocks{};  // entries of the next V copy
  auto iter = [&](int st, auto par_c, auto last_c) {
    constexpr bool PAR = decltype(par_c)::value;
    constexpr bool LAST = decltype(last_c)::value;
    constexpr std::integral_constant<int, PAR ? 1 : 0> P_;
    uint8_t* kb_read = PAR ? kb0 : kb1;
    uint8_t* vb_read = PAR ? vb1 : vb0;
    uint8_t* vb_fill = PAR ? vb0 : vb1;
    // -- phase K
    if constexpr (!LAST) wait_groups(st == 0 ? 1 : 1 + (st + 2 < n_step));
    barrier();
    if constexpr (!PAR) {
      if (st == 0 && n_step > 2) issue(kbase, koff, blk_k, kb0);
    }
    if constexpr (!LAST) issue(vbase, voff, blk_v, vb_fill);
    if constexpr (!PAR) {
      if (st == 0 && n_step > 3) blk_k = blocks_of(3);
    }
    if (st + 2 < n_step) blk_v = blocks_of(st + 2);
    if constexpr (LAST) {
      exp_only(P_);
    } else {
      phase_k(kb_read, P_, T_());
      if (st + 1 >= e_step) mask_scores(sbuf[PAR ? 0 : 1], st + 1);
    }
    // -- phase V
    wait_groups((st + 2 < n_step) + (st + 1 < n_step));
    barrier();
    if (st + 3 < n_step) {
      issue(kbase, koff, blk_k, kb_read);
      if (st + 4 < n_step) blk_k = blocks_of(st + 4);
    }
    if constexpr (LAST) {
      if (partial) {  // values of keys past the range may be any bits (NaN)
        zero_tail(vb_read, it.kv_end - (it.kv_begin + st * BN));
        barrier();
      }
    }
    float alpha[RG];
    const bool resc = phase_v(vb_read, P_, std::integral_constant<bool, !LAST>(), alpha);
    if constexpr (!LAST) {
      if (resc) rescale(alpha);
      static_for<0, RG>([&](auto rg_c) {
        constexpr int rg = decltype(rg_c)::value;
        l_run[rg] *= alpha[rg];
      });
    }
  };
  // iterations in pairs (even parity first), then the last one
  int st = 0;
  for (; st + 2 < n_step; st += 2) {
    iter(st, F_(), F_());
    iter(st + 1, T_(), F_());
  }
  if (st + 1 < n_step) {
    iter(st, F_(), F_());
    iter(st + 1, T_(), T_());
  } else {
    iter(st, F_(), T_());
  }

  // ---- finish: the two lane halves hold disjoint keys of the same query.
  // Each wave stages its rows through LDS (a slice of the four tile buffers,
  // free once every wave is past the last step) and stores whole rows: 16
  // lanes per 256-byte run, instead of 16-byte pieces of 32 rows per store.
  if constexpr (RG == 1) {
    constexpr int SLICE = 4 * C::TILE_BYTES / NW;   // staging bytes per wave
    barrier();  // every wave has read its last V tile
    const int bsel = (wave * SLICE) / C::TILE_BYTES;
    uint8_t* const st = (bsel == 0 ? kb0 : bsel == 1 ? kb1 : bsel == 2 ? vb0 : vb1) +
                        (wave * SLICE) % C::TILE_BYTES;
    const float l_tot = halves_sum(l_run[0]);
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const int wrow0 = wave * 32;  // first tile row of this wave
    if (it.part < 0) {
      // bf16 rows of D * 2 bytes; 16-byte unit u of row r stored at u ^ (r % U)
      constexpr int RB = D * 2, U = RB / 16;
      static_assert(32 * RB <= SLICE, "bf16 staging");
      static_for<0, NDT>([&](auto dt_c) {
        constexpr int dt = decltype(dt_c)::value;
        static_for<0, 4>([&](auto i_c) {
          constexpr int i = decltype(i_c)::value;
          uint2 w;
          w.x = pack_bf16x2(oacc[0][dt][4 * i + 0] * inv, oacc[0][dt][4 * i + 1] * inv);
          w.y = pack_bf16x2(oacc[0][dt][4 * i + 2] * inv, oacc[0][dt][4 * i + 3] * inv);
          constexpr int u = dt * 4 + i;  // features [8u, 8u + 8): this lane's half g
          *reinterpret_cast<uint2*>(st + col * RB + ((u ^ (col % U)) * 16) + 8 * g) = w;
        });
      });
      constexpr int RPI = 64 / U;  // rows per store instruction
      static_for<0, 32 / RPI>([&](auto k_c) {
        constexpr int k = decltype(k_c)::value;
        const int r = k * RPI + lane / U, c = lane % U;
        const uint4 v = *reinterpret_cast<const uint4*>(st + r * RB + ((c ^ (r % U)) * 16));
        const int row = wrow0 + r, t = row / G;
        if (t < it.n_tok)
          *reinterpret_cast<uint4*>(
              out + ((int64_t)(it.tok0 + t) * hq + kvh * G + row % G) * D + c * 8) = v;
      });
    } else {
      // fp32 rows in PASSES column passes of DP features (RB bytes a row)
      constexpr int PASSES = 32 * D * 4 > SLICE ? 2 : 1;
      constexpr int DP = D / PASSES, RB = DP * 4, U = RB / 16;
      static_assert(32 * RB <= SLICE && U <= 32, "fp32 staging");
      static_for<0, PASSES>([&](auto p_c) {
        constexpr int pass = decltype(p_c)::value;
        static_for<pass * NDT / PASSES, (pass + 1) * NDT / PASSES>([&](auto dt_c) {
          constexpr int dt = decltype(dt_c)::value;
          static_for<0, 4>([&](auto i_c) {
            constexpr int i = decltype(i_c)::value;
            const int u = (dt - pass * NDT / PASSES) * 8 + 2 * i + g;  // features [4u, 4u + 4)
            *reinterpret_cast<float4*>(st + col * RB + ((u ^ (col % U)) * 16)) =
                make_float4(oacc[0][dt][4 * i + 0] * inv, oacc[0][dt][4 * i + 1] * inv,
                            oacc[0][dt][4 * i + 2] * inv, oacc[0][dt][4 * i + 3] * inv);
          });
        });
        constexpr int RPI = 64 / U;
        static_for<0, 32 / RPI>([&](auto k_c) {
          constexpr int k = decltype(k_c)::value;
          const int r = k * RPI + lane / U, c = lane % U;
          const float4 v = *reinterpret_cast<const float4*>(st + r * RB + ((c ^ (r % U)) * 16));
          const int row = wrow0 + r;
          if (row / G < it.n_tok)
            *reinterpret_cast<float4*>(part_o + (int64_t)(it.part + row) * D + pass * DP + c * 4) =
                v;
        });
      });
      if (g == 0 && row_valid[0]) part_lse[it.part + wrow0 + col] =
          l_tot > 0.f ? m_run[0] + __log2f(l_tot) : -INFINITY;
    }
  } else {
    // row groups of more than one: each lane stores its own pieces
    static_for<0, RG>([&](auto rg_c) {
      constexpr int rg = decltype(rg_c)::value;
      const float l_tot = halves_sum(l_run[rg]);
      if (!row_valid[rg]) return;
      const int row = (wave * RG + rg) * 32 + col;
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      if (it.part < 0) {
        uint16_t* op = out + ((int64_t)(it.tok0 + tl[rg]) * hq + kvh * G + row % G) * D + 4 * g;
        static_for<0, NDT>([&](auto dt_c) {
          constexpr int dt = decltype(dt_c)::value;
          static_for<0, 4>([&](auto i_c) {
            constexpr int i = decltype(i_c)::value;
            uint2 w;
            w.x = pack_bf16x2(oacc[rg][dt][4 * i + 0] * inv, oacc[rg][dt][4 * i + 1] * inv);
            w.y = pack_bf16x2(oacc[rg][dt][4 * i + 2] * inv, oacc[rg][dt][4 * i + 3] * inv);
            *reinterpret_cast<uint2*>(op + dt * 32 + 8 * i) = w;
          });
        });
      } else {
        const int prow = it.part + row;
        float* pp = part_o + (int64_t)prow * D + 4 * g;
        static_for<0, NDT>([&](auto dt_c) {
          constexpr int dt = decltype(dt_c)::value;
          static_for<0, 4>([&](auto i_c) {
            constexpr int i = decltype(i_c)::value;
            *reinterpret_cast<float4*>(pp + dt * 32 + 8 * i) =
                make_float4(oacc[rg][dt][4 * i + 0] * inv, oacc[rg][dt][4 * i + 1] * inv,
                            oacc[rg][dt][4 * i + 2] * inv, oacc[rg][dt][4 * i + 3] * inv);
          });
        });
        if (g == 0) part_lse[prow] = l_tot > 0.f ? m_run[rg] + __log2f(l_tot) : -INFINITY;
      }
    });
  }
}

template <int D, int B, int G, int NW>
static hipError_t launch_prefill_t(const PrefillRec* recs, int n, int n_units, const AttnArgs& a,
                                   hipStream_t s) {
  hipLaunchKernelGGL((prefill_kernel<D, B, G, NW, kPrefillRG>), dim3(n), dim3(NW * 64), 0, s, recs,
                     a.q, a.k_cache, a.v_cache, a.bt, a.out, a.part_o, a.part_lse, a.hq, a.hkv,
                     a.mbr, a.scale_log2, a.decode, n_units);
  return hipGetLastError();
}

template <int D, int B, int NW>
static hipError_t launch_prefill_g(int G, const PrefillRec* recs, int n, int n_units,
                                   const AttnArgs& a, hipStream_t s) {
  switch (G) {
    case 1: return launch_prefill_t<D, B, 1, NW>(recs, n, n_units, a, s);
    case 2: return launch_prefill_t<D, B, 2, NW>(recs, n, n_units, a, s);
    case 4: return launch_prefill_t<D, B, 4, NW>(recs, n, n_units, a, s);
    case 8: return launch_prefill_t<D, B, 8, NW>(recs, n, n_units, a, s);
  }
  return hipErrorInvalidValue;
}

template <int NW>
static hipError_t launch_prefill_w(int D, int G, const PrefillRec* recs, int n, int n_units,
                                   const AttnArgs& a, hipStream_t s) {
  if (D == 128 && a.block_size == 16) return launch_prefill_g<128, 16, NW>(G, recs, n, n_units, a, s);
  if (D == 128 && a.block_size == 32) return launch_prefill_g<128, 32, NW>(G, recs, n, n_units, a, s);
  if (D == 64 && a.block_size == 16) return launch_prefill_g<64, 16, NW>(G, recs, n, n_units, a, s);
  if (D == 64 && a.block_size == 32) return launch_prefill_g<64, 32, NW>(G, recs, n, n_units, a, s);
  return hipErrorInvalidValue;
}

// 256-row and 128-row tiles: 32 * kPrefillRG rows per wave; one workgroup per
// record.  The launch the plan names also runs the decode units.
hipError_t launch_prefill(int D, int G, const AttnArgs& a, hipStream_t s) {
  constexpr int kWide = kPrefillRowsWide / (32 * kPrefillRG), kNarrow = kPrefillRows / (32 * kPrefillRG);
  const int units = a.n_decode * a.hkv;
  hipError_t e = hipSuccess;
  if (a.n_prefill_wide_items > 0)
    e = launch_prefill_w<kWide>(D, G, a.prefill_wide, a.n_prefill_wide_items,
                                a.decode_in_prefill == 2 ? units : 0, a, s);
  if (e == hipSuccess && a.n_prefill_items > 0)
    e = launch_prefill_w<kNarrow>(D, G, a.prefill, a.n_prefill_items,
                                  a.decode_in_prefill == 1 ? units : 0, a, s);
  return e;
}

}  // namespace cpattn
