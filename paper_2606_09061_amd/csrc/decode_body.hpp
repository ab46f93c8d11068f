// Split-K decode attention for one (row, block range, kv head) unit, run by
// four waves: the body of the decode kernel, and of the decode blocks that
// the prefill kernel runs beside its tiles when a step's decode rows are
// overlapped with its prefill chunks.
//
// Decode is memory-bandwidth bound (Sec. 1 and 2.1 of the paper): every key
// and value of the context is read once per kv head and used by only G q
// heads, so the unit is organised around streaming the paged blocks at full
// HBM rate and keeping the VALU work per byte small.
//
// The range is walked in tiles of 16 keys (a block holds B / 16), wave w
// taking tiles w, w+4, ..., with the next tile's loads issued before the
// current one is used.
//
// Per tile every lane issues NL 16-byte loads of K and NL of V.
//   K tile [16][D] (contiguous inside the block): instruction i of the wave
//     reads bytes [1024 i, 1024 i + 1024) of it; lane holds 8 features
//     (chunk lane % (D/8)) of NL keys.
//     Scores: bf16 dot2 against the lane's 8 features of each of the G q
//     heads, then a butterfly reduce-scatter over the D/8 lanes of a key row
//     (DPP inside rows of 16) leaves each lane with whole scores.
//   V tile: the tile's 16 slots of each feature row of the [D][B] block; a
//     lane holds 8 consecutive keys (chunk lane % 2) of NL feature rows.
//     Weights of those 8 keys come from a per-wave LDS slot, and the
//     weighted sum is again bf16 dot2 with fp32 accumulation.
// Online softmax runs in base 2 with a lazily updated running max per head.
// The 4 waves' (max, sum, output) states are combined through LDS; a unit
// covering the whole context writes the bf16 output, a split unit writes its
// normalised fp32 output and log2-sum-exp for the merge pass.
#pragma once

#include "device.hpp"

namespace cpattn {

namespace decode_impl {

constexpr int TK = 16;  // keys per tile

// Butterfly reduce-scatter of N partial sums over the lanes selected by
// lane bits Dist, Dist/2, ..., 1.  While more than one value is left the
// lane keeps the half picked by its own bit and adds its partner's copy of
// that half; once one value is left the remaining bits are all-reduced.
template <int N, int Dist>
__device__ __forceinline__ void reduce_scatter(float* v, int lane) {
  if constexpr (Dist >= 1) {
    if constexpr (N > 1) {
      constexpr int H = N / 2;
      const bool hi = (lane & Dist) != 0;
#pragma unroll
      for (int k = 0; k < H; ++k) {
        const float keep = hi ? v[H + k] : v[k];
        const float send = hi ? v[k] : v[H + k];
        v[k] = keep + lane_partner<Dist>(send);
      }
      reduce_scatter<H, Dist / 2>(v, lane);
    } else {
      v[0] += lane_partner<Dist>(v[0]);
      reduce_scatter<1, Dist / 2>(v, lane);
    }
  }
}

// LDS of one unit, in bytes: weights [4][G][TK] bf16, wave states
// [4][G][D] + 2 x [4][G] fp32, query [G][D] bf16 (when kept in LDS).
template <int D, int G>
struct DecodeLds {
  static constexpr int kWaves = kDecodeWaves;
  static constexpr bool kQLds = G * D >= 1024;  // query in LDS (3 waves per SIMD)
  static constexpr int P_BYTES = kWaves * G * TK * 2;
  static constexpr int O_BYTES = kWaves * G * D * 4;
  static constexpr int ML_BYTES = kWaves * G * 4;
  static constexpr int Q_BYTES = kQLds ? G * D * 2 : 0;
  // the small arrays together (weights first: 16-byte aligned reads)
  static constexpr int SMALL_BYTES = P_BYTES + 2 * ML_BYTES + Q_BYTES;
};

// Pointers into LDS for one unit.  `o` holds O_BYTES; `small` SMALL_BYTES,
// 16-byte aligned.
struct DecodeLdsPtrs {
  float* o;
  uint8_t* small;
};

}  // namespace decode_impl

// Runs one decode unit with the four waves whose workgroup-local thread ids
// are `tid` in [0, 256).  Every wave of the workgroup must call this the
// same number of times, with active == false for a group that has no unit:
// the unit synchronises the whole workgroup (one or two barriers).
template <int D, int B, int G>
__device__ __forceinline__ void decode_unit(
    const DecodeItem& it, int kvh, bool active, int tid, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ k_cache, const uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ bt, uint16_t* __restrict__ out, float* __restrict__ part_o,
    float* __restrict__ part_lse, int hq, int hkv, int mbr, float scale_log2,
    decode_impl::DecodeLdsPtrs lds) {
  using namespace decode_impl;
  using Lds = DecodeLds<D, G>;
  constexpr int NL = TK * D * 2 / 1024; // 16-byte loads per lane per tile, K and V each
  constexpr int LPR = D / 8;            // lanes sharing one K row
  constexpr int TPI = 64 / LPR;         // K rows per load instruction
  constexpr int LPD = TK / 8;           // lanes sharing one V feature row
  constexpr int DPI = 64 / LPD;         // V feature rows per load instruction
  constexpr int NV = NL * G;            // partial scores per lane
  constexpr int NVL = NV >= LPR ? NV / LPR : 1;
  constexpr int DUP = NV >= LPR ? 1 : LPR / NV;  // lanes holding the same score
  constexpr int kWaves = Lds::kWaves;
  constexpr bool kQLds = Lds::kQLds;
  static_assert(NL * TPI == TK && NL * DPI == D && B % TK == 0 && LPD == 2, "tile geometry");

  uint16_t* p_lds = reinterpret_cast<uint16_t*>(lds.small);                // [kWaves][G][TK]
  float* red_o = lds.o;                                                     // [kWaves][G][D]
  float* red_m = reinterpret_cast<float*>(lds.small + Lds::P_BYTES);        // [kWaves][G]
  float* red_l = red_m + kWaves * G;                                        // [kWaves][G]
  uint16_t* q_lds = reinterpret_cast<uint16_t*>(lds.small + Lds::P_BYTES + 2 * Lds::ML_BYTES);

  const int part = it.part < 0 ? -1 : it.part + kvh * it.part_kvh_stride;
  const int lane = tid & 63;
  // wave-uniform in a scalar register, so that the tile loop, its branches
  // and the block-table reads are scalar and leave the vector memory counter
  // to the K/V loads (the prefetched tile stays in flight during a tile)
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int sub = lane % LPR;
  const int krow = lane / LPR;
  const int tc = lane % LPD;
  const int vrow = lane / LPD;

  // Large head groups keep the query in LDS (read again every tile) so that
  // the kernel stays at three waves per SIMD; small ones keep it in registers.
  uint4 qv[kQLds ? 1 : G];
  if constexpr (kQLds) {
    if (active) {
      const uint16_t* qb = q + ((int64_t)it.tok * hq + kvh * G) * D;
      for (int x = tid; x < G * D / 8; x += 256)
        *reinterpret_cast<uint4*>(q_lds + x * 8) = ld_global16(qb + x * 8);
    }
    __syncthreads();
  } else {
    if (active) {
      const uint16_t* qb = q + ((int64_t)it.tok * hq + kvh * G) * D + sub * 8;
#pragma unroll
      for (int h = 0; h < G; ++h) qv[h] = ld_global16(qb + h * D);
    }
    __builtin_amdgcn_sched_barrier(0);  // query loads stay older than the tile loads
  }
  auto qop = [&](int h) -> uint4 { return *reinterpret_cast<const uint4*>(q_lds + h * D + sub * 8); };

  // reduced-score slot k of this lane -> (head, key within tile)
  int s_head[NVL], s_key[NVL];
#pragma unroll
  for (int k = 0; k < NVL; ++k) {
    const int v = NV >= LPR ? sub * NVL + k : sub / DUP;
    s_head[k] = v % G;
    s_key[k] = (v / G) * TPI + krow;
  }
  const bool owner = (sub % DUP) == 0;

  float m_run[G], m_lane[NVL], l_lane[NVL], o[G][NL];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m_run[h] = -INFINITY;
#pragma unroll
    for (int i = 0; i < NL; ++i) o[h][i] = 0.f;
  }
#pragma unroll
  for (int k = 0; k < NVL; ++k) {
    m_lane[k] = -INFINITY;
    l_lane[k] = 0.f;
  }

  const int64_t head_elems = (int64_t)B * D;
  const int kt0 = it.kv_begin / TK;
  const int kt1 = (it.kv_end + TK - 1) / TK;
  const int32_t* bt_row = bt + (int64_t)it.req * mbr;
  // tile t: K rows [t*TK % B, +TK) of its block (contiguous), and the same
  // slots of every V feature row of the block.  Each K/V byte is read by one
  // workgroup only, so the loads are non-temporal (streamed past the caches
  // instead of displacing lines other workgroups reuse).
  auto load_tile = [&](int t, uint4* kr, uint4* vr) {
    const int64_t blk = ((int64_t)bt_row[(t * TK) / B] * hkv + kvh) * head_elems;
    const int toff = (t * TK) % B;
    const uint16_t* kp = k_cache + blk + toff * D + lane * 8;
    const uint16_t* vp = v_cache + blk + vrow * B + toff + tc * 8;
#pragma unroll
    for (int i = 0; i < NL; ++i) kr[i] = ld_global16_nt(kp + i * 512);
#pragma unroll
    for (int i = 0; i < NL; ++i) vr[i] = ld_global16_nt(vp + i * DPI * B);
  };

  // one tile: scores, online softmax, weighted values
  auto step = [&](const uint4* kr, uint4* vr, int kt) {
    const int valid = min(TK, it.kv_end - kt * TK);

    // ---- scores
    float sv[NV];
    auto score = [&](int i, int h, const uint4& qh) {
      float acc = 0.f;
      acc = dot2_bf16(kr[i].x, qh.x, acc);
      acc = dot2_bf16(kr[i].y, qh.y, acc);
      acc = dot2_bf16(kr[i].z, qh.z, acc);
      acc = dot2_bf16(kr[i].w, qh.w, acc);
      sv[i * G + h] = acc;
    };
    if constexpr (kQLds) {  // one LDS read of each head's query piece
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const uint4 qh = qop(h);
#pragma unroll
        for (int i = 0; i < NL; ++i) score(i, h, qh);
      }
    } else {
#pragma unroll
      for (int i = 0; i < NL; ++i)
#pragma unroll
        for (int h = 0; h < G; ++h) score(i, h, qv[h]);
    }
    reduce_scatter<NV, LPR / 2>(sv, lane);
    float s[NVL];
    bool grow = false;
#pragma unroll
    for (int k = 0; k < NVL; ++k) {
      s[k] = s_key[k] < valid ? sv[k] * scale_log2 : -INFINITY;
      grow |= s[k] > m_lane[k] + kRescaleThreshold;
    }
    if (__builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float x = -INFINITY;
#pragma unroll
        for (int k = 0; k < NVL; ++k)
          if (s_head[k] == h) x = fmaxf(x, s[k]);
        x = wave_max(x);
        const float mnew = fmaxf(m_run[h], x);
        const float alpha = (m_run[h] == -INFINITY) ? 0.f : exp2f(m_run[h] - mnew);
        m_run[h] = mnew;
#pragma unroll
        for (int i = 0; i < NL; ++i) o[h][i] *= alpha;
#pragma unroll
        for (int k = 0; k < NVL; ++k)
          if (s_head[k] == h) {
            l_lane[k] *= alpha;
            m_lane[k] = mnew;
          }
      }
    }
    // ---- weights -> LDS
#pragma unroll
    for (int k = 0; k < NVL; ++k) {
      const float p = exp2f(s[k] - m_lane[k]);
      const uint16_t pb = to_bf16(p);
      if (owner) {
        l_lane[k] += __uint_as_float((uint32_t)pb << 16);
        p_lds[(wave * G + s_head[k]) * TK + s_key[k]] = pb;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // ---- zero values of keys past the end of the range (may hold NaN)
    if (valid < TK) {
      const int t0 = tc * 8;
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        uint32_t* w = reinterpret_cast<uint32_t*>(&vr[i]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t lo = (t0 + 2 * e) < valid ? 0x0000ffffu : 0u;
          const uint32_t hi = (t0 + 2 * e + 1) < valid ? 0xffff0000u : 0u;
          w[e] &= (lo | hi);
        }
      }
    }
    // ---- weighted values (each head's 8 weights read just before use)
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const uint4 pv = *reinterpret_cast<const uint4*>(p_lds + (wave * G + h) * TK + tc * 8);
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        float acc = o[h][i];
        acc = dot2_bf16(vr[i].x, pv.x, acc);
        acc = dot2_bf16(vr[i].y, pv.y, acc);
        acc = dot2_bf16(vr[i].z, pv.z, acc);
        acc = dot2_bf16(vr[i].w, pv.w, acc);
        o[h][i] = acc;
      }
    }
    __builtin_amdgcn_wave_barrier();
  };

  // Two register sets in turn: the loads of a wave's next tile are in flight
  // while it works on the current one.  The prefetch is unconditional (past
  // the range it re-reads the range's last tile, which is unused) so that
  // the compiler's wait counts stay exact and never drain the prefetch.
  if (active) {
    uint4 ka[NL], va[NL], kb[NL], vb[NL];
    const int last = kt1 - 1;  // units are never empty
    int kt = kt0 + wave;
    load_tile(min(kt, last), ka, va);
    for (; kt < kt1; kt += 2 * kWaves) {
      load_tile(min(kt + kWaves, last), kb, vb);
      step(ka, va, kt);
      if (kt + kWaves >= kt1) break;
      load_tile(min(kt + 2 * kWaves, last), ka, va);
      step(kb, vb, kt + kWaves);
    }
  }

  // ---- combine inside the wave: feature rows are split over LPD lanes
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      float x = o[h][i];
      x += dpp<kXor1>(x);  // the two lanes of a V feature row
      o[h][i] = x;
    }
  float lsum[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float x = 0.f;
#pragma unroll
    for (int k = 0; k < NVL; ++k)
      if (s_head[k] == h && owner) x += l_lane[k];
    lsum[h] = wave_sum(x);
  }
  if (tc == 0) {
#pragma unroll
    for (int i = 0; i < NL; ++i)
#pragma unroll
      for (int h = 0; h < G; ++h) red_o[(wave * G + h) * D + i * DPI + vrow] = o[h][i];
  }
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      red_m[wave * G + h] = m_run[h];
      red_l[wave * G + h] = lsum[h];
    }
  }
  __syncthreads();
  if (!active) return;

  // ---- combine the waves and write
  for (int x = tid; x < G * D; x += 256) {
    const int h = x / D;
    const int d = x % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, red_m[w * G + h]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float mw = red_m[w * G + h];
      const float f = mw == -INFINITY ? 0.f : exp2f(mw - M);
      L += f * red_l[w * G + h];
      O += f * red_o[(w * G + h) * D + d];
    }
    const float val = L > 0.f ? O / L : 0.f;
    if (part < 0) {
      out[((int64_t)it.tok * hq + kvh * G + h) * D + d] = to_bf16(val);
    } else {
      part_o[(int64_t)(part + h) * D + d] = val;
      if (d == 0) part_lse[part + h] = L > 0.f ? M + __log2f(L) : -INFINITY;
    }
  }
}

}  // namespace cpattn
