// Paged KV append: scatters the batch's new K/V rows into their cache slots.
//
// One workgroup per (request, logical block) span of new tokens and kv head;
// the span list comes from device memory or, when short, from the kernel
// arguments (where a step's attention plan copy can share the launch).
// K rows are token-major inside a block, so each 16-byte chunk of a new K row
// is one aligned vector copy.  V is feature-major inside a block ([D][B]): a
// thread transposes an 8-slot x 8-feature tile in registers, reading token
// rows and writing feature runs with 16-byte accesses.  Every load is issued
// before the first store.
#include "copy_body.hpp"
#include "device.hpp"
#include "kernels.hpp"

namespace cpattn {

template <int D, int B>
__device__ __forceinline__ void append_span(const AppendItem& it, int h,
                                            const uint16_t* __restrict__ k_new,
                                            const uint16_t* __restrict__ v_new,
                                            uint16_t* __restrict__ k_cache,
                                            uint16_t* __restrict__ v_cache,
                                            const int32_t* __restrict__ bt, int hkv, int mbr) {
  const int req = it.req_slot0 >> 8;
  const int slot0 = it.req_slot0 & 0xff;
  const int64_t blk = bt[(int64_t)req * mbr + it.block];
  const int tid = threadIdx.x;
  constexpr int kChunks = D / 8;           // 16-byte chunks per K row
  constexpr int kPer = (B * kChunks + 255) / 256;
  // K: span rows of this head, 16-byte chunks; all loads before any store.
  // Loads are unconditional (rows past the span re-read its last row and are
  // not stored), which keeps the staging array in registers.
  u32x4_t kv[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int x = i * 256 + tid;
    const int j = min(x / kChunks, it.n_tok - 1);
    kv[i] = *reinterpret_cast<const u32x4_t*>(k_new + ((int64_t)(it.tok0 + j) * hkv + h) * D +
                                              (x % kChunks) * 8);
  }
  // V: thread (slot tile ts, feature group fg) loads the 16-byte pieces of
  // features [8 fg, 8 fg + 8) of the tokens in slots [8 ts, 8 ts + 8), turns
  // the 8x8 tile around in registers and writes one 8-slot run per feature:
  // a 16-byte store when the span covers the whole tile.
  constexpr int NTS = B / 8, NFG = D / 8;
  static_assert(NTS * NFG <= 256, "one V tile per thread");
  const int ts = tid / NFG;
  const int fg = tid % NFG;
  const int s_lo = max(8 * ts, slot0);
  const int s_hi = min(8 * ts + 8, slot0 + it.n_tok);
  const bool vwork = tid < NTS * NFG && s_lo < s_hi;
  u32x4_t w[8];  // w[e]: token in slot 8 ts + e, features 8 fg .. 8 fg + 7
  if (vwork) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {  // slots outside the span re-read one inside it
      const int slot = min(max(8 * ts + e, s_lo), s_hi - 1);
      w[e] = *reinterpret_cast<const u32x4_t*>(
          v_new + ((int64_t)(it.tok0 + slot - slot0) * hkv + h) * D + fg * 8);
    }
  }
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int x = i * 256 + tid;
    const int j = x / kChunks;
    if (j < it.n_tok)
      *reinterpret_cast<u32x4_t*>(k_cache + ((blk * hkv + h) * B + slot0 + j) * D +
                                  (x % kChunks) * 8) = kv[i];
  }
  if (vwork) {
    uint16_t* dst = v_cache + ((blk * hkv + h) * D + fg * 8) * B + 8 * ts;
    const bool whole = s_lo == 8 * ts && s_hi == 8 * ts + 8;
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      // feature 8 fg + f of the 8 slots
      uint32_t v16[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v16[e] = (w[e][f / 2] >> (16 * (f % 2))) & 0xffffu;
      if (whole) {
        u32x4_t o;
        o[0] = v16[0] | (v16[1] << 16);
        o[1] = v16[2] | (v16[3] << 16);
        o[2] = v16[4] | (v16[5] << 16);
        o[3] = v16[6] | (v16[7] << 16);
        *reinterpret_cast<u32x4_t*>(dst + f * B) = o;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (8 * ts + e >= s_lo && 8 * ts + e < s_hi) dst[f * B + e] = (uint16_t)v16[e];
      }
    }
  }
}

template <int D, int B>
__global__ __launch_bounds__(256) void kv_append_kernel(const AppendItem* __restrict__ items,
                                                        const uint16_t* __restrict__ k_new,
                                                        const uint16_t* __restrict__ v_new,
                                                        uint16_t* __restrict__ k_cache,
                                                        uint16_t* __restrict__ v_cache,
                                                        const int32_t* __restrict__ bt, int hkv,
                                                        int mbr) {
  append_span<D, B>(items[blockIdx.x], blockIdx.y, k_new, v_new, k_cache, v_cache, bt, hkv, mbr);
}

template <int D, int B>
__global__ __launch_bounds__(256) void kv_append_inline_kernel(const AppendInline inl,
                                                               const uint16_t* __restrict__ k_new,
                                                               const uint16_t* __restrict__ v_new,
                                                               uint16_t* __restrict__ k_cache,
                                                               uint16_t* __restrict__ v_cache,
                                                               const int32_t* __restrict__ bt,
                                                               int hkv, int mbr) {
  append_span<D, B>(inl.items[blockIdx.x], blockIdx.y, k_new, v_new, k_cache, v_cache, bt, hkv,
                    mbr);
}

// The append of a step together with the copy of its attention plan, one
// launch: workgroups [0, n_copy) copy the staged plan (host round trips),
// the rest append (item (b - n_copy) / hkv, kv head (b - n_copy) % hkv), so
// the plan's trip over PCIe overlaps the append instead of following it.
template <int D, int B>
__global__ __launch_bounds__(256) void kv_append_copy_kernel(
    const AppendInline inl, const uint16_t* __restrict__ k_new,
    const uint16_t* __restrict__ v_new, uint16_t* __restrict__ k_cache,
    uint16_t* __restrict__ v_cache, const int32_t* __restrict__ bt, int hkv, int mbr,
    PlanCopyArgs cp) {
  const int b = blockIdx.x;
  if (b < cp.n_blocks) {
    plan_copy_body<256>(cp.src, cp.dst, cp.n16, cp.done, cp.seq, b, cp.n_blocks, threadIdx.x);
    return;
  }
  const int a = b - cp.n_blocks;
  append_span<D, B>(inl.items[a / hkv], a % hkv, k_new, v_new, k_cache, v_cache, bt, hkv, mbr);
}

template <int D, int B>
static hipError_t launch_append_t(const AppendArgs& a, const AppendInline* inl, hipStream_t s) {
  if (inl) {
    if (a.n_items > kAppendInlineItems) return hipErrorInvalidValue;
    hipLaunchKernelGGL((kv_append_inline_kernel<D, B>), dim3(a.n_items, a.hkv), dim3(256), 0, s,
                       *inl, a.k_new, a.v_new, a.k_cache, a.v_cache, a.bt, a.hkv, a.mbr);
  } else {
    hipLaunchKernelGGL((kv_append_kernel<D, B>), dim3(a.n_items, a.hkv), dim3(256), 0, s, a.items,
                       a.k_new, a.v_new, a.k_cache, a.v_cache, a.bt, a.hkv, a.mbr);
  }
  return hipGetLastError();
}

template <int D, int B>
static hipError_t launch_append_copy_t(const AppendArgs& a, const AppendInline& inl,
                                       const PlanCopyArgs& cp, hipStream_t s) {
  if (a.n_items > kAppendInlineItems) return hipErrorInvalidValue;
  hipLaunchKernelGGL((kv_append_copy_kernel<D, B>), dim3(cp.n_blocks + a.n_items * a.hkv),
                     dim3(256), 0, s, inl, a.k_new, a.v_new, a.k_cache, a.v_cache, a.bt, a.hkv,
                     a.mbr, cp);
  return hipGetLastError();
}

hipError_t launch_append_copy(int D, int B, const AppendArgs& a, const AppendInline& inl,
                              const PlanCopyArgs& cp, hipStream_t s) {
  if (D == 128 && B == 16) return launch_append_copy_t<128, 16>(a, inl, cp, s);
  if (D == 128 && B == 32) return launch_append_copy_t<128, 32>(a, inl, cp, s);
  if (D == 64 && B == 16) return launch_append_copy_t<64, 16>(a, inl, cp, s);
  if (D == 64 && B == 32) return launch_append_copy_t<64, 32>(a, inl, cp, s);
  return hipErrorInvalidValue;
}

hipError_t launch_append(int D, int B, const AppendArgs& a, const AppendInline* inl,
                         hipStream_t s) {
  if (D == 128 && B == 16) return launch_append_t<128, 16>(a, inl, s);
  if (D == 128 && B == 32) return launch_append_t<128, 32>(a, inl, s);
  if (D == 64 && B == 16) return launch_append_t<64, 16>(a, inl, s);
  if (D == 64 && B == 32) return launch_append_t<64, 32>(a, inl, s);
  return hipErrorInvalidValue;
}

}  // namespace cpattn
