// Paged KV append: scatters the batch's new K/V rows into their cache slots.
//
// One workgroup per (request, logical block) span of new tokens and kv head.
// K rows are token-major inside a block, so each 16-byte chunk of a new K row
// is one aligned vector copy.  V is feature-major inside a block ([D][B]):
// thread d gathers the span's values of feature d and writes them as one run
// of its feature row (one 16-byte store per 8 slots when the span fills the
// block).  Every load is issued before the first store.
#include "device.hpp"
#include "kernels.hpp"

namespace cpattn {

template <int D, int B>
__global__ __launch_bounds__(256) void kv_append_kernel(const AppendItem* __restrict__ items,
                                                        const uint16_t* __restrict__ k_new,
                                                        const uint16_t* __restrict__ v_new,
                                                        uint16_t* __restrict__ k_cache,
                                                        uint16_t* __restrict__ v_cache,
                                                        const int32_t* __restrict__ bt, int hkv,
                                                        int mbr) {
  const AppendItem it = items[blockIdx.x];
  const int h = blockIdx.y;
  const int req = it.req_slot0 >> 8;
  const int slot0 = it.req_slot0 & 0xff;
  const int64_t blk = bt[(int64_t)req * mbr + it.block];
  const int tid = threadIdx.x;
  constexpr int kChunks = D / 8;           // 16-byte chunks per K row
  constexpr int kPer = (B * kChunks + 255) / 256;
  // K: span rows of this head, 16-byte chunks; all loads before any store
  uint4 kv[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int x = i * 256 + tid;
    const int j = x / kChunks;
    if (j < it.n_tok)
      kv[i] = *reinterpret_cast<const uint4*>(k_new + ((int64_t)(it.tok0 + j) * hkv + h) * D +
                                              (x % kChunks) * 8);
  }
  // V: thread d gathers the span's values of feature d (coalesced over d)
  uint16_t vv[B];
  const bool vthread = tid < D;
  if (vthread) {
    const uint16_t* src = v_new + ((int64_t)it.tok0 * hkv + h) * D + tid;
#pragma unroll
    for (int j = 0; j < B; ++j)
      if (j < it.n_tok) vv[j] = src[(int64_t)j * hkv * D];
  }
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int x = i * 256 + tid;
    const int j = x / kChunks;
    if (j < it.n_tok)
      *reinterpret_cast<uint4*>(k_cache + ((blk * hkv + h) * B + slot0 + j) * D +
                                (x % kChunks) * 8) = kv[i];
  }
  if (vthread) {
    uint16_t* dst = v_cache + ((blk * hkv + h) * D + tid) * B;
    if (it.n_tok == B) {
#pragma unroll
      for (int j = 0; j < B / 8; ++j) {
        uint4 w;
        w.x = (uint32_t)vv[8 * j + 0] | ((uint32_t)vv[8 * j + 1] << 16);
        w.y = (uint32_t)vv[8 * j + 2] | ((uint32_t)vv[8 * j + 3] << 16);
        w.z = (uint32_t)vv[8 * j + 4] | ((uint32_t)vv[8 * j + 5] << 16);
        w.w = (uint32_t)vv[8 * j + 6] | ((uint32_t)vv[8 * j + 7] << 16);
        reinterpret_cast<uint4*>(dst)[j] = w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < B; ++j)
        if (j < it.n_tok) dst[slot0 + j] = vv[j];
    }
  }
}

template <int D, int B>
static hipError_t launch_append_t(const AppendArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((kv_append_kernel<D, B>), dim3(a.n_items, a.hkv), dim3(256), 0, s, a.items,
                     a.k_new,
                     a.v_new, a.k_cache, a.v_cache, a.bt, a.hkv, a.mbr);
  return hipGetLastError();
}

hipError_t launch_append(int D, int B, const AppendArgs& a, hipStream_t s) {
  if (D == 128 && B == 16) return launch_append_t<128, 16>(a, s);
  if (D == 128 && B == 32) return launch_append_t<128, 32>(a, s);
  if (D == 64 && B == 16) return launch_append_t<64, 16>(a, s);
  if (D == 64 && B == 32) return launch_append_t<64, 32>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace cpattn
