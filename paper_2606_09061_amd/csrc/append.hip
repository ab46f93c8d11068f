// Paged KV append: scatters the batch's new K/V rows into their cache slots.
//
// One workgroup per (request, logical block) span of new tokens.  K rows are
// token-major inside a block, so each 16-byte chunk of a new K row is one
// aligned vector copy.  V is feature-major inside a block ([D][B]), so each
// new token contributes one 2-byte element per feature; a workgroup writes
// the span's slots of one feature row next to each other.
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
  const int req = it.req_slot0 >> 8;
  const int slot0 = it.req_slot0 & 0xff;
  const int64_t blk = bt[(int64_t)req * mbr + it.block];
  constexpr int kChunks = D / 8;  // 16-byte chunks per K row
  const int n_k = it.n_tok * hkv * kChunks;
  for (int x = threadIdx.x; x < n_k; x += 256) {
    const int c = x % kChunks;
    const int rh = x / kChunks;
    const int h = rh % hkv;
    const int j = rh / hkv;
    const uint4* src =
        reinterpret_cast<const uint4*>(k_new + ((int64_t)(it.tok0 + j) * hkv + h) * D + c * 8);
    uint4* dst = reinterpret_cast<uint4*>(k_cache + ((blk * hkv + h) * B + slot0 + j) * D + c * 8);
    *dst = *src;
  }
  const int n_v = it.n_tok * hkv * D;
  for (int x = threadIdx.x; x < n_v; x += 256) {
    const int j = x % it.n_tok;
    const int hd = x / it.n_tok;
    const int d = hd % D;
    const int h = hd / D;
    v_cache[((blk * hkv + h) * D + d) * B + slot0 + j] =
        v_new[((int64_t)(it.tok0 + j) * hkv + h) * D + d];
  }
}

template <int D, int B>
static hipError_t launch_append_t(const AppendArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((kv_append_kernel<D, B>), dim3(a.n_items), dim3(256), 0, s, a.items, a.k_new,
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
