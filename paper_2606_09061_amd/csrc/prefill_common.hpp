// Shared pieces of the prefill kernels: LDS tile layout and lane helpers.
#pragma once

#include "device.hpp"

namespace cpattn {

namespace prefill_detail {

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

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

}  // namespace prefill_detail

using prefill_detail::BN;
using prefill_detail::sigma;
using prefill_detail::acc_key;
using prefill_detail::uniform;

template <int D, int B>
struct PrefillLayout {
  static constexpr int KCH = D / 8;          // 16-byte chunks per K row
  static constexpr int K_BYTES = BN * D * 2;
  static constexpr int V_BYTES = BN * D * 2;
  static constexpr int BUF = K_BYTES + V_BYTES;  // one step's K and V^T
  static constexpr int VSLOTS = B / 8;       // 16-byte slots per V^T row
  // K row `key`, chunk c -> byte offset
  __device__ static int k_off(int key, int c) {
    return key * D * 2 + ((c ^ (sigma(key & 15) & (KCH - 1))) << 4);
  }
  // V^T of step-block bi, feature row d, slot s (8 keys) -> byte offset
  __device__ static int v_off(int bi, int d, int s) {
    const int h = B == 16 ? (((d >> 2) ^ (d >> 3)) & 1) : ((d >> 2) & 3);
    return K_BYTES + bi * D * B * 2 + d * B * 2 + ((s ^ h) << 4);
  }
};

}  // namespace cpattn
