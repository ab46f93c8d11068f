// Split-K decode attention (one query token per row, G q heads per kv head):
// one workgroup of 4 waves per (row, range of whole blocks) and kv head
// blockIdx.y.  The body is decode_unit (decode_body.hpp), which the prefill
// kernel also runs for the decode blocks it carries when a step's decode
// rows are overlapped with its prefill tiles.
#include "decode_body.hpp"
#include "kernels.hpp"

namespace cpattn {

template <int D, int B, int G>
__global__ __launch_bounds__(256, G * D >= 512 ? 3 : 4) void decode_kernel(
    const DecodeItem* __restrict__ items, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ k_cache, const uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ bt, uint16_t* __restrict__ out, float* __restrict__ part_o,
    float* __restrict__ part_lse, int hq, int hkv, int mbr, float scale_log2) {
  using Lds = decode_impl::DecodeLds<D, G>;
  __shared__ __attribute__((aligned(16))) float red_o[Lds::O_BYTES / 4];
  __shared__ __attribute__((aligned(16))) uint8_t small[Lds::SMALL_BYTES];
  decode_unit<D, B, G>(items[blockIdx.x], blockIdx.y, true, threadIdx.x, q, k_cache, v_cache, bt,
                       out, part_o, part_lse, hq, hkv, mbr, scale_log2,
                       decode_impl::DecodeLdsPtrs{red_o, small});
}

template <int D, int B, int G>
static hipError_t launch_decode_t(const AttnArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((decode_kernel<D, B, G>), dim3(a.n_decode, a.hkv), dim3(256), 0, s, a.decode, a.q,
                     a.k_cache, a.v_cache, a.bt, a.out, a.part_o, a.part_lse, a.hq, a.hkv, a.mbr,
                     a.scale_log2);
  return hipGetLastError();
}

template <int D, int B>
static hipError_t launch_decode_g(int G, const AttnArgs& a, hipStream_t s) {
  switch (G) {
    case 1: return launch_decode_t<D, B, 1>(a, s);
    case 2: return launch_decode_t<D, B, 2>(a, s);
    case 4: return launch_decode_t<D, B, 4>(a, s);
    case 8: return launch_decode_t<D, B, 8>(a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_decode(int D, int B, int G, const AttnArgs& a, hipStream_t s) {
  if (D == 128 && B == 16) return launch_decode_g<128, 16>(G, a, s);
  if (D == 128 && B == 32) return launch_decode_g<128, 32>(G, a, s);
  if (D == 64 && B == 16) return launch_decode_g<64, 16>(G, a, s);
  if (D == 64 && B == 32) return launch_decode_g<64, 32>(G, a, s);
  return hipErrorInvalidValue;
}

}  // namespace cpattn
