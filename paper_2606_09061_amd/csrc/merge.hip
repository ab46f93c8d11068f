// Merge of split key ranges.  Each split of a row left its normalised output
// O_s and L_s = log2(sum of its unnormalised weights) in base-2 units; the
// full-range output is
//     O = sum_s 2^(L_s - M) O_s / sum_s 2^(L_s - M),   M = max_s L_s,
// which is exact for any partition of the keys (softmax is shift invariant).
#include "device.hpp"
#include "kernels.hpp"

namespace cpattn {

template <int D>
__global__ __launch_bounds__(256) void merge_kernel(const MergeGroup* __restrict__ groups,
                                                    const float* __restrict__ part_o,
                                                    const float* __restrict__ part_lse,
                                                    uint16_t* __restrict__ out, int hq, int G) {
  const MergeGroup mg = groups[blockIdx.x];
  constexpr int DQ = D / 4;  // threads per row, 4 features each
  const int rl = threadIdx.x / DQ;
  if (rl >= mg.n_rows) return;
  const int dq = threadIdx.x % DQ;
  const int rows = mg.n_tok * G;
  const int kvh = blockIdx.y;
  const int r = mg.row0 + rl;
  const int base = mg.part0 + kvh * mg.n_split * rows + r;
  float M = -INFINITY;
#pragma unroll 4
  for (int s = 0; s < mg.n_split; ++s) M = fmaxf(M, part_lse[base + s * rows]);
  float wsum = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
  for (int s = 0; s < mg.n_split; ++s) {
    const int pr = base + s * rows;
    const float ls = part_lse[pr];
    const float w = ls == -INFINITY ? 0.f : exp2f(ls - M);
    const float4 o = *reinterpret_cast<const float4*>(part_o + (int64_t)pr * D + dq * 4);
    wsum += w;
    acc.x += w * o.x;
    acc.y += w * o.y;
    acc.z += w * o.z;
    acc.w += w * o.w;
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  const int tok = mg.tok0 + r / G;
  const int h = kvh * G + r % G;
  uint2 w2;
  w2.x = pack_bf16x2(acc.x * inv, acc.y * inv);
  w2.y = pack_bf16x2(acc.z * inv, acc.w * inv);
  *reinterpret_cast<uint2*>(out + ((int64_t)tok * hq + h) * D + dq * 4) = w2;
}

hipError_t launch_merge(int D, int G, const AttnArgs& a, hipStream_t s) {
  if (D == 128)
    hipLaunchKernelGGL(merge_kernel<128>, dim3(a.n_merge, a.hkv), dim3(256), 0, s, a.merge, a.part_o,
                       a.part_lse, a.out, a.hq, G);
  else if (D == 64)
    hipLaunchKernelGGL(merge_kernel<64>, dim3(a.n_merge, a.hkv), dim3(256), 0, s, a.merge, a.part_o,
                       a.part_lse, a.out, a.hq, G);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace cpattn
