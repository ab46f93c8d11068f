// Copy of a staged plan from pinned host memory into the workspace, shared by
// the plan copy kernel and the combined append + copy kernel.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cpattn {

// Workgroup `blk` of `nblk` (NT threads, thread `tid`) copies pieces of
// PER * NT 16-byte words of src[0, n16) to dst, every load of a piece issued
// before its first store; when all its reads have returned it writes seq to
// done[blk] (a word in the staging slot itself, which the host polls before
// reusing the slot).
template <int NT, int PER = 8>
__device__ __forceinline__ void plan_copy_body(const uint4* __restrict__ src,
                                               uint4* __restrict__ dst, int n16,
                                               uint32_t* __restrict__ done, uint32_t seq, int blk,
                                               int nblk, int tid) {
  for (int base = blk * PER * NT + tid; base < n16; base += nblk * PER * NT) {
    uint4 v[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i = base + k * NT;
      v[k] = i < n16 ? src[i] : make_uint4(0, 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);  // every load issued before the first store
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i = base + k * NT;
      if (i < n16) dst[i] = v[k];
    }
  }
  __syncthreads();  // every read of this workgroup has returned
  if (tid == 0)
    __hip_atomic_store(done + blk, seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

}  // namespace cpattn
