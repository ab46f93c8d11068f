// Microbenchmarks of the practical matrix-core and HBM peaks (include/cp_peaks.h).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cp_peaks.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4_t ld_nt(const uint4* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
}

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& v) {
  return __builtin_bit_cast(bf16x8_t, v);
}

__global__ void mfma_loop_kernel(const uint4* __restrict__ src, int64_t n16, float* __restrict__ out,
                                 int iters, int random_operands) {
  const int64_t gtid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint4 a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t ia = random_operands ? (gtid * 8 + i) % n16 : 0;
    const int64_t ib = random_operands ? (gtid * 8 + 4 + i) % n16 : 0;
    a[i] = src[ia];
    b[i] = src[ib];
  }
  f32x16_t acc[4];
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[m][r] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int m = 0; m < 4; ++m)
        acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a[(m + k) & 3]),
                                                         as_bf16x8(b[k]), acc[m], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[m][r];
  out[gtid] = s;
}

__global__ __launch_bounds__(256) void read_stream_kernel(const uint4* __restrict__ src, int64_t n16,
                                                          uint32_t* __restrict__ out) {
  const int64_t gtid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * 256;
  uint32_t x = 0;
  int64_t i = gtid;
  // four independent loads in flight per thread
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u32x4_t v0 = ld_nt(src + i);
    const u32x4_t v1 = ld_nt(src + i + stride);
    const u32x4_t v2 = ld_nt(src + i + 2 * stride);
    const u32x4_t v3 = ld_nt(src + i + 3 * stride);
    x ^= v0[0] ^ v1[1] ^ v2[2] ^ v3[3];
  }
  for (; i < n16; i += stride) {
    const u32x4_t v = ld_nt(src + i);
    x ^= v[0] ^ v[3];
  }
  out[gtid] = x;
}

int launched() { return hipGetLastError() == hipSuccess ? 0 : -5; }

}  // namespace

extern "C" {

int cpk_device_info(int32_t device, int32_t* compute_units, int32_t* clock_khz,
                    int32_t* mem_clock_khz, int32_t* mem_bus_bits) {
  if (!compute_units || !clock_khz || !mem_clock_khz || !mem_bus_bits) return -1;
  int v[4];
  const hipDeviceAttribute_t attr[4] = {hipDeviceAttributeMultiprocessorCount,
                                        hipDeviceAttributeClockRate,
                                        hipDeviceAttributeMemoryClockRate,
                                        hipDeviceAttributeMemoryBusWidth};
  for (int i = 0; i < 4; ++i)
    if (hipDeviceGetAttribute(&v[i], attr[i], device) != hipSuccess) return -5;
  *compute_units = v[0];
  *clock_khz = v[1];
  *mem_clock_khz = v[2];
  *mem_bus_bits = v[3];
  return 0;
}

int cpk_mfma_loop(const void* operands, int64_t n16, float* out, int32_t blocks, int32_t threads,
                  int32_t iters, int32_t random_operands, void* stream) {
  if (!operands || !out || n16 < 8 || blocks < 1 || iters < 1 ||
      (threads != 64 && threads != 128 && threads != 256 && threads != 512))
    return -1;
  (void)hipGetLastError();
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(blocks), dim3(threads), 0, (hipStream_t)stream,
                     (const uint4*)operands, n16, out, iters, random_operands);
  return launched();
}

int cpk_read_stream(const void* src, int64_t n16, uint32_t* out, int32_t blocks, void* stream) {
  if (!src || !out || n16 < 1 || blocks < 1) return -1;
  (void)hipGetLastError();
  hipLaunchKernelGGL(read_stream_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream,
                     (const uint4*)src, n16, out);
  return launched();
}

}  // extern "C"
