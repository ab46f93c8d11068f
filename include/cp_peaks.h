/*
 * cp_peaks.h — C ABI of the microbenchmarks that measure the practical peaks
 * the attention kernels are compared with, on AMD Instinct MI355X (gfx950):
 * the matrix-core rate of a register-only bf16 MFMA loop and the HBM rate of
 * a streaming read.  The datasheet peaks (2.5 PFLOP/s dense bf16, 8 TB/s)
 * assume the nominal clock and ideal access; these kernels show what this
 * GPU sustains, and the device attributes that the datasheet figures rest on.
 *
 * All pointers are device pointers owned by the caller; nothing is
 * allocated.  Launches are asynchronous on `stream`; time them with events.
 * Functions return 0, or -1 for an invalid argument (nothing is launched),
 * or -5 when the HIP runtime reports an error.
 */
#ifndef CP_PEAKS_H
#define CP_PEAKS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Compute units, peak engine clock (kHz), memory clock (kHz) and memory bus
 * width (bits) of device `device`, from the HIP device attributes. */
int cpk_device_info(int32_t device, int32_t* compute_units, int32_t* clock_khz,
                    int32_t* mem_clock_khz, int32_t* mem_bus_bits);

/* Register-only loop of v_mfma_f32_32x32x16_bf16: every wave keeps four
 * 32x32 fp32 accumulators and issues 16 MFMAs per iteration for `iters`
 * iterations (32768 flop each), on operands read once from `operands`
 * (n16 16-byte elements, bf16 bits).  random_operands = 0 makes every wave
 * read element 0 (constant operands); otherwise each lane reads its own
 * elements (indices taken modulo n16).  out receives one float per thread
 * (blocks * threads) so that the work is kept.  threads in {64, 128, 256,
 * 512}, blocks >= 1, iters >= 1, n16 >= 8. */
int cpk_mfma_loop(const void* operands, int64_t n16, float* out, int32_t blocks, int32_t threads,
                  int32_t iters, int32_t random_operands, void* stream);

/* Streaming read of n16 16-byte elements of src with non-temporal loads,
 * grid-stride over `blocks` workgroups of 256 threads; out receives one word
 * per thread (blocks * 256) derived from what it read. */
int cpk_read_stream(const void* src, int64_t n16, uint32_t* out, int32_t blocks, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CP_PEAKS_H */
