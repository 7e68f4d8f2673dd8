/* gs_peaks.h -- C ABI of the rate-calibration kernels (libgs_peaks.so).
 *
 * These kernels are not part of the Gauss sum: they measure, on the GPU the
 * library runs on, the three rates that bound its kernels, so that a
 * kernel's achieved throughput can be reported against the measured rate as
 * well as the published one:
 *   - the dense fp16 matrix-core rate (independent chains of one MFMA shape),
 *   - the transcendental rate of v_exp_f32 (independent chains of exp2; the
 *     Gauss sum evaluates one exponential per (query, key) pair, Eq. 1),
 *   - the fp32 FMA rate of the vector ALU (unpacked, as the library builds it),
 *   - the streaming read bandwidth of device memory,
 *   - the read bandwidth of the local data share (ds_read_b128 on linear
 *     addresses; the main kernels read their MFMA operands from LDS).
 *
 * Every kernel runs `workgroups` workgroups of GS_PEAKS_THREADS threads and
 * writes one 32-bit value per thread to `out` (so the work cannot be removed
 * by the compiler); `out` is a device buffer of workgroups * GS_PEAKS_THREADS
 * elements owned by the caller.  Work per launch (the caller divides by the
 * launch's duration):
 *   mfma:  workgroups * 4 waves * iters * GS_PEAKS_MFMA_CHAINS * flop(shape),
 *          flop(0) = 32*32*16*2 (v_mfma_f32_32x32x16_f16),
 *          flop(1) = 16*16*32*2 (v_mfma_f32_16x16x32_f16)
 *   exp:   workgroups * GS_PEAKS_THREADS * iters * GS_PEAKS_CHAINS exp2
 *   fma:   workgroups * GS_PEAKS_THREADS * iters * GS_PEAKS_CHAINS fma (2 flop each)
 *   read:  `bytes` bytes of `in`, read once
 *   lds:   workgroups * GS_PEAKS_THREADS * iters * GS_PEAKS_LDS_READS * 16 bytes
 *          read from LDS (each workgroup first fills 32 KiB of LDS)
 * All calls are asynchronous on `stream`; arguments are checked before the
 * launch.  Return value: 0 on success, 1 for an invalid argument (NULL
 * pointer, non-positive size, `bytes` not a multiple of 16, `in` not 16-byte
 * aligned, `shape` not 0 or 1, more than 2^31 - 1 workgroups), 2 if the
 * launch failed (hipGetLastError).
 */
#ifndef GS_PEAKS_H
#define GS_PEAKS_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GS_PEAKS_THREADS 256
#define GS_PEAKS_MFMA_CHAINS 4
#define GS_PEAKS_CHAINS 8
#define GS_PEAKS_LDS_READS 4

int gs_peaks_mfma(float* out, int64_t workgroups, int32_t iters, int32_t shape, hipStream_t stream);
int gs_peaks_exp(float* out, int64_t workgroups, int32_t iters, hipStream_t stream);
int gs_peaks_fma(float* out, int64_t workgroups, int32_t iters, hipStream_t stream);
int gs_peaks_read(const void* in, int64_t bytes, uint32_t* out, int64_t workgroups, hipStream_t stream);
int gs_peaks_lds(uint32_t* out, int64_t workgroups, int32_t iters, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* GS_PEAKS_H */
