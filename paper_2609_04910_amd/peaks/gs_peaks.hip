// Rate-calibration kernels for gfx950: matrix-core, transcendental, vector
// FMA and streaming-read rates measured on the device itself.  They share
// nothing with the Gauss-sum kernels; the C ABI and the work each launch does
// are documented in gs_peaks.h.
#include <hip/hip_runtime.h>

#include "gs_peaks.h"

namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float4v __attribute__((ext_vector_type(4)));
typedef float float16v __attribute__((ext_vector_type(16)));

constexpr int kThreads = GS_PEAKS_THREADS;

// shape 0: v_mfma_f32_32x32x16_f16, shape 1: v_mfma_f32_16x16x32_f16; four
// independent accumulator chains per wave keep the matrix pipe full.
template <int kShape>
__global__ __launch_bounds__(kThreads) void k_mfma(float* out, int iters) {
  half8 a, b;
  for (int t = 0; t < 8; ++t) {
    a[t] = (_Float16)(0.001f * (threadIdx.x + t));
    b[t] = (_Float16)(0.002f * (threadIdx.x - t));
  }
  float r;
  if constexpr (kShape == 0) {
    float16v c0 = {}, c1 = {}, c2 = {}, c3 = {};
    c1[0] = 1.f, c2[0] = 2.f, c3[0] = 3.f;  // distinct chains: none can be merged
    for (int i = 0; i < iters; ++i) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c3, 0, 0, 0);
    }
    r = c0[0] + c1[5] + c2[10] + c3[15];
  } else {
    float4v c0 = {}, c1 = {}, c2 = {}, c3 = {};
    c1[0] = 1.f, c2[0] = 2.f, c3[0] = 3.f;
    for (int i = 0; i < iters; ++i) {
      c0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c3, 0, 0, 0);
    }
    r = c0[0] + c1[1] + c2[2] + c3[3];
  }
  out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = r;
}

// Eight independent chains x <- 2^(-x) per lane: values stay in [1/2, 1], so
// no input ever takes a special path of the instruction.
__global__ __launch_bounds__(kThreads) void k_exp(float* out, int iters) {
  float x[GS_PEAKS_CHAINS];
  for (int c = 0; c < GS_PEAKS_CHAINS; ++c) x[c] = 0.5f + 1e-3f * c + 1e-6f * threadIdx.x;
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < GS_PEAKS_CHAINS; ++c) x[c] = __builtin_amdgcn_exp2f(-x[c]);
  }
  float r = 0.f;
  for (int c = 0; c < GS_PEAKS_CHAINS; ++c) r += x[c];
  out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = r;
}

// Eight independent fp32 FMA chains per lane (contracting towards 1).
__global__ __launch_bounds__(kThreads) void k_fma(float* out, int iters) {
  float x[GS_PEAKS_CHAINS];
  for (int c = 0; c < GS_PEAKS_CHAINS; ++c) x[c] = 0.25f + 1e-3f * c + 1e-6f * threadIdx.x;
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < GS_PEAKS_CHAINS; ++c) x[c] = fmaf(x[c], 0.999f, 0.001f);
  }
  float r = 0.f;
  for (int c = 0; c < GS_PEAKS_CHAINS; ++c) r += x[c];
  out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = r;
}

// Grid-stride read of n 16-byte words, four loads in flight per lane, folded
// into one word per lane by xor.
__global__ __launch_bounds__(kThreads) void k_read(const uint4* in, int64_t n, uint32_t* out) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  uint32_t acc = 0;
  for (; i + 3 * stride < n; i += 4 * stride) {
    const uint4 a = in[i], b = in[i + stride], c = in[i + 2 * stride], d = in[i + 3 * stride];
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w;
    acc ^= c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  for (; i < n; i += stride) {
    const uint4 a = in[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc;
}

// LDS read bandwidth: every wave reads four independent 1-KiB rows per
// iteration (lane l takes the 16 bytes at 16 l of each row, ds_read_b128 on
// linear addresses), walking over the workgroup's kLdsBytes of LDS, folded
// into one word per lane by xor.
constexpr int kLdsBytes = 32768;
__global__ __launch_bounds__(kThreads) void k_lds(uint32_t* out, int iters) {
  __shared__ uint4 buf[kLdsBytes / 16];
  for (int i = threadIdx.x; i < kLdsBytes / 16; i += kThreads)
    buf[i] = uint4{(uint32_t)i, (uint32_t)(3 * i), (uint32_t)(5 * i), (uint32_t)(7 * i)};
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int kRows = kLdsBytes / 1024;  // 1-KiB rows
  uint32_t acc = 0;
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int u = 0; u < GS_PEAKS_LDS_READS; ++u) {
      const int row = (i * GS_PEAKS_LDS_READS + u + 8 * wave) & (kRows - 1);
      const uint4 a = buf[row * 64 + lane];
      acc ^= a.x ^ a.y ^ a.z ^ a.w;
    }
  }
  out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc;
}

bool bad_grid(int64_t workgroups) { return workgroups <= 0 || workgroups > 0x7fffffff; }

int launched() { return hipGetLastError() == hipSuccess ? 0 : 2; }

}  // namespace

extern "C" int gs_peaks_mfma(float* out, int64_t workgroups, int32_t iters, int32_t shape,
                             hipStream_t stream) {
  if (!out || bad_grid(workgroups) || iters <= 0 || (shape != 0 && shape != 1)) return 1;
  (void)hipGetLastError();
  if (shape == 0)
    k_mfma<0><<<dim3((unsigned)workgroups), dim3(kThreads), 0, stream>>>(out, iters);
  else
    k_mfma<1><<<dim3((unsigned)workgroups), dim3(kThreads), 0, stream>>>(out, iters);
  return launched();
}

extern "C" int gs_peaks_exp(float* out, int64_t workgroups, int32_t iters, hipStream_t stream) {
  if (!out || bad_grid(workgroups) || iters <= 0) return 1;
  (void)hipGetLastError();
  k_exp<<<dim3((unsigned)workgroups), dim3(kThreads), 0, stream>>>(out, iters);
  return launched();
}

extern "C" int gs_peaks_fma(float* out, int64_t workgroups, int32_t iters, hipStream_t stream) {
  if (!out || bad_grid(workgroups) || iters <= 0) return 1;
  (void)hipGetLastError();
  k_fma<<<dim3((unsigned)workgroups), dim3(kThreads), 0, stream>>>(out, iters);
  return launched();
}

extern "C" int gs_peaks_read(const void* in, int64_t bytes, uint32_t* out, int64_t workgroups,
                             hipStream_t stream) {
  if (!in || !out || bytes <= 0 || bytes % 16 != 0 || (reinterpret_cast<uintptr_t>(in) & 15) ||
      bad_grid(workgroups))
    return 1;
  (void)hipGetLastError();
  k_read<<<dim3((unsigned)workgroups), dim3(kThreads), 0, stream>>>(static_cast<const uint4*>(in),
                                                                    bytes / 16, out);
  return launched();
}

extern "C" int gs_peaks_lds(uint32_t* out, int64_t workgroups, int32_t iters, hipStream_t stream) {
  if (!out || bad_grid(workgroups) || iters <= 0) return 1;
  (void)hipGetLastError();
  k_lds<<<dim3((unsigned)workgroups), dim3(kThreads), 0, stream>>>(out, iters);
  return launched();
}
