// gs_prep.h -- per-point and per-value preparation kernels (linear cost).
//
//  * points: padded RT-layout copy in the input dtype (operand of q.k), the
//    fp32 half squared norm -||x||^2/2 (from the exact input values, summed in
//    fp64), and optionally a KS-layout fp16 copy (operand of sum_n P_mn k_n).
//  * values: exact power-of-two scaling so the largest |value| lies in [1, 2),
//    then fp16 copies in RT layout (contraction over C) and / or KS layout
//    (contraction over keys).
//  * row bound: for every query, the largest exponent over a fixed strided
//    sample of keys, a lower bound of its row maximum used to pick between
//    the unshifted and the row-max-shifted evaluation of the kernel values.
#pragma once

#include "gs_common.h"

namespace gs {

__global__ void k_fill_u32(uint32_t* __restrict__ p, int n, uint32_t val) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = val;
}

__global__ void k_fill_f32(float* __restrict__ p, int64_t n, float val) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = val;
}

// dtype codes follow gs_dtype: 0 = fp32, 1 = fp16, 2 = bf16.
__device__ __forceinline__ float load_any(const void* p, int64_t i, int dtype) {
  if (dtype == 0) return static_cast<const float*>(p)[i];
  uint16_t b = static_cast<const uint16_t*>(p)[i];
  return dtype == 1 ? F16::to_float(b) : BF16::to_float(b);
}

// max |x| over count elements into *slot (float bits; |x| >= 0 so unsigned
// comparison of the bit patterns orders them; NaN compares largest).
__global__ void k_absmax(const void* __restrict__ x, int64_t count, int dtype,
                         uint32_t* __restrict__ slot) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  uint32_t mb = 0;
  for (; i < count; i += stride) {
    uint32_t b = __builtin_bit_cast(uint32_t, fabsf(load_any(x, i, dtype)));
    mb = b > mb ? b : mb;
  }
  for (int off = 32; off > 0; off >>= 1) {
    uint32_t o = (uint32_t)__shfl_xor((int)mb, off, kWave);
    mb = o > mb ? o : mb;
  }
  if ((threadIdx.x & (kWave - 1)) == 0 && mb != 0) atomicMax(slot, mb);
}

// Points: xs[RT] = x (padding rows / columns = 0), one thread per element.
__global__ void k_points_rt(const uint16_t* __restrict__ x, int64_t n, int D, int64_t n_pad, int W,
                            uint16_t* __restrict__ xs) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n_pad * W; t += stride) {
    int64_t r = t / W;
    int w = (int)(t - r * W);
    uint16_t b = (r < n && w < D) ? x[r * D + w] : (uint16_t)0;
    xs[rt_index(r, w, W)] = b;
  }
}

// nh[r] = -||x_r||^2 / 2 summed in fp64 from the exact input values, rounded
// once to fp32; padding rows get kPadBias so their kernel value is 0.
template <typename T>
__global__ void k_points_norm(const uint16_t* __restrict__ x, int64_t n, int D, int64_t n_pad,
                              float* __restrict__ nh) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < n_pad; r += stride) {
    if (r >= n) { nh[r] = kPadBias; continue; }
    double acc = 0.0;
    const uint16_t* row = x + r * D;
    for (int d = 0; d < D; ++d) {
      double v = (double)T::to_float(row[d]);
      acc += v * v;
    }
    nh[r] = (float)(-0.5 * acc);
  }
}

// Points, KS-layout fp16 copy scaled by 2^e (e from *slot when slot != NULL,
// needed for bf16 inputs whose range exceeds fp16).  One thread per element,
// keys fastest so that the writes of a wave stay within a few 64-byte lines.
template <typename T>
__global__ void k_points_ks(const uint16_t* __restrict__ x, int64_t n, int D, int64_t n_pad, int R,
                            const uint32_t* __restrict__ slot, uint16_t* __restrict__ xt) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float s = slot ? ldexpf(1.0f, scale_exponent(*slot)) : 1.0f;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n_pad * R; t += stride) {
    int64_t blk = t / (32 * (int64_t)R);
    int rem = (int)(t - blk * 32 * (int64_t)R);
    int w = rem >> 5;
    int64_t r = blk * 32 + (rem & 31);
    float v = (r < n && w < D) ? T::to_float(x[r * D + w]) * s : 0.0f;
    _Float16 h = (_Float16)v;
    xt[ks_index(r, w, R)] = __builtin_bit_cast(uint16_t, h);
  }
}

// Values (fp32 / fp16 / bf16) scaled by 2^e(*slot) into fp16, RT layout
// (W = C padded to 32) and / or KS layout (R = C padded to 16).
__global__ void k_values_rt(const void* __restrict__ v, int dtype, int64_t n, int C, int64_t n_pad,
                            int W, const uint32_t* __restrict__ slot, uint16_t* __restrict__ vs) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float s = ldexpf(1.0f, scale_exponent(*slot));
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n_pad * W; t += stride) {
    int64_t r = t / W;
    int w = (int)(t - r * W);
    float val = (r < n && w < C) ? load_any(v, r * C + w, dtype) * s : 0.0f;
    _Float16 h = (_Float16)val;
    vs[rt_index(r, w, W)] = __builtin_bit_cast(uint16_t, h);
  }
}

__global__ void k_values_ks(const void* __restrict__ v, int dtype, int64_t n, int C, int64_t n_pad,
                            int R, const uint32_t* __restrict__ slot, uint16_t* __restrict__ vt) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float s = ldexpf(1.0f, scale_exponent(*slot));
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n_pad * R; t += stride) {
    int64_t blk = t / (32 * (int64_t)R);
    int rem = (int)(t - blk * 32 * (int64_t)R);
    int w = rem >> 5;
    int64_t r = blk * 32 + (rem & 31);
    float val = (r < n && w < C) ? load_any(v, r * C + w, dtype) * s : 0.0f;
    _Float16 h = (_Float16)val;
    vt[ks_index(r, w, R)] = __builtin_bit_cast(uint16_t, h);
  }
}

// Row bound: L[m] = max over a strided sample of keys of the log2 kernel value
// tau' * (q_m.k_n - ||q_m||^2/2 - ||k_n||^2/2), from the RT copies.  Rows past
// M get 0 (they never force the shifted evaluation).
template <typename T>
__global__ void k_row_bound(const uint16_t* __restrict__ qs, const float* __restrict__ nhq, int64_t M,
                            int64_t m_pad, const uint16_t* __restrict__ ks,
                            const float* __restrict__ nhk, int64_t N, int D, int W, float tau2,
                            int samples, float* __restrict__ L) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; m < m_pad; m += stride) {
    if (m >= M || N == 0) { L[m] = 0.0f; continue; }
    float best = -__builtin_inff();
    for (int j = 0; j < samples; ++j) {
      int64_t n = ((int64_t)j * N) / samples;
      float dot = 0.0f;
      for (int d = 0; d < D; ++d)
        dot = fmaf(T::to_float(qs[rt_index(m, d, W)]), T::to_float(ks[rt_index(n, d, W)]), dot);
      float x = tau2 * (dot + nhq[m] + nhk[n]);
      best = fmaxf(best, x);
    }
    L[m] = best;
  }
}

// out[m, w] = sum_s part[s, m, w] in split order (deterministic).
__global__ void k_combine(const float* __restrict__ part, int splits, int64_t count,
                          float* __restrict__ out) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < count; i += stride) {
    float acc = 0.0f;
    for (int s = 0; s < splits; ++s) acc += part[(int64_t)s * count + i];
    out[i] = acc;
  }
}

}  // namespace gs
