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

__global__ void k_fill_u32(uint32_t* __restrict__ p, int n, uint32_t val, Bz bz) {
  p = zoff(p, bz.ws);
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = val;
}

__global__ void k_fill_f32(float* __restrict__ p, int64_t n, float val) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = val;
}


// max |x| over count elements into *slot (float bits; |x| >= 0 so unsigned
// comparison of the bit patterns orders them; NaN compares largest).  Reduced
// within the workgroup first: one atomic per workgroup.
__global__ void k_absmax(const void* __restrict__ x, int64_t count, int dtype,
                         uint32_t* __restrict__ slot, Bz bz) {
  __shared__ uint32_t wmax[kWavesPerBlock];
  x = zoff(x, bz.in);
  slot = zoff(slot, bz.ws);
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  uint32_t mb = 0;
  auto take = [&](float f) {
    const uint32_t b = __builtin_bit_cast(uint32_t, fabsf(f));
    mb = b > mb ? b : mb;
  };
  if ((reinterpret_cast<uintptr_t>(x) & 15) == 0) {
    // 16-byte loads (4 fp32 or 8 fp16 / bf16 elements), two in flight per
    // thread; the tail of fewer than one vector's elements falls through
    const int per = dtype == 0 ? 4 : 8;
    const int64_t nv = count / per;
    const uint4* xv = static_cast<const uint4*>(x);
    auto vec = [&](const uint4 w) {
      const uint32_t u[4] = {w.x, w.y, w.z, w.w};
      if (dtype == 0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) take(__builtin_bit_cast(float, u[e]));
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint16_t lo = (uint16_t)(u[e] & 0xffffu), hi = (uint16_t)(u[e] >> 16);
          take(dtype == 1 ? F16::to_float(lo) : BF16::to_float(lo));
          take(dtype == 1 ? F16::to_float(hi) : BF16::to_float(hi));
        }
      }
    };
    int64_t j = i;
    for (; j + stride < nv; j += 2 * stride) {
      const uint4 a = xv[j], b = xv[j + stride];
      vec(a);
      vec(b);
    }
    for (; j < nv; j += stride) vec(xv[j]);
    i = nv * per + i;  // scalar tail
  }
  // four independent loads in flight per thread
  for (; i + 3 * stride < count; i += 4 * stride) {
    uint32_t b[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) b[u] = __builtin_bit_cast(uint32_t, fabsf(load_any(x, i + u * stride, dtype)));
#pragma unroll
    for (int u = 0; u < 4; ++u) mb = b[u] > mb ? b[u] : mb;
  }
  for (; i < count; i += stride) {
    uint32_t b = __builtin_bit_cast(uint32_t, fabsf(load_any(x, i, dtype)));
    mb = b > mb ? b : mb;
  }
  for (int off = 32; off > 0; off >>= 1) {
    uint32_t o = (uint32_t)__shfl_xor((int)mb, off, kWave);
    mb = o > mb ? o : mb;
  }
  if ((threadIdx.x & (kWave - 1)) == 0) wmax[threadIdx.x / kWave] = mb;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kWavesPerBlock; ++w) mb = wmax[w] > mb ? wmax[w] : mb;
    if (mb != 0) atomicMax(slot, mb);
  }
}

// Points, RT copy and half norms in one pass.  Thread (r, c) moves columns
// 8c .. 8c+7 of row r (one 16-byte store into the RT copy: those eight
// columns are contiguous there) and sums their squares in fp64; the W/8
// threads of a row are consecutive lanes, reduced with shuffles, so
// nh[r] = -||x_r||^2 / 2 is rounded once to fp32.  Padding rows / columns are
// zero, padding rows get kPadBias.  n_pad * W/8 is a multiple of the wave
// size, so every lane of a wave runs the same iterations of the grid-stride
// loop and the shuffles see whole waves.  vec: rows start on 16-byte
// boundaries and D is a multiple of 8, so the eight columns are one 16-byte
// load.  rt_norm_item is one thread's share: item t (row t / cpr, columns
// 8 (t % cpr) .. +7); it returns the row's half norm (the same value in
// every lane of the row).
template <typename T>
__device__ __forceinline__ float rt_norm_item(const uint16_t* __restrict__ x, int64_t n, int D, int W,
                                              uint16_t* __restrict__ xs, float* __restrict__ nh, int vec,
                                              int64_t t) {
  const int cpr = W >> 3;  // threads per row (4, 8, 16 or 32)
  {
    const int64_t r = t / cpr;
    const int c = (int)(t - r * cpr);
    uint16_t h[8];
    if (vec) {
      uint4 u = make_uint4(0, 0, 0, 0);
      if (r < n && 8 * c < D) u = *reinterpret_cast<const uint4*>(x + r * D + 8 * c);
      const uint32_t wd[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) h[e] = (uint16_t)(wd[e >> 1] >> (16 * (e & 1)));
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int w = 8 * c + e;
        h[e] = (r < n && w < D) ? x[r * D + w] : (uint16_t)0;
      }
    }
    double acc = 0.0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const double v = (double)T::to_float(h[e]);
      acc += v * v;
    }
    for (int off = cpr >> 1; off > 0; off >>= 1) acc += __shfl_xor(acc, off, kWave);
    uint4 pk;
    pk.x = h[0] | ((uint32_t)h[1] << 16);
    pk.y = h[2] | ((uint32_t)h[3] << 16);
    pk.z = h[4] | ((uint32_t)h[5] << 16);
    pk.w = h[6] | ((uint32_t)h[7] << 16);
    *reinterpret_cast<uint4*>(xs + rt_index(r, 8 * c, W)) = pk;
    const float half = r < n ? (float)(-0.5 * acc) : kPadBias;
    if (c == 0) nh[r] = half;
    return half;
  }
}

template <typename T>
__global__ void k_points_rt_norm(const uint16_t* __restrict__ x, int64_t n, int D, int64_t n_pad,
                                 int W, uint16_t* __restrict__ xs, float* __restrict__ nh, int vec,
                                 Bz bz) {
  x = zoff(x, bz.in);
  xs = zoff(xs, bz.ws);
  nh = zoff(nh, bz.ws);
  const int cpr = W >> 3;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n_pad * cpr; t += stride)
    (void)rt_norm_item<T>(x, n, D, W, xs, nh, vec, t);
}

// Points, KS-layout fp16 copy scaled by 2^e (e = point_scale_exponent(*slot)
// when slot != NULL, for bf16 inputs whose range exceeds fp16) and, when sgn != NULL,
// multiplied by the sign of the single-channel value sgn[r] (exact).  Thread
// (32-key block, row w, quarter a) writes the eight key slots 8a .. 8a+7 of
// row w (one 16-byte store); consecutive threads write consecutive 16 bytes.
template <typename T>
__global__ void k_points_ks(const uint16_t* __restrict__ x, int64_t n, int D, int64_t n_pad, int R,
                            const uint32_t* __restrict__ slot, const void* __restrict__ sgn,
                            int sgn_dtype, uint16_t* __restrict__ xt, Bz bz) {
  x = zoff(x, bz.in);
  slot = zoff(slot, bz.ws);
  sgn = zoff(sgn, bz.in2);
  xt = zoff(xt, bz.ws);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float s = slot ? ldexpf(1.0f, point_scale_exponent(*slot)) : 1.0f;
  const int64_t total = (n_pad >> 5) * R * 4;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
    const int a = (int)(t & 3);
    const int64_t rest = t >> 2;
    const int64_t blk = rest / R;
    const int w = (int)(rest - blk * R);
    uint16_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int z = 8 * a + e;
      const int64_t r = blk * 32 + 16 * ((z & 7) >> 2) + 4 * (z >> 3) + (z & 3);
      float v = (r < n && w < D) ? T::to_float(x[r * D + w]) * s : 0.0f;
      if (sgn && r < n && load_any(sgn, r, sgn_dtype) < 0.0f) v = -v;
      h[e] = __builtin_bit_cast(uint16_t, (_Float16)v);
    }
    uint4 pk;
    pk.x = h[0] | ((uint32_t)h[1] << 16);
    pk.y = h[2] | ((uint32_t)h[3] << 16);
    pk.z = h[4] | ((uint32_t)h[5] << 16);
    pk.w = h[6] | ((uint32_t)h[7] << 16);
    *reinterpret_cast<uint4*>(xt + ((blk * R + w) * 32 + 8 * a)) = pk;
  }
}

// Values (fp32 / fp16 / bf16) scaled by 2^e(*slot) into fp16, RT layout
// (W = C padded to 32) and / or KS layout (R = C padded to 16).
__global__ void k_values_rt(const void* __restrict__ v, int dtype, int64_t n, int C, int64_t n_pad,
                            int W, const uint32_t* __restrict__ slot, uint16_t* __restrict__ vs,
                            Bz bz) {
  v = zoff(v, bz.in);
  slot = zoff(slot, bz.ws);
  vs = zoff(vs, bz.ws);
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

// With sign_only (single-channel values, whose magnitudes enter the exponent
// through the step scalars) row 0 holds sign(v) = +-1 instead.  Thread
// (32-key block, row w, quarter a) writes the eight key slots 8a .. 8a+7 of
// row w (one 16-byte store), as k_points_ks.
__device__ __forceinline__ void values_ks_item(const void* __restrict__ v, int dtype, int64_t n, int C, int R,
                                               float s, int sign_only, uint16_t* __restrict__ vt, int64_t t) {
  {
    const int a = (int)(t & 3);
    const int64_t rest = t >> 2;
    const int64_t blk = rest / R;
    const int w = (int)(rest - blk * R);
    uint16_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int z = 8 * a + e;
      const int64_t r = blk * 32 + 16 * ((z & 7) >> 2) + 4 * (z >> 3) + (z & 3);
      float val = (r < n && w < C) ? load_any(v, r * C + w, dtype) * s : 0.0f;
      if (sign_only) val = (r < n && w == 0) ? (val < 0.0f ? -1.0f : 1.0f) : 0.0f;
      h[e] = __builtin_bit_cast(uint16_t, (_Float16)val);
    }
    uint4 pk;
    pk.x = h[0] | ((uint32_t)h[1] << 16);
    pk.y = h[2] | ((uint32_t)h[3] << 16);
    pk.z = h[4] | ((uint32_t)h[5] << 16);
    pk.w = h[6] | ((uint32_t)h[7] << 16);
    *reinterpret_cast<uint4*>(vt + ((blk * R + w) * 32 + 8 * a)) = pk;
  }
}

__global__ void k_values_ks(const void* __restrict__ v, int dtype, int64_t n, int C, int64_t n_pad,
                            int R, const uint32_t* __restrict__ slot, int sign_only,
                            uint16_t* __restrict__ vt, Bz bz) {
  v = zoff(v, bz.in);
  slot = zoff(slot, bz.ws);
  vt = zoff(vt, bz.ws);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float s = ldexpf(1.0f, scale_exponent(*slot));
  const int64_t total = (n_pad >> 5) * R * 4;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride)
    values_ks_item(v, dtype, n, C, R, s, sign_only, vt, t);
}

// Row-bound sample of a point set: rows n_j = floor(j N / kSampleRows) for
// j < kSampleRows (repeats when N is smaller), in RT layout (input dtype) with
// their half norms.  Stored coarse-first: positions 0 .. kSampleCoarse-1 hold
// j = 0, 16, 32, ... (the rows floor(i N / kSampleCoarse)), the remaining
// positions the other j in increasing order, so that the coarse sample is the
// first kSampleCoarse / 16 RT tiles.  nh: the half norms of the point set
// (k_points_rt_norm), copied so that sampled and streamed keys agree exactly.
__global__ void k_sample(const uint16_t* __restrict__ x, int64_t n, int D, int W,
                         const float* __restrict__ nh, uint16_t* __restrict__ srt,
                         float* __restrict__ snh, Bz bz) {
  constexpr int kStride = kSampleRows / kSampleCoarse;
  x = zoff(x, bz.in);
  nh = zoff(nh, bz.ws);
  srt = zoff(srt, bz.ws);
  snh = zoff(snh, bz.ws);
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= kSampleRows * W) return;
  const int pos = t / W, w = t - (t / W) * W;
  int j;
  if (pos < kSampleCoarse) {
    j = kStride * pos;
  } else {
    const int q = pos - kSampleCoarse;
    j = (q / (kStride - 1)) * kStride + q % (kStride - 1) + 1;
  }
  const bool real = n > 0;
  const int64_t r = real ? ((int64_t)j * n) / kSampleRows : 0;
  srt[rt_index(pos, w, W)] = (real && w < D) ? x[r * D + w] : (uint16_t)0;
  if (w == 0) snh[pos] = real ? nh[r] : kPadBias;  // the row's own half norm (same value)
}

// Per-step key scalars, 64 floats (256 bytes) per 32-key step:
//   [0, 32)  key bias b_n = -||k_n||^2/2, and for single-channel values
//            (v != NULL) additionally log2|v_n 2^e| / tau' with e from *slot
//            putting max |v 2^e| in [0.5, 1): the magnitude of v_n then enters
//            the exponent in fp32 (log2 0 = -inf gives an exact 0);
//   [32, 48) for single-channel values, sign(v_n) as fp16 +-1 in key-slot
//            order (the order of the MFMA B operand built from two score
//            tiles), two per float; otherwise 0;
//   [48, 64) unused, 0.
// Entry i < 32 of a step's scalars: the key bias of key r from its half
// norm (plus log2 |v_r sc| / tau' for single-channel values v != NULL).
__device__ __forceinline__ float key_bias(float half, const void* __restrict__ v, int dtype, int64_t n,
                                          int64_t r, float sc, float tau2) {
  float val = half;
  if (v && r < n) val += log2f(fabsf(load_any(v, r, dtype) * sc)) / tau2;
  return val;
}
// Entry i in [32, 64) of the scalars of step s: two fp16 signs of v in key-slot
// order for i < 48 and single-channel values (v != NULL), else 0.
__device__ __forceinline__ float step_sign_word(const void* __restrict__ v, int dtype, int64_t n, int64_t s,
                                                int i) {
  if (i >= 48 || !v) return 0.0f;
  uint32_t bits = 0;
  for (int h = 0; h < 2; ++h) {
    const int z = 2 * (i - 32) + h;
    const int64_t r = s * 32 + 16 * ((z & 7) >> 2) + 4 * (z >> 3) + (z & 3);
    const bool neg = r < n && load_any(v, r, dtype) < 0.0f;
    bits |= (neg ? 0xBC00u : 0x3C00u) << (16 * h);
  }
  return __builtin_bit_cast(float, bits);
}

__global__ void k_step_scalars(const float* __restrict__ nh, const void* __restrict__ v, int dtype,
                               int64_t n, int64_t n_pad, const uint32_t* __restrict__ slot, float tau2,
                               float* __restrict__ out, Bz bz) {
  nh = zoff(nh, bz.ws);
  v = zoff(v, bz.in);
  slot = zoff(slot, bz.ws);
  out = zoff(out, bz.ws);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float sc = v ? ldexpf(1.0f, scale_exponent(*slot) - 1) : 0.0f;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n_pad * 2; t += stride) {
    const int64_t s = t >> 6;
    const int i = (int)(t & 63);
    out[t] = i < 32 ? key_bias(nh[s * 32 + i], v, dtype, n, s * 32 + i, sc, tau2)
                    : step_sign_word(v, dtype, n, s, i);
  }
}

// All per-call preparation of a small forward problem in one launch (the
// chain fill / |v| maximum / copies / scalars takes nine dependent launches
// of a few microseconds each otherwise): every workgroup first reduces
// max |v| over all N x C values itself (no atomics, nothing to clear; the
// caller keeps N C small), then the grid-stride items are, in order, the RT
// copy and half norms of q (segment A), of k with the first 32 step scalars
// of each key (B; skipped when q and k are the same array), the KS copy of
// the values (C) and the sign words of the step scalars (D).  Segment lengths
// are multiples of the wave size, so the lanes of a point row stay in one
// wave.  slot receives max |v| (as gauss_sum's prep would write it).  The
// results are bitwise those of the separate kernels.
template <typename T>
__global__ __launch_bounds__(256) void k_prep_fwd_small(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, int alias, const void* __restrict__ v,
    int vdt, int64_t M, int64_t N, int D, int C, int64_t Mp, int64_t Np, int W, int R, int vecq, int veck,
    float tau2, uint16_t* __restrict__ qrt, float* __restrict__ qnh, uint16_t* __restrict__ krt,
    float* __restrict__ knh, uint16_t* __restrict__ vks, float* __restrict__ scal,
    uint32_t* __restrict__ slot) {
  __shared__ uint32_t wmax[256 / kWave];
  uint32_t mb = 0;
  for (int64_t i = threadIdx.x; i < N * C; i += blockDim.x) {
    const uint32_t b = __builtin_bit_cast(uint32_t, fabsf(load_any(v, i, vdt)));
    mb = b > mb ? b : mb;
  }
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t o = (uint32_t)__shfl_xor((int)mb, off, kWave);
    mb = o > mb ? o : mb;
  }
  if ((threadIdx.x & (kWave - 1)) == 0) wmax[threadIdx.x / kWave] = mb;
  __syncthreads();
  mb = wmax[0];
  for (int w = 1; w < (int)(blockDim.x / kWave); ++w) mb = wmax[w] > mb ? wmax[w] : mb;
  if (blockIdx.x == 0 && threadIdx.x == 0) *slot = mb;
  const int e = scale_exponent(mb);
  const float sv = ldexpf(1.0f, e);                           // values (KS copy)
  const void* v1 = C == 1 ? v : nullptr;                      // single channel: |v| in the scalars
  const float sc = v1 ? ldexpf(1.0f, e - 1) : 0.0f;
  const int cpr = W >> 3;
  const int64_t nA = Mp * cpr, nB = alias ? 0 : Np * cpr, nC = (Np >> 5) * R * 4, nD = Np;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < nA + nB + nC + nD; t += stride) {
    if (t < nA) {
      const float half = rt_norm_item<T>(q, M, D, W, qrt, qnh, vecq, t);
      const int64_t r = t / cpr;
      if (alias && t - r * cpr == 0) scal[(r >> 5) * 64 + (r & 31)] = key_bias(half, v1, vdt, N, r, sc, tau2);
    } else if (t < nA + nB) {
      const int64_t u = t - nA;
      const float half = rt_norm_item<T>(k, N, D, W, krt, knh, veck, u);
      const int64_t r = u / cpr;
      if (u - r * cpr == 0) scal[(r >> 5) * 64 + (r & 31)] = key_bias(half, v1, vdt, N, r, sc, tau2);
    } else if (t < nA + nB + nC) {
      values_ks_item(v, vdt, N, C, R, sv, C == 1, vks, t - nA - nB);
    } else {
      const int64_t u = t - nA - nB - nC;
      const int64_t s = u >> 5;
      const int i = 32 + (int)(u & 31);
      scal[s * 64 + i] = step_sign_word(v1, vdt, N, s, i);
    }
  }
}

// Inner product sum_m v_m s_m in fp64, fixed order: workgroup b sums the
// elements b*256 + t + k*gridDim*256 of thread t in index order, then a
// fixed tree over its threads; k_dot_final adds the workgroup partials in
// index order.  So the result does not depend on timing.
__global__ void k_dot_partial(const void* __restrict__ v, int dtype, const float* __restrict__ s,
                              int64_t n, double* __restrict__ part) {
  __shared__ double red[256];
  double acc = 0.0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    acc += (double)load_any(v, i, dtype) * (double)s[i];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) part[blockIdx.x] = red[0];
}

__global__ void k_dot_final(const double* __restrict__ part, int parts, double* __restrict__ out) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  double acc = 0.0;
  for (int b = 0; b < parts; ++b) acc += part[b];
  *out = acc;
}

// out[m, w] = sum_s part[s, m, w] in split order (deterministic); four
// elements per thread where count allows 16-byte accesses, the loads of up to
// eight splits issued together before they are added in order.
__global__ void k_combine(const float* __restrict__ part, int splits, int64_t count,
                          float* __restrict__ out, Bz bz) {
  part = zoff(part, bz.ws);
  out = zoff(out, bz.out);
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if ((count & 3) == 0) {
    const int64_t c4 = count >> 2;
    const float4* p4 = reinterpret_cast<const float4*>(part);
    for (; i < c4; i += stride) {
      float4 acc = p4[i];
      for (int s0 = 1; s0 < splits; s0 += 8) {
        float4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (s0 + u < splits) v[u] = p4[(int64_t)(s0 + u) * c4 + i];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (s0 + u < splits) {
            acc.x += v[u].x;
            acc.y += v[u].y;
            acc.z += v[u].z;
            acc.w += v[u].w;
          }
      }
      reinterpret_cast<float4*>(out)[i] = acc;
    }
    return;
  }
  for (; i < count; i += stride) {
    float acc = part[i];
    for (int s0 = 1; s0 < splits; s0 += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (s0 + u < splits) v[u] = part[(int64_t)(s0 + u) * count + i];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (s0 + u < splits) acc += v[u];
    }
    out[i] = acc;
  }
}

}  // namespace gs
