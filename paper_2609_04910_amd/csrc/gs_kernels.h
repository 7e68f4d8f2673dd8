// gs_kernels.h -- the fused Gauss-sum kernels for gfx950.
//
// k_fwd  : s_m = sum_n Phi(q_m, k_n) v_n                      (Eq. 1)
// k_dq   : dq_m = tau sum_n Phi w_mn (k_n - q_m)              (Sec. 3 gradient)
//          with w_mn = <g_m, v_n>, evaluated as tau (sum_n P k_n - q_m sum_n P),
//          P = Phi * w.  The same kernel gives dk with the roles of (q, g) and
//          (k, v) exchanged, and k_fwd gives dv = sum_m Phi g_m likewise.
//
// Work decomposition: a workgroup is 4 waves that share one stream of key
// steps (32 keys each) through LDS; wave w owns 16*QT queries whose operands
// stay in registers.  Step s+1 is copied HBM -> LDS with the gfx950 direct
// loads (global_load_lds_dwordx4, no register round trip) while step s is
// computed, one barrier per step.  Per step and query tile a wave computes two
// 16x16 tiles of S~^T[n][m] = q_m.k_n - ||k_n||^2/2 on the matrix cores (the
// key half-norm enters as the accumulator input, so it costs no vector
// instruction), forms the exponent x = tau' S~ + (-tau'||q_m||^2/2 - off_m)
// with one fma (tau' = tau log2 e), takes exp2 clamped to [0, 1] on the
// transcendental unit and rounds pairs to fp16 with one v_cvt_pk; the eight
// values per lane are exactly the B operand of the next MFMA over the 32 keys.
// Nothing of size M x N is ever stored.
//
// Range: kernel values are fp16 numbers in [0, 1].  When every row maximum of
// the wave's queries over a fixed sample of 64 keys is at least 2^-8 the
// offset off_m is 0; otherwise the wave first walks its keys once to find the
// exact row maximum of the exponent and uses it as off_m (so the largest value
// of every row is 1 and fp16 keeps full relative precision for all values
// within 2^-14 of it); the epilogue multiplies by 2^off_m.  Values and
// upstream gradients are pre-scaled by exact powers of two (largest magnitude
// in [1, 2)), undone in the epilogue.
#pragma once

#include "gs_common.h"

namespace gs {

// Waves whose sampled row maximum of the log2 kernel value falls below this
// evaluate the row maxima exactly first.
constexpr float kShiftBelow = -8.0f;
constexpr int kSampleKeys = 64;        // keys in the row-bound sample (2 steps)
constexpr int kScalarFloats = 64;      // per step: 32 half norms, 32 scaled C = 1 values

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void glb_void;

// One wave copies 1 KiB: lane l moves 16 bytes from src + 16 l to dst + 16 l.
__device__ __forceinline__ void dma_1k(const char* src, char* dst, int lane) {
  __builtin_amdgcn_global_load_lds((glb_void*)(src + 16 * lane), (lds_void*)dst, 16, 0, 0);
}
// One wave copies 256 bytes: lane l moves 4 bytes.
__device__ __forceinline__ void dma_256(const char* src, char* dst, int lane) {
  __builtin_amdgcn_global_load_lds((glb_void*)(src + 4 * lane), (lds_void*)dst, 4, 0, 0);
}
// Wait until this wave's outstanding vector-memory loads (including the
// direct-to-LDS ones) have landed.
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

__device__ __forceinline__ float max4(floatx4 a) {
  return fmaxf(fmaxf(a[0], a[1]), fmaxf(a[2], a[3]));
}

__device__ __forceinline__ float wave_max_over_g(float x) {
  x = fmaxf(x, __shfl_xor(x, 16, kWave));
  x = fmaxf(x, __shfl_xor(x, 32, kWave));
  return x;
}

template <typename T, int DP>
__device__ __forceinline__ floatx4 score_tile(const uint4 (&kr)[DP], const uint4 (&qr)[DP], floatx4 cin) {
  floatx4 acc = cin;
#pragma unroll
  for (int dc = 0; dc < DP; ++dc) acc = mfma_qk<T>(kr[dc], qr[dc], acc);
  return acc;
}

// Loads the A operands of one 16-key tile (RT layout, `tile` relative to base).
template <int DP>
__device__ __forceinline__ void load_k_tile(const uint4* base, int64_t tile, int j, int g, uint4 (&kr)[DP]) {
#pragma unroll
  for (int dc = 0; dc < DP; ++dc) kr[dc] = base[((tile * DP + dc) * 16 + j) * 4 + g];
}

// Per-wave prologue: query operands, biases, and the offset decision.
//   sample_rt / sample_nh: 64 sampled keys of the key set (RT layout, half norms)
// Returns in off[] 0, or (when needed) a marker to compute exact maxima.
template <typename T, int DP, int QT>
__device__ __forceinline__ bool needs_shift(const uint4* __restrict__ sample_rt,
                                            const float* __restrict__ sample_nh,
                                            const uint4 (&qreg)[QT][DP], const float (&bq)[QT],
                                            float tau2, int64_t q0, int64_t M, int j, int g) {
  float smax[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) smax[qt] = -__builtin_inff();
#pragma unroll
  for (int t = 0; t < kSampleKeys / 16; ++t) {
    uint4 kr[DP];
    load_k_tile<DP>(sample_rt, t, j, g, kr);
    const floatx4 cin = *reinterpret_cast<const floatx4*>(sample_nh + 16 * t + 4 * g);
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) smax[qt] = fmaxf(smax[qt], max4(score_tile<T, DP>(kr, qreg[qt], cin)));
  }
  bool low = false;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const float L = fmaf(wave_max_over_g(smax[qt]), tau2, bq[qt]);
    low |= (q0 + 16 * qt + j < M) && (L < kShiftBelow);
  }
  return __any(low);
}

// Exact row maxima of S~ over the wave's key range, from the RT key copy in
// global memory (identical MFMA inputs and order as the main loop).
template <typename T, int DP, int QT>
__device__ __forceinline__ void exact_offsets(const uint4* __restrict__ ks, const float* __restrict__ scal,
                                           const uint4 (&qreg)[QT][DP], int s_begin, int s_end,
                                           int j, int g, float tau2, float (&bq)[QT], float (&off)[QT]) {
  float smax[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) smax[qt] = -__builtin_inff();
  for (int s = s_begin; s < s_end; ++s) {
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      uint4 kr[DP];
      load_k_tile<DP>(ks, 2 * (int64_t)s + kt, j, g, kr);
      const floatx4 cin =
          *reinterpret_cast<const floatx4*>(scal + (int64_t)s * kScalarFloats + 16 * kt + 4 * g);
#pragma unroll
      for (int qt = 0; qt < QT; ++qt)
        smax[qt] = fmaxf(smax[qt], max4(score_tile<T, DP>(kr, qreg[qt], cin)));
    }
  }
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    off[qt] = fmaf(wave_max_over_g(smax[qt]), tau2, bq[qt]);
    if (!(off[qt] > -__builtin_inff())) off[qt] = 0.0f;  // empty key range
    bq[qt] -= off[qt];
  }
}

__device__ __forceinline__ uint4 pack_tile_pair(const float (&p)[2][4]) {
  uint4 b;
  b.x = pack_f16(p[0][0], p[0][1]);
  b.y = pack_f16(p[0][2], p[0][3]);
  b.z = pack_f16(p[1][0], p[1][1]);
  b.w = pack_f16(p[1][2], p[1][3]);
  return b;
}

// ---------------------------------------------------------------- forward

template <typename T, int DP, int CT, int QT>
__global__ __launch_bounds__(kBlockThreads) void k_fwd(
    const uint4* __restrict__ qs, const float* __restrict__ nhq, const uint4* __restrict__ samp_rt,
    const float* __restrict__ samp_nh, const uint4* __restrict__ ks, const float* __restrict__ scal,
    const uint4* __restrict__ vt, const uint32_t* __restrict__ vslot, float tau2, int64_t M, int C,
    int steps_total, int steps_per_split, float* __restrict__ out, int64_t part_stride) {
  constexpr int KCH = 2 * DP;   // 1-KiB chunks of keys per step
  constexpr int NCH = KCH + CT; // + chunks of V^T
  constexpr int STAGE = NCH * 1024 + kScalarFloats * 4;
  __shared__ __attribute__((aligned(1024))) char lds[2 * STAGE];

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int j = lane & 15, g = lane >> 4;
  const int64_t q0 = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * (16 * QT);
  const int s_begin = blockIdx.y * steps_per_split;
  const int s_end = min(steps_total, s_begin + steps_per_split);
  out += blockIdx.y * part_stride;

  auto issue = [&](int s, int stage) {
    char* base = lds + stage * STAGE;
    for (int c = wave; c < NCH; c += kWavesPerBlock) {
      const char* src = c < KCH ? reinterpret_cast<const char*>(ks) + ((int64_t)s * KCH + c) * 1024
                                : reinterpret_cast<const char*>(vt) + ((int64_t)s * CT + (c - KCH)) * 1024;
      dma_1k(src, base + c * 1024, lane);
    }
    if (wave == kWavesPerBlock - 1)
      dma_256(reinterpret_cast<const char*>(scal + (int64_t)s * kScalarFloats), base + NCH * 1024, lane);
  };
  if (s_begin < s_end) issue(s_begin, 0);

  uint4 qreg[QT][DP];
  float bq[QT], off[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    load_k_tile<DP>(qs, q0 / 16 + qt, j, g, qreg[qt]);
    bq[qt] = tau2 * nhq[q0 + 16 * qt + j];
    off[qt] = 0.0f;
  }
  if (needs_shift<T, DP, QT>(samp_rt, samp_nh, qreg, bq, tau2, q0, M, j, g))
    exact_offsets<T, DP, QT>(ks, scal, qreg, s_begin, s_end, j, g, tau2, bq, off);

  floatx4 O[QT][CT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) O[qt][ct] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

  for (int s = s_begin; s < s_end; ++s) {
    const int stage = (s - s_begin) & 1;
    wait_loads();
    __syncthreads();
    if (s + 1 < s_end) issue(s + 1, stage ^ 1);
    const char* base = lds + stage * STAGE;
    const uint4* kb = reinterpret_cast<const uint4*>(base);
    const float* sc = reinterpret_cast<const float*>(base + NCH * 1024);
    floatx4 cin[2];
    uint4 kr[2][DP];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      cin[kt] = *reinterpret_cast<const floatx4*>(sc + 16 * kt + 4 * g);
      load_k_tile<DP>(kb, kt, j, g, kr[kt]);
    }
    uint4 vr[CT];
    const uint4* vb = reinterpret_cast<const uint4*>(base + KCH * 1024);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) vr[ct] = vb[(16 * ct + j) * 4 + g];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float p[2][4];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const floatx4 acc = score_tile<T, DP>(kr[kt], qreg[qt], cin[kt]);
#pragma unroll
        for (int r = 0; r < 4; ++r) p[kt][r] = exp2_clamped(fmaf(acc[r], tau2, bq[qt]));
      }
      const uint4 b = pack_tile_pair(p);
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) O[qt][ct] = mfma_f16(vr[ct], b, O[qt][ct]);
    }
  }

  const int ev = scale_exponent(*vslot);
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int64_t m = q0 + 16 * qt + j;
    if (m >= M) continue;
    const float f = exp2f(off[qt]);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int c = 16 * ct + 4 * g + r;
        if (c < C) out[m * C + c] = ldexpf(O[qt][ct][r] * f, -ev);
      }
  }
}

// ---------------------------------------------------------------- gradient
//
// CW = 0 selects the single-channel form (C = 1): w_mn = g_m v_n, so
// P = Phi v_n uses the per-key scaled values from the step scalars (one
// v_mul per pair, no W contraction) and g_m multiplies the epilogue.

template <typename T, int DP, int CW, int QT>
__global__ __launch_bounds__(kBlockThreads) void k_dq(
    const uint4* __restrict__ qs, const float* __restrict__ nhq, const uint4* __restrict__ samp_rt,
    const float* __restrict__ samp_nh, const uint4* __restrict__ ks, const float* __restrict__ scal,
    const uint4* __restrict__ kt_ks, const uint32_t* __restrict__ kslot, const uint4* __restrict__ vs,
    const uint32_t* __restrict__ vslot, const uint4* __restrict__ gs,
    const uint32_t* __restrict__ gslot, float tau2, float tau, int64_t M, int D, int steps_total,
    int steps_per_split, float* __restrict__ out, int64_t part_stride) {
  constexpr int DT = 2 * DP;                // 16-row tiles of K^T (KS layout)
  constexpr int KCH = 2 * DP;               // chunks of K (RT) per step
  constexpr int VCH = 2 * CW;               // chunks of V (RT) per step
  constexpr int TCH = DT;                   // chunks of K^T (KS) per step: 32 DP rows x 64 B
  constexpr int NCH = KCH + VCH + TCH;
  constexpr int STAGE = NCH * 1024 + kScalarFloats * 4;
  constexpr int GW = CW > 0 ? CW : 1;       // RT chunks of the upstream gradient
  __shared__ __attribute__((aligned(1024))) char lds[2 * STAGE];

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int j = lane & 15, g = lane >> 4;
  const int64_t q0 = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * (16 * QT);
  const int s_begin = blockIdx.y * steps_per_split;
  const int s_end = min(steps_total, s_begin + steps_per_split);
  out += blockIdx.y * part_stride;

  auto issue = [&](int s, int stage) {
    char* base = lds + stage * STAGE;
    for (int c = wave; c < NCH; c += kWavesPerBlock) {
      const char* src;
      if (c < KCH)
        src = reinterpret_cast<const char*>(ks) + ((int64_t)s * KCH + c) * 1024;
      else if (c < KCH + VCH)
        src = reinterpret_cast<const char*>(vs) + ((int64_t)s * VCH + (c - KCH)) * 1024;
      else
        src = reinterpret_cast<const char*>(kt_ks) + ((int64_t)s * TCH + (c - KCH - VCH)) * 1024;
      dma_1k(src, base + c * 1024, lane);
    }
    if (wave == kWavesPerBlock - 1)
      dma_256(reinterpret_cast<const char*>(scal + (int64_t)s * kScalarFloats), base + NCH * 1024, lane);
  };
  if (s_begin < s_end) issue(s_begin, 0);

  uint4 qreg[QT][DP];
  uint4 greg[QT][GW];
  float bq[QT], off[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    load_k_tile<DP>(qs, q0 / 16 + qt, j, g, qreg[qt]);
    if constexpr (CW > 0) load_k_tile<GW>(gs, q0 / 16 + qt, j, g, greg[qt]);
    bq[qt] = tau2 * nhq[q0 + 16 * qt + j];
    off[qt] = 0.0f;
  }
  if (needs_shift<T, DP, QT>(samp_rt, samp_nh, qreg, bq, tau2, q0, M, j, g))
    exact_offsets<T, DP, QT>(ks, scal, qreg, s_begin, s_end, j, g, tau2, bq, off);

  floatx4 dQ[QT][DT];
  floatx4 rs[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    rs[qt] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) dQ[qt][dt] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
  }
  const uint4 ones = {0x3C003C00u, 0x3C003C00u, 0x3C003C00u, 0x3C003C00u};  // fp16 1.0

  for (int s = s_begin; s < s_end; ++s) {
    const int stage = (s - s_begin) & 1;
    wait_loads();
    __syncthreads();
    if (s + 1 < s_end) issue(s + 1, stage ^ 1);
    const char* base = lds + stage * STAGE;
    const uint4* kb = reinterpret_cast<const uint4*>(base);
    const uint4* vb = reinterpret_cast<const uint4*>(base + KCH * 1024);
    const uint4* tb = reinterpret_cast<const uint4*>(base + (KCH + VCH) * 1024);
    const float* sc = reinterpret_cast<const float*>(base + NCH * 1024);
    floatx4 cin[2], vv[2];
    uint4 kr[2][DP];
    uint4 vr[2][GW];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      cin[kt] = *reinterpret_cast<const floatx4*>(sc + 16 * kt + 4 * g);
      load_k_tile<DP>(kb, kt, j, g, kr[kt]);
      if constexpr (CW > 0)
        load_k_tile<GW>(vb, kt, j, g, vr[kt]);
      else
        vv[kt] = *reinterpret_cast<const floatx4*>(sc + 32 + 16 * kt + 4 * g);
    }
    uint4 ktr[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) ktr[dt] = tb[(16 * dt + j) * 4 + g];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float p[2][4];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const floatx4 acc = score_tile<T, DP>(kr[kt], qreg[qt], cin[kt]);
        floatx4 w;
        if constexpr (CW > 0) {
          w = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int cw = 0; cw < CW; ++cw) w = mfma_f16(vr[kt][cw], greg[qt][cw], w);
        } else {
          w = vv[kt];
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) p[kt][r] = exp2_clamped(fmaf(acc[r], tau2, bq[qt])) * w[r];
      }
      const uint4 b = pack_tile_pair(p);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) dQ[qt][dt] = mfma_f16(ktr[dt], b, dQ[qt][dt]);
      rs[qt] = mfma_f16(ones, b, rs[qt]);
    }
  }

  const int ev = scale_exponent(*vslot);
  const int eg = scale_exponent(*gslot);
  const int ek = kslot ? scale_exponent(*kslot) : 0;
  const uint16_t* q16 = reinterpret_cast<const uint16_t*>(qs);
  const uint16_t* g16 = reinterpret_cast<const uint16_t*>(gs);
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int64_t m = q0 + 16 * qt + j;
    if (m >= M) continue;
    float f = tau * exp2f(off[qt]);
    int e = -ev;
    if constexpr (CW > 0) {
      e -= eg;
    } else {
      // single channel: w = g_m v_n, with g_m from its scaled fp16 copy
      f *= (float)__builtin_bit_cast(_Float16, g16[rt_index(m, 0, 32)]);
      e -= eg;
    }
    const float rm = rs[qt][0];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int d = 16 * dt + 4 * g + r;
        if (d < D) {
          const float qv = T::to_float(q16[rt_index(m, d, 32 * DP)]);
          const float val = ldexpf(dQ[qt][dt][r], -ek) - qv * rm;
          out[m * D + d] = ldexpf(val * f, e);
        }
      }
  }
}

}  // namespace gs
