// gs_kernels.h -- the fused Gauss-sum kernels for gfx950.
//
// k_fwd  : s_m = sum_n Phi(q_m, k_n) v_n                      (Eq. 1)
// k_dq   : dq_m = tau sum_n Phi w_mn (k_n - q_m)              (Sec. 3 gradient)
//          with w_mn = <g_m, v_n>, evaluated as tau (sum_n P k_n - q_m sum_n P),
//          P = Phi * w.  The same kernel gives dk with the roles of (q, g) and
//          (k, v) exchanged, and k_fwd gives dv = sum_m Phi g_m likewise.
//
// Work decomposition: a workgroup is 4 independent waves; wave w owns
// 16*QT queries and walks the key range of its split (blockIdx.y) in steps of
// 32 keys.  Per step and query tile it computes two 16x16 tiles of
// S~^T[n][m] = q_m.k_n - ||k_n||^2/2 on the matrix cores (the key half-norm
// enters as the accumulator input, so it costs no vector instruction), forms
// the exponent x = tau' S~ + (-tau'||q_m||^2/2 - off_m) with one fma
// (tau' = tau log2 e), takes exp2 clamped to [0, 1] on the transcendental unit
// and rounds to fp16; the eight values per lane are exactly the B operand of
// the next MFMA over the 32 keys.  Nothing of size M x N is ever stored.
//
// Range: kernel values are fp16 numbers in [0, 1].  When every sampled row
// maximum of the wave's queries is at least 2^-8 the offset off_m is 0;
// otherwise the wave first walks its keys once to find the exact row maximum
// of the exponent and uses it as off_m (so the largest value of every row is
// 1 and fp16 keeps full relative precision for all values within 2^-14 of
// it); the epilogue multiplies by 2^off_m.  Values and upstream gradients are
// pre-scaled by exact powers of two (largest magnitude in [1, 2)), undone in
// the epilogue.
#pragma once

#include "gs_common.h"

namespace gs {

// Waves whose sampled row maximum of the log2 kernel value falls below this
// evaluate the row maxima exactly first.
constexpr float kShiftBelow = -8.0f;

__device__ __forceinline__ float max4(floatx4 a) {
  return fmaxf(fmaxf(a[0], a[1]), fmaxf(a[2], a[3]));
}

__device__ __forceinline__ float wave_max_over_g(float x) {
  x = fmaxf(x, __shfl_xor(x, 16, kWave));
  x = fmaxf(x, __shfl_xor(x, 32, kWave));
  return x;
}

// S~^T tile (16 keys x 16 queries) for key tile `kt16` (global 16-key tile
// index) against the query operand of one query tile.
template <typename T, int DP>
__device__ __forceinline__ floatx4 score_tile(const uint4 (&kr)[DP], const uint4 (&qr)[DP], floatx4 cin) {
  floatx4 acc = cin;
#pragma unroll
  for (int dc = 0; dc < DP; ++dc) acc = mfma_qk<T>(kr[dc], qr[dc], acc);
  return acc;
}

// Walks keys [s_begin, s_end) once and returns, per query tile, the exact row
// maximum of S~ (identical MFMA inputs and order as the main loop).
template <typename T, int DP, int QT>
__device__ __forceinline__ void row_max(const uint4* __restrict__ ks, const float* __restrict__ nhk,
                                        const uint4 (&qreg)[QT][DP], int s_begin, int s_end, int j,
                                        int g, float (&smax)[QT]) {
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) smax[qt] = -__builtin_inff();
  for (int s = s_begin; s < s_end; ++s) {
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int64_t tile = 2 * (int64_t)s + kt;
      floatx4 cin = *reinterpret_cast<const floatx4*>(nhk + tile * 16 + 4 * g);
      uint4 kr[DP];
#pragma unroll
      for (int dc = 0; dc < DP; ++dc) kr[dc] = ks[((tile * DP + dc) * 16 + j) * 4 + g];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt)
        smax[qt] = fmaxf(smax[qt], max4(score_tile<T, DP>(kr, qreg[qt], cin)));
    }
  }
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) smax[qt] = wave_max_over_g(smax[qt]);
}

template <typename T, int DP, int CT, int QT>
__global__ __launch_bounds__(kBlockThreads) void k_fwd(
    const uint4* __restrict__ qs, const float* __restrict__ nhq, const float* __restrict__ Lq,
    const uint4* __restrict__ ks, const float* __restrict__ nhk, const uint4* __restrict__ vt,
    const uint32_t* __restrict__ vslot, float tau2, int64_t M, int C, int steps_total,
    int steps_per_split, float* __restrict__ out, int64_t part_stride) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int j = lane & 15, g = lane >> 4;
  const int64_t q0 = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * (16 * QT);
  const int s_begin = blockIdx.y * steps_per_split;
  const int s_end = min(steps_total, s_begin + steps_per_split);
  out += blockIdx.y * part_stride;

  uint4 qreg[QT][DP];
  float bq[QT], off[QT];
  float lmin = 0.0f;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int64_t tile = q0 / 16 + qt;
#pragma unroll
    for (int dc = 0; dc < DP; ++dc) qreg[qt][dc] = qs[((tile * DP + dc) * 16 + j) * 4 + g];
    bq[qt] = tau2 * nhq[q0 + 16 * qt + j];
    off[qt] = 0.0f;
    lmin = fminf(lmin, Lq[q0 + 16 * qt + j]);
  }
  if (__any(lmin < kShiftBelow)) {
    float smax[QT];
    row_max<T, DP, QT>(ks, nhk, qreg, s_begin, s_end, j, g, smax);
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      off[qt] = fmaf(smax[qt], tau2, bq[qt]);
      if (!(off[qt] > -__builtin_inff())) off[qt] = 0.0f;  // empty key range
      bq[qt] -= off[qt];
    }
  }

  floatx4 O[QT][CT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) O[qt][ct] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

  for (int s = s_begin; s < s_end; ++s) {
    floatx4 cin[2];
    uint4 kr[2][DP];
    uint4 vr[CT];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int64_t tile = 2 * (int64_t)s + kt;
      cin[kt] = *reinterpret_cast<const floatx4*>(nhk + tile * 16 + 4 * g);
#pragma unroll
      for (int dc = 0; dc < DP; ++dc) kr[kt][dc] = ks[((tile * DP + dc) * 16 + j) * 4 + g];
    }
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) vr[ct] = vt[((int64_t)s * (16 * CT) + 16 * ct + j) * 4 + g];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float p[2][4];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        floatx4 acc = score_tile<T, DP>(kr[kt], qreg[qt], cin[kt]);
#pragma unroll
        for (int r = 0; r < 4; ++r) p[kt][r] = exp2_clamped(fmaf(acc[r], tau2, bq[qt]));
      }
      uint4 b;
      b.x = pack_f16(p[0][0], p[0][1]);
      b.y = pack_f16(p[0][2], p[0][3]);
      b.z = pack_f16(p[1][0], p[1][1]);
      b.w = pack_f16(p[1][2], p[1][3]);
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

template <typename T, int DP, int CW, int QT>
__global__ __launch_bounds__(kBlockThreads) void k_dq(
    const uint4* __restrict__ qs, const float* __restrict__ nhq, const float* __restrict__ Lq,
    const uint4* __restrict__ ks, const float* __restrict__ nhk, const uint4* __restrict__ kt_ks,
    const uint32_t* __restrict__ kslot, const uint4* __restrict__ vs,
    const uint32_t* __restrict__ vslot, const uint4* __restrict__ gs,
    const uint32_t* __restrict__ gslot, float tau2, float tau, int64_t M, int D, int steps_total,
    int steps_per_split, float* __restrict__ out, int64_t part_stride) {
  constexpr int DT = 2 * DP;  // 16-row tiles of the KS copy of the key points
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int j = lane & 15, g = lane >> 4;
  const int64_t q0 = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * (16 * QT);
  const int s_begin = blockIdx.y * steps_per_split;
  const int s_end = min(steps_total, s_begin + steps_per_split);
  out += blockIdx.y * part_stride;

  uint4 qreg[QT][DP];
  uint4 greg[QT][CW];
  float bq[QT], off[QT];
  float lmin = 0.0f;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int64_t tile = q0 / 16 + qt;
#pragma unroll
    for (int dc = 0; dc < DP; ++dc) qreg[qt][dc] = qs[((tile * DP + dc) * 16 + j) * 4 + g];
#pragma unroll
    for (int cw = 0; cw < CW; ++cw) greg[qt][cw] = gs[((tile * CW + cw) * 16 + j) * 4 + g];
    bq[qt] = tau2 * nhq[q0 + 16 * qt + j];
    off[qt] = 0.0f;
    lmin = fminf(lmin, Lq[q0 + 16 * qt + j]);
  }
  if (__any(lmin < kShiftBelow)) {
    float smax[QT];
    row_max<T, DP, QT>(ks, nhk, qreg, s_begin, s_end, j, g, smax);
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      off[qt] = fmaf(smax[qt], tau2, bq[qt]);
      if (!(off[qt] > -__builtin_inff())) off[qt] = 0.0f;
      bq[qt] -= off[qt];
    }
  }

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
    floatx4 cin[2];
    uint4 kr[2][DP];
    uint4 vr[2][CW];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int64_t tile = 2 * (int64_t)s + kt;
      cin[kt] = *reinterpret_cast<const floatx4*>(nhk + tile * 16 + 4 * g);
#pragma unroll
      for (int dc = 0; dc < DP; ++dc) kr[kt][dc] = ks[((tile * DP + dc) * 16 + j) * 4 + g];
#pragma unroll
      for (int cw = 0; cw < CW; ++cw) vr[kt][cw] = vs[((tile * CW + cw) * 16 + j) * 4 + g];
    }
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float p[2][4];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        floatx4 acc = score_tile<T, DP>(kr[kt], qreg[qt], cin[kt]);
        floatx4 w = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int cw = 0; cw < CW; ++cw) w = mfma_f16(vr[kt][cw], greg[qt][cw], w);
#pragma unroll
        for (int r = 0; r < 4; ++r) p[kt][r] = exp2_clamped(fmaf(acc[r], tau2, bq[qt])) * w[r];
      }
      uint4 b;
      b.x = pack_f16(p[0][0], p[0][1]);
      b.y = pack_f16(p[0][2], p[0][3]);
      b.z = pack_f16(p[1][0], p[1][1]);
      b.w = pack_f16(p[1][2], p[1][3]);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        dQ[qt][dt] = mfma_f16(kt_ks[((int64_t)s * (16 * DT) + 16 * dt + j) * 4 + g], b, dQ[qt][dt]);
      rs[qt] = mfma_f16(ones, b, rs[qt]);
    }
  }

  const int ev = scale_exponent(*vslot);
  const int eg = scale_exponent(*gslot);
  const int ek = kslot ? scale_exponent(*kslot) : 0;
  const uint16_t* q16 = reinterpret_cast<const uint16_t*>(qs);
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int64_t m = q0 + 16 * qt + j;
    if (m >= M) continue;
    const float f = tau * exp2f(off[qt]);
    const float rm = rs[qt][0];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int d = 16 * dt + 4 * g + r;
        if (d < D) {
          const float qv = T::to_float(q16[rt_index(m, d, 32 * DP)]);
          const float val = ldexpf(dQ[qt][dt][r], -ek) - qv * rm;
          out[m * D + d] = ldexpf(val * f, -ev - eg);
        }
      }
  }
}

}  // namespace gs
