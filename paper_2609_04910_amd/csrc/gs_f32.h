// gs_f32.h -- the fp32-accuracy tier of the forward sum (Eq. 1) for fp32
// points and a single value channel (the single-precision setting of App.
// A.2: C = 1).
//
// Scores.  Each fp32 point set is scaled by an exact power of two 2^e (its
// largest magnitude into [2^14, 2^15)) and split into two fp16 numbers,
// x 2^e = hi + lo with hi = fp16(x 2^e) and lo = fp16(x 2^e - hi) (the
// difference is exact in fp32), so hi + lo carries 22 significant bits and
// no part leaves the fp16 range.  q.k is then three fp16 MFMAs per operand
// chunk, lo.hi + hi.lo + hi.hi (lo.lo, below 2^-22 of the product, is
// dropped), accumulated in fp32 on top of the key bias, in scaled units
// 2^(eq + ek); the exponent fma folds the scale back into tau'.
//
// Values.  As in the fp16 tier, |v_n| enters the exponent (log2 |v_n 2^ev| in
// the key bias, max |v 2^ev| in [0.5, 1)), so exp2 yields Phi |v_n| in fp32
// directly.  Nothing is rounded to fp16 after the exponent: the signed sum
// sum_n sign(v_n) Phi |v_n| is accumulated in fp32 on the vector unit, with
// the signs read as +-1.0f from the step scalars in the row order of the
// score tile, in three levels: the eight terms of a lane in one step, the
// steps of a block of kAccBlock steps, and the blocks, added with Kahan's
// compensation (a flat fp32 sum over N/32 steps would lose about
// 2^-24 sqrt(N/32) / 3 of the sum).  So no row-maximum shift is needed: the
// only values lost are those below the fp32 normal range.
#pragma once

#include "gs_kernels.h"

namespace gs {

// Scale exponent of the split copies: max |x| 2^e in [2^14, 2^15).
constexpr int kSplitHeadroom = 14;
// Key steps per block of the blocked, compensated row sum.
constexpr int kAccBlock = 16;

// Queries per wave (16-row tiles) of the fp32-tier forward kernel.
constexpr int f32_qt(int DP) { return DP >= 8 ? 1 : 8 / DP; }

// fp32 points -> scaled hi / lo fp16 copies (RT layout) and fp32 half norms
// -||x||^2/2 (exact fp32 inputs, squares summed in fp64).  Thread (r, c) moves
// columns 8c .. 8c+7 of row r, as k_points_rt_norm (whole waves per row
// group, so the shuffles are safe).  slot: max |x| bits (k_absmax).
__global__ void k_points_split(const float* __restrict__ x, int64_t n, int D, int64_t n_pad, int W,
                               const uint32_t* __restrict__ slot, uint16_t* __restrict__ hi,
                               uint16_t* __restrict__ lo, float* __restrict__ nh, Bz bz) {
  x = zoff(x, bz.in);
  slot = zoff(slot, bz.ws);
  hi = zoff(hi, bz.ws);
  lo = zoff(lo, bz.ws);
  nh = zoff(nh, bz.ws);
  const int e = scale_exponent(*slot) + kSplitHeadroom;
  const int cpr = W >> 3;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n_pad * cpr; t += stride) {
    const int64_t r = t / cpr;
    const int c = (int)(t - r * cpr);
    uint16_t h[8], l[8];
    double acc = 0.0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int w = 8 * c + k;
      const float xv = (r < n && w < D) ? x[r * D + w] : 0.0f;
      acc += (double)xv * (double)xv;
      const float xs = ldexpf(xv, e);
      const _Float16 hh = (_Float16)xs;
      h[k] = __builtin_bit_cast(uint16_t, hh);
      l[k] = __builtin_bit_cast(uint16_t, (_Float16)(xs - (float)hh));
    }
    for (int off = cpr >> 1; off > 0; off >>= 1) acc += __shfl_xor(acc, off, kWave);
    uint4 ph, pl;
    ph.x = h[0] | ((uint32_t)h[1] << 16);
    ph.y = h[2] | ((uint32_t)h[3] << 16);
    ph.z = h[4] | ((uint32_t)h[5] << 16);
    ph.w = h[6] | ((uint32_t)h[7] << 16);
    pl.x = l[0] | ((uint32_t)l[1] << 16);
    pl.y = l[2] | ((uint32_t)l[3] << 16);
    pl.z = l[4] | ((uint32_t)l[5] << 16);
    pl.w = l[6] | ((uint32_t)l[7] << 16);
    *reinterpret_cast<uint4*>(hi + rt_index(r, 8 * c, W)) = ph;
    *reinterpret_cast<uint4*>(lo + rt_index(r, 8 * c, W)) = pl;
    if (c == 0) nh[r] = r < n ? (float)(-0.5 * acc) : kPadBias;
  }
}

// Per-step scalars of the fp32 tier, 64 floats per 32-key step (v = NULL for
// several value channels: the bias is the scaled half norm alone, signs +1):
//   [0, 32)  2^(eq + ek) (b_n + log2 |v_n 2^ev| / tau'), the key bias in the
//            scaled units of the split scores (-inf for padding keys and for
//            v_n = 0: an exact zero term);
//   [32, 64) sign(v_n) as +-1.0f, key 32 s + i at position 32 + i (the row
//            order of the two 16-key score tiles).
// slot_v / slot_q / slot_k: max |v|, max |q|, max |k| bits.  The bias is
// formed in fp64 and rounded once (the fp32 log2 and its division would add
// about one ulp of a systematic error to every term).
__global__ void k_step_scalars32(const float* __restrict__ nh, const void* __restrict__ v, int dtype,
                                 int64_t n, int64_t n_pad, const uint32_t* __restrict__ slot_v,
                                 const uint32_t* __restrict__ slot_q, const uint32_t* __restrict__ slot_k,
                                 float tau2, float* __restrict__ out, Bz bz) {
  nh = zoff(nh, bz.ws);
  v = zoff(v, bz.in);
  slot_v = zoff(slot_v, bz.ws);
  slot_q = zoff(slot_q, bz.ws);
  slot_k = zoff(slot_k, bz.ws);
  out = zoff(out, bz.ws);
  const int ev = scale_exponent(*slot_v) - 1;
  const int es = scale_exponent(*slot_q) + scale_exponent(*slot_k) + 2 * kSplitHeadroom;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n_pad * 2; t += stride) {
    const int64_t r = (t >> 6) * 32 + (t & 31);
    float val;
    if ((t & 63) < 32) {
      val = -__builtin_inff();
      if (r < n) {
        const double lv = v ? log2(fabs((double)load_any(v, r, dtype))) + ev : 0.0;
        val = (float)ldexp((double)nh[r] + lv / (double)tau2, es);
      }
    } else {
      val = (v && r < n && load_any(v, r, dtype) < 0.0f) ? -1.0f : 1.0f;
    }
    out[t] = val;
  }
}

// Values (several channels) for the fp32 tier: v 2^ev (max |v| 2^ev in [1, 2))
// split into fp16 hi + lo, both in KS layout (R = C padded to 16), written as
// k_values_ks does (eight key slots of one row per thread, 16-byte stores).
__global__ void k_values_ks_split(const void* __restrict__ v, int dtype, int64_t n, int C, int64_t n_pad,
                                  int R, const uint32_t* __restrict__ slot, uint16_t* __restrict__ vh,
                                  uint16_t* __restrict__ vl, Bz bz) {
  v = zoff(v, bz.in);
  slot = zoff(slot, bz.ws);
  vh = zoff(vh, bz.ws);
  vl = zoff(vl, bz.ws);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int ev = scale_exponent(*slot);
  const int64_t total = (n_pad >> 5) * R * 4;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
    const int a = (int)(t & 3);
    const int64_t rest = t >> 2;
    const int64_t blk = rest / R;
    const int w = (int)(rest - blk * R);
    uint16_t h[8], l[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int z = 8 * a + e;
      const int64_t r = blk * 32 + 16 * ((z & 7) >> 2) + 4 * (z >> 3) + (z & 3);
      const float x = (r < n && w < C) ? ldexpf(load_any(v, r * C + w, dtype), ev) : 0.0f;
      const _Float16 hh = (_Float16)x;
      h[e] = __builtin_bit_cast(uint16_t, hh);
      l[e] = __builtin_bit_cast(uint16_t, (_Float16)(x - (float)hh));
    }
    uint4 ph, pl;
    ph.x = h[0] | ((uint32_t)h[1] << 16);
    ph.y = h[2] | ((uint32_t)h[3] << 16);
    ph.z = h[4] | ((uint32_t)h[5] << 16);
    ph.w = h[6] | ((uint32_t)h[7] << 16);
    pl.x = l[0] | ((uint32_t)l[1] << 16);
    pl.y = l[2] | ((uint32_t)l[3] << 16);
    pl.z = l[4] | ((uint32_t)l[5] << 16);
    pl.w = l[6] | ((uint32_t)l[7] << 16);
    const int64_t o = (blk * R + w) * 32 + 8 * a;
    *reinterpret_cast<uint4*>(vh + o) = ph;
    *reinterpret_cast<uint4*>(vl + o) = pl;
  }
}

// s_m = sum_n Phi(q_m, k_n) v_n for fp32 points, C = 1 (see the top of this
// file).  qh / ql, kh / kl: split copies (RT layout); nhq: query half norms;
// scal: k_step_scalars32; slots: [0] max |v|, [2] max |q|, [3] max |k| (the
// key slot is [2] when q and k are the same array: kslot selects it).
// Key steps are split over grid.y as in k_fwd (partials at part_stride);
// problems of a batch on grid.z (strides of bz).
template <int DP>
__global__ __launch_bounds__(kBlockThreads) void k_fwd32(
    const uint4* __restrict__ qh, const uint4* __restrict__ ql, const float* __restrict__ nhq,
    const uint4* __restrict__ kh, const uint4* __restrict__ kl, const float* __restrict__ scal,
    const uint32_t* __restrict__ slots, int kslot, float tau2, int64_t M, int steps_total,
    int steps_per_split, float* __restrict__ out, int64_t part_stride, Bz bz) {
  qh = zoff(qh, bz.ws);
  ql = zoff(ql, bz.ws);
  nhq = zoff(nhq, bz.ws);
  kh = zoff(kh, bz.ws);
  kl = zoff(kl, bz.ws);
  scal = zoff(scal, bz.ws);
  slots = zoff(slots, bz.ws);
  out = zoff(out, bz.out);
  constexpr int QT = f32_qt(DP);
  constexpr int KCH = 2 * DP;    // 1-KiB chunks of one key copy per step
  constexpr int NCH = 2 * KCH;   // hi and lo
  constexpr int STAGE = NCH * 1024 + kScalarFloats * 4;
  constexpr int NS = ring_stages(STAGE, NCH + 1);
  __shared__ __attribute__((aligned(1024))) char lds[NS * STAGE];

  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t dlane = dma_lane_offset(lane);
  const int wave = threadIdx.x / kWave;
  const int j = lane & 15, g = lane >> 4;
  const int64_t q0 = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * (16 * QT);
  const int s_begin = blockIdx.y * steps_per_split;
  const int s_end = min(steps_total, s_begin + steps_per_split);
  out += blockIdx.y * part_stride;

  const bool mine = g == wave;
  const uint32_t nsteps = (uint32_t)max(0, s_end - s_begin);
  const auto rkh = make_rsrc(reinterpret_cast<const char*>(kh) + (int64_t)s_begin * KCH * 1024,
                             nsteps * KCH * 1024);
  const auto rkl = make_rsrc(reinterpret_cast<const char*>(kl) + (int64_t)s_begin * KCH * 1024,
                             nsteps * KCH * 1024);
  const auto rsc = make_rsrc(scal + (int64_t)s_begin * kScalarFloats, nsteps * kScalarFloats * 4);
  const uint32_t lds0 = lds_address(lds);
  auto issue = [&](int s, int stage) {
    if (!mine) return;
    const uint32_t base = lds0 + stage * STAGE;
    const uint32_t ls = (uint32_t)(s - s_begin);
#pragma unroll
    for (int c = 0; c < KCH; ++c) dma_x4(rkh, (ls * KCH + c) * 1024, base + c * 1024, dlane);
#pragma unroll
    for (int c = 0; c < KCH; ++c) dma_x4(rkl, (ls * KCH + c) * 1024, base + (KCH + c) * 1024, dlane);
    dma_x1(rsc, ls * kScalarFloats * 4, base + NCH * 1024, 4 * lane);
  };

  const int es = scale_exponent(slots[2]) + scale_exponent(slots[kslot]) + 2 * kSplitHeadroom;
  const float tau2s = ldexpf(tau2, -es);
  uint4 qhr[QT][DP], qlr[QT][DP];
  float bq[QT], A[QT], Ac[QT], blk[QT];  // sum of blocks, its compensation, current block
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    load_k_tile<DP>(qh, q0 / 16 + qt, j, g, qhr[qt]);
    load_k_tile<DP>(ql, q0 / 16 + qt, j, g, qlr[qt]);
    bq[qt] = tau2 * nhq[q0 + 16 * qt + j];
    A[qt] = Ac[qt] = blk[qt] = 0.0f;
  }
  settle(qhr);
  settle(qlr);
  settle(bq);
  // Kahan: A + Ac carries the sum of the finished blocks
  auto close_block = [&]() {
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      const float y = blk[qt] - Ac[qt];
      const float t = A[qt] + y;
      Ac[qt] = (t - A[qt]) - y;
      A[qt] = t;
      blk[qt] = 0.0f;
    }
  };
  int in_block = 0;

  auto compute = [&](int stage) {
    const char* base = lds + stage * STAGE;
    const uint4* khb = reinterpret_cast<const uint4*>(base);
    const uint4* klb = reinterpret_cast<const uint4*>(base + KCH * 1024);
    const float* sc = reinterpret_cast<const float*>(base + NCH * 1024);
    float part[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) part[qt] = 0.0f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const floatx4 cin = *reinterpret_cast<const floatx4*>(sc + 16 * kt + 4 * g);
      const floatx4 sg = *reinterpret_cast<const floatx4*>(sc + 32 + 16 * kt + 4 * g);
      uint4 khr[DP], klr[DP];
      load_k_tile_lds<DP>(khb, kt, j, g, khr);
      load_k_tile_lds<DP>(klb, kt, j, g, klr);
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        floatx4 acc = cin;
#pragma unroll
        for (int dc = 0; dc < DP; ++dc) {
          acc = mfma_f16(klr[dc], qhr[qt][dc], acc);
          acc = mfma_f16(khr[dc], qlr[qt][dc], acc);
        }
#pragma unroll
        for (int dc = 0; dc < DP; ++dc) acc = mfma_f16(khr[dc], qhr[qt][dc], acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) part[qt] = fmaf(exp2_clamped(fmaf(acc[r], tau2s, bq[qt])), sg[r], part[qt]);
      }
    }
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) blk[qt] += part[qt];
    if (++in_block == kAccBlock) {
      close_block();
      in_block = 0;
    }
  };
  key_stream<NS, NCH + 1>(s_begin, s_end, issue, compute);
  close_block();

  // the four row groups of the tile hold disjoint key subsets: add them in a
  // fixed order (every lane gets the same value)
  const int ev = scale_exponent(slots[0]) - 1;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    float x = A[qt] - Ac[qt];
    x += __shfl_xor(x, 16, kWave);
    x += __shfl_xor(x, 32, kWave);
    const int64_t m = q0 + 16 * qt + j;
    if (g == 0 && m < M) out[m] = ldexpf(x, -ev);
  }
}

}  // namespace gs

namespace gs {

// Several value channels (fp32 points, C > 1).  Two passes over the wave's
// keys through the LDS ring.  The first takes the exact row maximum of the
// exponent, with the same split scores as the second, so the largest scaled
// value of a row is exactly 2^kPScale.  The second evaluates
// P' = 2^(x - off + kPScale) in fp32, splits it into fp16 hi + lo (hi = P'
// rounded, lo = P' - hi rounded; the scale keeps lo out of the fp16
// subnormals for every value within 2^-14 of the row maximum) and contracts
// with the split values (v 2^ev = vh + vl): vh.Ph into a block accumulator
// that is added to the running sum with Kahan's compensation every kAccBlock
// steps, vl.Ph + vh.Pl (about 2^-11 of it) into a second accumulator.
constexpr int kPScale = 11;
// Queries per wave (16-row tiles) of the several-channel kernel.
constexpr int f32c_qt(int DP, int CT) { return (DP >= 4 || CT >= 4) ? 1 : 2; }
// Channels per launch of the several-channel kernel (16 * CT at most).
constexpr int kF32MaxChannels = 64;

// vh / vl: split values in KS layout, already advanced to this launch's first
// channel; vstep: bytes per key step of those arrays (R * 64); cw: channels
// of this launch; C: row stride of out (the problem's channel count); out
// already advanced to the first channel.
template <int DP, int CT>
__global__ __launch_bounds__(kBlockThreads) void k_fwd32c(
    const uint4* __restrict__ qh, const uint4* __restrict__ ql, const float* __restrict__ nhq,
    const uint4* __restrict__ kh, const uint4* __restrict__ kl, const float* __restrict__ scal,
    const uint4* __restrict__ vh, const uint4* __restrict__ vl, int vstep,
    const uint32_t* __restrict__ slots, int kslot, float tau2, int64_t M, int C, int cw, int steps_total,
    int steps_per_split, float* __restrict__ out, int64_t part_stride, Bz bz) {
  qh = zoff(qh, bz.ws);
  ql = zoff(ql, bz.ws);
  nhq = zoff(nhq, bz.ws);
  kh = zoff(kh, bz.ws);
  kl = zoff(kl, bz.ws);
  scal = zoff(scal, bz.ws);
  vh = zoff(vh, bz.ws);
  vl = zoff(vl, bz.ws);
  slots = zoff(slots, bz.ws);
  out = zoff(out, bz.out);
  constexpr int QT = f32c_qt(DP, CT);
  constexpr int KCH = 2 * DP;           // 1-KiB chunks of one key copy per step
  constexpr int NCH = 2 * KCH + 2 * CT; // key hi, lo, value hi, lo
  constexpr int STAGE = NCH * 1024 + kScalarFloats * 4;
  constexpr int NS = ring_stages(STAGE, NCH + 1);
  __shared__ __attribute__((aligned(1024))) char lds[NS * STAGE];

  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t dlane = dma_lane_offset(lane);
  const int wave = threadIdx.x / kWave;
  const int j = lane & 15, g = lane >> 4;
  const int64_t q0 = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * (16 * QT);
  const int s_begin = blockIdx.y * steps_per_split;
  const int s_end = min(steps_total, s_begin + steps_per_split);
  out += blockIdx.y * part_stride;

  const bool mine = g == wave;
  const uint32_t nsteps = (uint32_t)max(0, s_end - s_begin);
  const auto rkh = make_rsrc(reinterpret_cast<const char*>(kh) + (int64_t)s_begin * KCH * 1024,
                             nsteps * KCH * 1024);
  const auto rkl = make_rsrc(reinterpret_cast<const char*>(kl) + (int64_t)s_begin * KCH * 1024,
                             nsteps * KCH * 1024);
  const auto rvh = make_rsrc(reinterpret_cast<const char*>(vh) + (int64_t)s_begin * vstep,
                             nsteps * (uint32_t)vstep);
  const auto rvl = make_rsrc(reinterpret_cast<const char*>(vl) + (int64_t)s_begin * vstep,
                             nsteps * (uint32_t)vstep);
  const auto rsc = make_rsrc(scal + (int64_t)s_begin * kScalarFloats, nsteps * kScalarFloats * 4);
  const uint32_t lds0 = lds_address(lds);
  // first pass: keys and scalars only
  auto issue_k = [&](int s, int stage) {
    if (!mine) return;
    const uint32_t base = lds0 + stage * STAGE;
    const uint32_t ls = (uint32_t)(s - s_begin);
#pragma unroll
    for (int c = 0; c < KCH; ++c) dma_x4(rkh, (ls * KCH + c) * 1024, base + c * 1024, dlane);
#pragma unroll
    for (int c = 0; c < KCH; ++c) dma_x4(rkl, (ls * KCH + c) * 1024, base + (KCH + c) * 1024, dlane);
    dma_x1(rsc, ls * kScalarFloats * 4, base + NCH * 1024, 4 * lane);
  };
  auto issue_all = [&](int s, int stage) {
    issue_k(s, stage);
    if (!mine) return;
    const uint32_t base = lds0 + stage * STAGE;
    const uint32_t ls = (uint32_t)(s - s_begin);
#pragma unroll
    for (int c = 0; c < CT; ++c)
      dma_x4(rvh, ls * (uint32_t)vstep + c * 1024, base + (2 * KCH + c) * 1024, dlane);
#pragma unroll
    for (int c = 0; c < CT; ++c)
      dma_x4(rvl, ls * (uint32_t)vstep + c * 1024, base + (2 * KCH + CT + c) * 1024, dlane);
  };

  const int es = scale_exponent(slots[2]) + scale_exponent(slots[kslot]) + 2 * kSplitHeadroom;
  const float tau2s = ldexpf(tau2, -es);
  uint4 qhr[QT][DP], qlr[QT][DP];
  float bq[QT], smax[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    load_k_tile<DP>(qh, q0 / 16 + qt, j, g, qhr[qt]);
    load_k_tile<DP>(ql, q0 / 16 + qt, j, g, qlr[qt]);
    bq[qt] = tau2 * nhq[q0 + 16 * qt + j];
    smax[qt] = -__builtin_inff();
  }
  settle(qhr);
  settle(qlr);
  settle(bq);
  auto score = [&](const uint4 (&khr)[DP], const uint4 (&klr)[DP], int qt, floatx4 cin) {
    floatx4 acc = cin;
#pragma unroll
    for (int dc = 0; dc < DP; ++dc) {
      acc = mfma_f16(klr[dc], qhr[qt][dc], acc);
      acc = mfma_f16(khr[dc], qlr[qt][dc], acc);
    }
#pragma unroll
    for (int dc = 0; dc < DP; ++dc) acc = mfma_f16(khr[dc], qhr[qt][dc], acc);
    return acc;
  };

  // pass 1: exact row maxima of the scaled score
  auto compute_max = [&](int stage) {
    const char* base = lds + stage * STAGE;
    const uint4* khb = reinterpret_cast<const uint4*>(base);
    const uint4* klb = reinterpret_cast<const uint4*>(base + KCH * 1024);
    const float* sc = reinterpret_cast<const float*>(base + NCH * 1024);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const floatx4 cin = *reinterpret_cast<const floatx4*>(sc + 16 * kt + 4 * g);
      uint4 khr[DP], klr[DP];
      load_k_tile_lds<DP>(khb, kt, j, g, khr);
      load_k_tile_lds<DP>(klb, kt, j, g, klr);
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) smax[qt] = max_into(smax[qt], score(khr, klr, qt, cin));
    }
  };
  key_stream<NS, 2 * KCH + 1>(s_begin, s_end, issue_k, compute_max);
  // every wave is done with the ring before the second pass refills it
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  float off[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    off[qt] = fmaf(wave_max_over_g(smax[qt]), tau2s, bq[qt]);
    if (!(off[qt] > -__builtin_inff())) off[qt] = 0.0f;  // empty key range
    bq[qt] = bq[qt] - off[qt] + (float)kPScale;
  }

  // pass 2
  floatx4 O1[QT][CT], O2[QT][CT], T[QT][CT], Tc[QT][CT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      O1[qt][ct] = O2[qt][ct] = T[qt][ct] = Tc[qt][ct] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
    }
  auto close_block = [&]() {
#pragma unroll
    for (int qt = 0; qt < QT; ++qt)
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float y = O1[qt][ct][r] - Tc[qt][ct][r];
          const float t = T[qt][ct][r] + y;
          Tc[qt][ct][r] = (t - T[qt][ct][r]) - y;
          T[qt][ct][r] = t;
          O1[qt][ct][r] = 0.0f;
        }
  };
  int in_block = 0;
  auto compute = [&](int stage) {
    const char* base = lds + stage * STAGE;
    const uint4* khb = reinterpret_cast<const uint4*>(base);
    const uint4* klb = reinterpret_cast<const uint4*>(base + KCH * 1024);
    const uint4* vhb = reinterpret_cast<const uint4*>(base + 2 * KCH * 1024);
    const uint4* vlb = reinterpret_cast<const uint4*>(base + (2 * KCH + CT) * 1024);
    const float* sc = reinterpret_cast<const float*>(base + NCH * 1024);
    uint4 vhr[CT], vlr[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      vhr[ct] = vhb[(16 * ct + j) * 4 + lds_col(j, g)];
      vlr[ct] = vlb[(16 * ct + j) * 4 + lds_col(j, g)];
    }
    float p[QT][2][4];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const floatx4 cin = *reinterpret_cast<const floatx4*>(sc + 16 * kt + 4 * g);
      uint4 khr[DP], klr[DP];
      load_k_tile_lds<DP>(khb, kt, j, g, khr);
      load_k_tile_lds<DP>(klb, kt, j, g, klr);
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        const floatx4 acc = score(khr, klr, qt, cin);
#pragma unroll
        for (int r = 0; r < 4; ++r) p[qt][kt][r] = __builtin_amdgcn_exp2f(fmaf(acc[r], tau2s, bq[qt]));
      }
    }
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      const uint4 bh = pack_tile_pair(p[qt]);
      const uint32_t hw[4] = {bh.x, bh.y, bh.z, bh.w};
      float lo[2][4];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const halfx2 h2 = __builtin_bit_cast(halfx2, hw[e >> 1]);
        lo[e >> 2][e & 3] = p[qt][e >> 2][e & 3] - (float)h2[e & 1];
      }
      const uint4 bl = pack_tile_pair(lo);
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        O1[qt][ct] = mfma_f16(vhr[ct], bh, O1[qt][ct]);
        O2[qt][ct] = mfma_f16(vlr[ct], bh, O2[qt][ct]);
        O2[qt][ct] = mfma_f16(vhr[ct], bl, O2[qt][ct]);
      }
    }
    if (++in_block == kAccBlock) {
      close_block();
      in_block = 0;
    }
  };
  key_stream<NS, NCH + 1>(s_begin, s_end, issue_all, compute);
  close_block();

  const int ev = scale_exponent(slots[0]);
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int64_t m = q0 + 16 * qt + j;
    if (m >= M) continue;
    // 2^(off - kPScale - ev), the integer part through ldexp (no denormal factor)
    const float fo = floorf(off[qt]);
    const float f = exp2f(off[qt] - fo);
    const int e = (int)fo - kPScale - ev;
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int c = 16 * ct + 4 * g + r;
        const float x = (T[qt][ct][r] - Tc[qt][ct][r]) + O2[qt][ct][r];
        if (c < cw) out[m * C + c] = ldexpf(x * f, e);
      }
  }
}

}  // namespace gs
