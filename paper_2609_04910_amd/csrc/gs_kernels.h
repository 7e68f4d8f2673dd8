// gs_kernels.h -- the fused Gauss-sum kernels for gfx950.
//
// k_fwd  : s_m = sum_n Phi(q_m, k_n) v_n                      (Eq. 1)
// k_dq   : dq_m = tau sum_n Phi w_mn (k_n - q_m)              (Sec. 3 gradient)
//          with w_mn = <g_m, v_n>, evaluated as tau (sum_n P k_n - q_m sum_n P),
//          P = Phi * w.  The same kernel gives dk with the roles of (q, g) and
//          (k, v) exchanged, and k_fwd gives dv = sum_m Phi g_m likewise.
//
// Work decomposition: a workgroup is 4 waves (8 for D > 64: one workgroup
// per CU, the same ring then feeds twice the queries) that share one stream
// of key steps (32 keys each) through a two- to four-stage LDS ring; wave w
// owns 16*QT queries whose operands stay in registers.  Later steps are
// copied HBM -> LDS with the gfx950 direct loads (buffer_load ... lds, no
// register round trip) while step s is computed, one barrier per step.  Per step and query tile a wave computes two
// 16x16 tiles of S~^T[n][m] = q_m.k_n - ||k_n||^2/2 on the matrix cores (the
// key half-norm enters as the accumulator input, so it costs no vector
// instruction), forms the exponent x = tau' S~ + (-tau'||q_m||^2/2 - off_m)
// with one fma (tau' = tau log2 e), takes exp2 clamped to [0, 1] on the
// transcendental unit and rounds pairs to fp16 with one v_cvt_pk; the eight
// values per lane are exactly the B operand of the next MFMA over the 32 keys.
// Nothing of size M x N is ever stored.
//
// Range: kernel values are fp16 numbers in [0, 1].  When every row maximum of
// the wave's queries over a fixed sample of keys (64 keys; the forward also
// 1024, via k_row_check) is at least 2^-8 the offset off_m is 0.  Otherwise
// the forward kernel rounds 2^15 Phi instead, the exponent still clamped at
// <= 0 before the exact shift by 15 (so values are at most 2^15, inside the
// fp16 range, and keep full relative precision down to Phi = 2^-29), as long
// as the sampled row maxima are at least 2^-23; below that, and in the
// gradient kernel below 2^-8, the wave first walks its keys once to find the
// exact row maximum of the exponent and uses it as off_m (so the largest value
// of every row is 1 and fp16 keeps full relative precision for all values
// within 2^-14 of it).  The epilogue multiplies by 2^off_m (off_m = -15 for
// the shifted rows).  Values and upstream gradients are pre-scaled by exact
// powers of two (largest magnitude in [1, 2)), undone in the epilogue.
#pragma once

#include "gs_common.h"

#include <type_traits>

namespace gs {

// Waves whose sampled row maximum of the log2 kernel value falls below
// kShiftBelow leave the plain [0, 1] range: the forward kernel shifts its
// kernel values by 2^kSigma (exponent clamped at <= 0 first) while the sampled
// maxima stay at or above kExactBelow, and evaluates the row maxima exactly
// below that; the gradient kernel always takes the exact maxima.
constexpr float kShiftBelow = -8.0f;
constexpr float kSigma = 15.0f;
constexpr float kExactBelow = kShiftBelow - kSigma;
constexpr int kScalarFloats = 64;      // per step: 32 half norms, 32 scaled C = 1 values

// 2^min(y, kSigma): the kernel value times 2^kSigma for y = exponent + kSigma,
// the exponent clamped at <= 0 (so the result never exceeds 2^kSigma).
__device__ __forceinline__ float exp2_shifted(float y) {
  return __builtin_amdgcn_exp2f(fminf(y, kSigma));
}

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void glb_void;

// Buffer resource over `bytes` bytes from `base` (raw, unswizzled; reads past
// the end return zeros).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}

// Direct HBM -> LDS copies (buffer_load ... lds): lane l moves `size` bytes
// from rsrc + voff + soff to LDS address m0 + size * l.  They are issued as
// inline assembly so that the compiler neither sees nor waits for the
// asynchronous LDS writes; the key stream below orders them explicitly
// (s_waitcnt vmcnt + s_barrier).  Every wave issues one load per 1-KiB chunk of
// a step, moving its quarter of it (lanes 16w .. 16w+15, 16 bytes each), and
// one dword load for its quarter of the 256 bytes of step scalars, so all
// waves issue the same number of loads per step and "step s has landed" is an
// exact vmcnt.  Addresses are a buffer resource (SGPRs), a per-lane VGPR
// offset fixed for the kernel and a per-step SGPR offset.
__device__ __forceinline__ void dma_x4(__amdgpu_buffer_rsrc_t rs, uint32_t soff, uint32_t lds,
                                       uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(rs), "s"(soff)
               : "memory", "m0");
}
__device__ __forceinline__ void dma_x1(__amdgpu_buffer_rsrc_t rs, uint32_t soff, uint32_t lds,
                                       uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, %3 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(rs), "s"(soff)
               : "memory", "m0");
}

// s_waitcnt vmcnt(N), as assembly so that it is kept exactly as written.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0, "vmcnt range");
  if constexpr (N >= 64) return;  // only in the unused branch of the two-stage ring
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return (uint32_t)(uintptr_t)(const lds_void*)p;
}

// LDS ring of NS (2 to 4) stages over the key steps [s_begin, s_end): step
// s+NS-1 streams in while step s is computed, with one barrier per step.
// issue(s, k) enqueues the NL loads of step s into stage k (waves that copy
// nothing see their wait satisfied at once and rely on the barrier, which
// follows the copying waves' waits); compute(k) consumes stage k.  With
// three stages the wait for step s leaves the NL loads of step s+1 in
// flight, with four those of steps s+1 and s+2.
template <int NS, int NL, typename Issue, typename Compute>
__device__ __forceinline__ void key_stream(int s_begin, int s_end, Issue issue, Compute compute) {
  static_assert(NS >= 2 && NS <= 4, "two to four stages");
  for (int k = 0; k < NS - 1; ++k)
    if (s_begin + k < s_end) issue(s_begin + k, k);
  int cur = 0;
  for (int s = s_begin; s < s_end; ++s) {
    if constexpr (NS == 4) {
      if (s + 2 < s_end)
        wait_vmcnt<2 * NL>();  // steps s+1 and s+2 may still be in flight
      else if (s + 1 < s_end)
        wait_vmcnt<NL>();
      else
        wait_vmcnt<0>();
    } else if constexpr (NS == 3) {
      if (s + 1 < s_end)
        wait_vmcnt<NL>();  // only step s+1 may still be in flight
      else
        wait_vmcnt<0>();
    } else {
      wait_vmcnt<0>();
    }
    // After the barrier step s is visible to all waves and the stage read in
    // step s-1 is free; the empty assembly keeps the compiler from moving
    // memory accesses across it.
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if (s + NS - 1 < s_end) issue(s + NS - 1, cur == 0 ? NS - 1 : cur - 1);
    compute(cur);
    cur = cur == NS - 1 ? 0 : cur + 1;
  }
}

// The four-stage ring with one barrier per two steps: at the barrier before
// step s (s - s_begin even) steps s and s+1 have landed and every wave has
// finished steps s-2 and s-1, whose stages then take steps s+2 and s+3.
// Between barriers the waves of a workgroup may drift apart by a step.
template <int NL, typename Issue, typename Compute>
__device__ __forceinline__ void key_stream_pairs(int s_begin, int s_end, Issue issue, Compute compute) {
  for (int k = 0; k < 2; ++k)
    if (s_begin + k < s_end) issue(s_begin + k, k);
  int cur = 0;
  for (int s = s_begin; s < s_end; s += 2) {
    wait_vmcnt<0>();  // only steps s and s+1 are in flight
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    const int nx = cur ^ 2;  // the stages of steps s-2 and s-1
    if (s + 2 < s_end) issue(s + 2, nx);
    if (s + 3 < s_end) issue(s + 3, nx + 1);
    compute(cur);
    if (s + 1 < s_end) compute(cur + 1);
    cur = nx;
  }
}

// Stages for an eight-wave workgroup (one per CU) and a step of
// `stage_bytes` with `loads` copies per copying wave: four if they fit in
// 160 KiB of LDS and the vmcnt field (two steps in flight), else three,
// else two.
constexpr int wide_stages(int stage_bytes, int loads) {
  if (4 * stage_bytes <= 160 * 1024 && 2 * loads < 64) return 4;
  if (3 * stage_bytes <= 160 * 1024 && loads < 64) return 3;
  return 2;
}

// Stages for a step of `stage_bytes`: three when two workgroups per CU still
// fit in 160 KiB of LDS (and the per-step load count fits the vmcnt field),
// else two if that keeps two workgroups per CU (a second resident workgroup
// is worth more than the deeper prefetch: the D = 256 gradient runs 1.5x
// faster), else three, else two.
constexpr int ring_stages(int stage_bytes, int loads) {
  if (3 * stage_bytes <= 80 * 1024 && loads < 64) return 3;
  if (2 * stage_bytes <= 80 * 1024) return 2;
  return (3 * stage_bytes <= 160 * 1024 && loads < 64) ? 3 : 2;
}

__device__ __forceinline__ float max4(floatx4 a) {
  return fmaxf(fmaxf(a[0], a[1]), fmaxf(a[2], a[3]));
}
// Running maximum m folded with the four values of a, as a chain the compiler
// turns into two three-operand maxima (v_max3_f32) instead of four maxima.
__device__ __forceinline__ float max_into(float m, floatx4 a) {
  return fmaxf(fmaxf(fmaxf(fmaxf(m, a[0]), a[1]), a[2]), a[3]);
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

// Key-side tiles in LDS are 1-KiB chunks of 16 rows x 64 bytes, and an MFMA
// operand read (ds_read_b128) has lane (j, g) take the 16-byte column g of
// row j.  Stored plainly, rows 4 apart share LDS banks and every such read
// takes two passes; the direct copies therefore store column c of row r at
// column c ^ ((r >> 1) & 3) (lane l of a copy fetches the global column that
// belongs in LDS slot l), and readers index through lds_col.  Global copies
// keep the plain layout.
__device__ __forceinline__ int lds_col(int j, int g) { return g ^ ((j >> 1) & 3); }
__device__ __forceinline__ uint32_t dma_lane_offset(int lane) {
  return 16u * (uint32_t)((lane & ~3) | ((lane ^ (lane >> 3)) & 3));
}
template <int DP>
__device__ __forceinline__ void load_k_tile_lds(const uint4* base, int tile, int j, int g, uint4 (&kr)[DP]) {
  const int c = lds_col(j, g);
#pragma unroll
  for (int dc = 0; dc < DP; ++dc) kr[dc] = base[((tile * DP + dc) * 16 + j) * 4 + c];
}

// Per-wave prologue of the gradient kernel: the coarse row-bound check.
// sample_rt / sample_nh: the sampled keys (RT layout, half norms, coarse
// sample first).  Returns whether some query of the wave has its sampled row
// maximum of the log2 kernel value below kShiftBelow over the coarse sample;
// the gradient kernel then takes the exact row maxima (a clustered key set
// only costs it time).  The forward kernel reads the per-row levels of
// k_row_check instead.
template <typename T, int DP, int QT>
__device__ __forceinline__ bool needs_shift(const uint4* __restrict__ sample_rt,
                                            const float* __restrict__ sample_nh,
                                            const uint4 (&qreg)[QT][DP], const float (&bq)[QT],
                                            float tau2, int64_t q0, int64_t M, int j, int g) {
  float smax[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) smax[qt] = -__builtin_inff();
#pragma unroll
  for (int t = 0; t < kSampleCoarse / 16; ++t) {
    uint4 kr[DP];
    load_k_tile<DP>(sample_rt, t, j, g, kr);
    const floatx4 cin = *reinterpret_cast<const floatx4*>(sample_nh + 16 * t + 4 * g);
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) smax[qt] = max_into(smax[qt], score_tile<T, DP>(kr, qreg[qt], cin));
  }
  bool low = false;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const float L = fmaf(wave_max_over_g(smax[qt]), tau2, bq[qt]);
    low |= (q0 + 16 * qt + j < M) && (L < kShiftBelow);
  }
  return __any(low);
}

// Row-bound check, one flag per query row from the largest log2 kernel value L
// of row m over the sampled keys (sample_rt / sample_nh: RT layout and half
// norms, coarse sample first): shift[m] = 0 for L >= kShiftBelow (plain
// range), 1 for kExactBelow <= L < kShiftBelow (shifted kernel values), 2 below
// kExactBelow (the row needs its exact maximum as offset).  A wave takes 64
// rows; it checks the coarse sample first and scans the full one only when
// some row fails (a clustered key set can hide a row's own cluster from a
// small sample; the full-sample maximum is never below the coarse one, so rows
// passing the coarse check pass the full one).  The forward kernel reads these
// flags.
// Key row of sample position pos (coarse positions first, as k_sample
// stores them): rows floor(j N / kSampleRows).
__device__ __forceinline__ int64_t sample_row(int pos, int64_t n) {
  constexpr int kStride = kSampleRows / kSampleCoarse;
  int j;
  if (pos < kSampleCoarse) {
    j = kStride * pos;
  } else {
    const int q = pos - kSampleCoarse;
    j = (q / (kStride - 1)) * kStride + q % (kStride - 1) + 1;
  }
  return ((int64_t)j * n) / kSampleRows;
}

// GATHER: the sample is not copied; sample_rt / sample_nh are then the key
// set's own RT copy and half norms (nk > 0 keys), and the sampled rows are
// read from there (the same values k_sample would copy).
template <typename T, int DP, bool GATHER>
__global__ __launch_bounds__(kBlockThreads) void k_row_check(
    const uint4* __restrict__ qs, const float* __restrict__ nhq, const uint4* __restrict__ sample_rt,
    const float* __restrict__ sample_nh, float tau2, int64_t M, uint32_t* __restrict__ shift, Bz bz,
    int64_t nk) {
  constexpr int QT = 4;
  qs = zoff(qs, bz.ws);
  nhq = zoff(nhq, bz.ws);
  sample_rt = zoff(sample_rt, bz.ws);
  sample_nh = zoff(sample_nh, bz.ws);
  shift = zoff(shift, bz.ws);
  const int lane = threadIdx.x & (kWave - 1);
  const int j = lane & 15, g = lane >> 4;
  const int64_t q0 = ((int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave) * (16 * QT);
  uint4 qreg[QT][DP];
  float bq[QT], smax[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    load_k_tile<DP>(qs, q0 / 16 + qt, j, g, qreg[qt]);
    bq[qt] = tau2 * nhq[q0 + 16 * qt + j];
    smax[qt] = -__builtin_inff();
  }
  auto scan = [&](int t0, int t1) {
    for (int t = t0; t < t1; ++t) {
      uint4 kr[DP];
      floatx4 cin;
      if constexpr (GATHER) {
        const int64_t r = sample_row(16 * t + j, nk);
#pragma unroll
        for (int dc = 0; dc < DP; ++dc) kr[dc] = sample_rt[(((r >> 4) * DP + dc) * 16 + (r & 15)) * 4 + g];
#pragma unroll
        for (int u = 0; u < 4; ++u) cin[u] = sample_nh[sample_row(16 * t + 4 * g + u, nk)];
      } else {
        load_k_tile<DP>(sample_rt, t, j, g, kr);
        cin = *reinterpret_cast<const floatx4*>(sample_nh + 16 * t + 4 * g);
      }
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) smax[qt] = max_into(smax[qt], score_tile<T, DP>(kr, qreg[qt], cin));
    }
  };
  uint32_t level[QT];
  auto decide = [&]() {
    bool any = false;
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      const float L = fmaf(wave_max_over_g(smax[qt]), tau2, bq[qt]);
      const bool valid = q0 + 16 * qt + j < M;
      level[qt] = !valid || L >= kShiftBelow ? 0u : L >= kExactBelow ? 1u : 2u;
      any |= level[qt] != 0u;
    }
    return __any(any);
  };
  scan(0, kSampleCoarse / 16);
  if (decide()) {
    scan(kSampleCoarse / 16, kSampleRows / 16);
    decide();
  }
  if (g == 0)
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) shift[q0 + 16 * qt + j] = level[qt];
}

// The flags of k_row_check for the rows queried against a sample are stored
// right after that sample's half norms.
__device__ __forceinline__ const uint32_t* row_flags(const float* sample_nh) {
  return reinterpret_cast<const uint32_t*>(sample_nh + kSampleRows);
}

// The largest k_row_check level (0, 1, 2) of the wave's 16 QT query rows.
template <int QT>
__device__ __forceinline__ int wave_shift_level(const uint32_t* __restrict__ shift, int64_t q0, int j) {
  uint32_t f = 0;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) f = max(f, shift[q0 + 16 * qt + j]);
  return __any(f >= 2u) ? 2 : __any(f >= 1u) ? 1 : 0;
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
        smax[qt] = max_into(smax[qt], score_tile<T, DP>(kr, qreg[qt], cin));
    }
  }
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    off[qt] = fmaf(wave_max_over_g(smax[qt]), tau2, bq[qt]);
    if (!(off[qt] > -__builtin_inff())) off[qt] = 0.0f;  // empty key range
    bq[qt] -= off[qt];
  }
}

// acc + sum over the 8 fp16 products a_i b_i (v_dot2_f32_f16, fp32 accumulation).
__device__ __forceinline__ float dot2_acc(uint4 a, uint4 b, float acc) {
  acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(halfx2, a.x), __builtin_bit_cast(halfx2, b.x), acc, false);
  acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(halfx2, a.y), __builtin_bit_cast(halfx2, b.y), acc, false);
  acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(halfx2, a.z), __builtin_bit_cast(halfx2, b.z), acc, false);
  acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(halfx2, a.w), __builtin_bit_cast(halfx2, b.w), acc, false);
  return acc;
}

__device__ __forceinline__ uint4 pack_tile_pair(const float (&p)[2][4]) {
  uint4 b;
  b.x = pack_f16(p[0][0], p[0][1]);
  b.y = pack_f16(p[0][2], p[0][3]);
  b.z = pack_f16(p[1][0], p[1][1]);
  b.w = pack_f16(p[1][2], p[1][3]);
  return b;
}

// Whether the gradient kernel runs a step in three phases (all score MFMAs,
// then the w contractions and exponentials, then the contractions over keys,
// each LDS operand read as it is used): several channels at D > 64 where the
// pass then fits in 256 registers without spills in the key loop (checked
// per instance: D <= 128 with C <= 128, D <= 256 with C <= 32 or C > 64;
// D > 128 with C > 64 takes one query tile per wave).  Measured against the
// plain step for fp16 and bf16, M = N = 32768, forward and full gradient:
// D = 256, C = 128 10.76 -> 4.65 ms (the plain step with two query tiles
// reloaded 27 spilled values in every key step; 5.3 ms with one); the plain
// step stays faster at D = 256, C = 64 (3.80 against 4.04 ms) and at
// D = 128, C = 256 (4.54 against 5.02 ms).
constexpr bool dq_phased(int DP, int CW) {
  return CW > 0 && ((DP == 4 && CW <= 4) || (DP == 8 && (CW == 1 || CW >= 4)));
}

// Whether the gradient kernel takes its K^T operands from the streamed RT
// key tiles by transposing LDS reads instead of streaming a KS copy of the
// keys: fp16 points only (the RT tiles then hold exactly the fp16 values the
// contraction needs; a bf16 KS copy is converted to fp16), in the three-phase
// step.  The host planner uses the same rule to leave out the KS copy.
constexpr bool dq_transposed_keys(bool f16_points, int DP, int CW) {
  return f16_points && dq_phased(DP, CW);
}

// The K^T operand (A of the dQ contraction, 16 dimensions x 32 keys in the
// KS key order) of d-tile dt, read straight from the step's RT key tiles in
// LDS with two transposing reads (ds_read_b64_tr_b16: within each 16-lane
// group, lane i receives for r = 0..3 the 16-bit element i % 4 of the 8 bytes
// that lane 4r + i / 4 of the group addresses).  Lane 16g + 4r + c addresses
// key row 4g + r of key tile 0 (first read: k-slots 8g .. 8g+3 hold keys
// 4g .. 4g+3) and of key tile 1 (second read: keys 16 + 4g .. +3), dimensions
// 16 dt + 4c .. +3, through the XOR swizzle of the LDS columns.  The lane's
// byte offsets within a chunk for even and odd dt (their 16-byte columns
// differ by an XOR with 2) come from tr_lane; everything else is an
// immediate offset of the read (chunk dt / 2 of key tile 0, and DP chunks
// further for key tile 1).
struct TrLane {
  int even, odd;
};
__device__ __forceinline__ TrLane tr_lane(int lane) {
  const int g = lane >> 4, r = (lane >> 2) & 3, c = lane & 3;
  const int row = 4 * g + r;
  const int col = (c >> 1) ^ ((row >> 1) & 3);
  return {row * 64 + col * 16 + (c & 1) * 8, row * 64 + (col ^ 2) * 16 + (c & 1) * 8};
}

// The lane index formed by an opaque instruction pair: values derived from
// it inside a key step are formed again in every step instead of being kept
// live across the key loop (where, short of registers, the compiler would
// otherwise spill them and reload them from scratch memory in every step).
__device__ __forceinline__ int opaque_lane() {
  int ln;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(ln));
  return ln;
}

// LDS reads issued as assembly with immediate offsets, for operands that are
// read well ahead of their use: the compiler neither sinks such a read to its
// first use nor counts it in its own waits, so the reader waits explicitly
// (lgkm_fence) before that use.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
template <int OFF>
__device__ __forceinline__ u32x2 ds_read_tr_b64_asm(uint32_t addr) {
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "n"(OFF));
  return r;
}
template <int OFF>
__device__ __forceinline__ u32x4 ds_read_b128_asm(uint32_t addr) {
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "n"(OFF));
  return r;
}
// Wait until at most N LDS operations of the wave are outstanding (LDS reads
// complete in order, so every read issued before the N newest is done).  The
// operands pass through the statement, so their uses cannot move above it.
template <int N>
__device__ __forceinline__ void lgkm_fence(u32x2& a, u32x2& b) {
  asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(a), "+v"(b) : "n"(N));
}
template <int N>
__device__ __forceinline__ void lgkm_fence(u32x4& a) {
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(a) : "n"(N));
}

// f(integral_constant<int, I>) for I = B .. E-1, for code whose immediates
// depend on the index.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// Rows of `width` floats starting at `base` can take 16-byte stores (every
// row start 16-byte aligned).
__device__ __forceinline__ bool vec4_rows(const float* base, int width) {
  return (width % 4 == 0) && ((reinterpret_cast<uintptr_t>(base) & 15) == 0);
}

// Elements c0 .. c0+3 of one output row (c0 a multiple of 4) with one 16-byte
// store when v4, else element by element up to `width`.
__device__ __forceinline__ void store_row4(float* row, int c0, int width, bool v4, float a, float b,
                                           float c, float d) {
  if (v4) {
    if (c0 < width) *reinterpret_cast<float4*>(row + c0) = float4{a, b, c, d};
  } else {
    if (c0 < width) row[c0] = a;
    if (c0 + 1 < width) row[c0 + 1] = b;
    if (c0 + 2 < width) row[c0 + 2] = c;
    if (c0 + 3 < width) row[c0 + 3] = d;
  }
}

// ---------------------------------------------------------------- forward

// ONE (single channel, C = 1): the magnitude of v_n enters the exponent via the
// step scalars (log2 |v_n 2^e| added to the key bias, max |v 2^e| in
// [0.5, 1)) and V^T holds only the signs, so v contributes no fp16 rounding.
//
// BZ: a batch of problems on grid.z (operands at the strides of bz); the
// instance for one problem never reads bz.
template <typename T, int DP, int CT, int QT, bool ONE, bool BZ, int WPB>
__global__ __launch_bounds__(kWave * WPB) void k_fwd(
    const uint4* __restrict__ qs, const float* __restrict__ nhq, const uint4* __restrict__ samp_rt,
    const float* __restrict__ samp_nh, const uint4* __restrict__ ks, const float* __restrict__ scal,
    const uint4* __restrict__ vt, const uint32_t* __restrict__ vslot, float tau2, int64_t M, int C,
    int steps_total, int steps_per_split, float* __restrict__ out, int64_t part_stride, Bz bz) {
  if constexpr (BZ) {
    qs = zoff(qs, bz.ws);
    nhq = zoff(nhq, bz.ws);
    samp_rt = zoff(samp_rt, bz.ws);
    samp_nh = zoff(samp_nh, bz.ws);
    ks = zoff(ks, bz.ws);
    scal = zoff(scal, bz.ws);
    vt = zoff(vt, bz.ws);
    vslot = zoff(vslot, bz.ws);
    out = zoff(out, bz.out);
  }
  constexpr int KCH = 2 * DP;   // 1-KiB chunks of keys per step
  constexpr int NCH = KCH + CT; // + chunks of V^T
  constexpr int STAGE = NCH * 1024 + kScalarFloats * 4;
  // eight waves (one workgroup per CU, up to four stages): waves 0-3 copy
  // every chunk, waves 4-7 none (splitting the copies between the two groups
  // measured slower)
  constexpr bool WIDE = WPB == 2 * kWavesPerBlock;
  constexpr int NS = WIDE ? wide_stages(STAGE, NCH + 1) : ring_stages(STAGE, NCH + 1);
  __shared__ __attribute__((aligned(1024))) char lds[NS * STAGE];

  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t dlane = dma_lane_offset(lane);
  const int wave = threadIdx.x / kWave;
  const int j = lane & 15, g = lane >> 4;
  const int64_t q0 = ((int64_t)blockIdx.x * WPB + wave) * (16 * QT);
  const int s_begin = blockIdx.y * steps_per_split;
  const int s_end = min(steps_total, s_begin + steps_per_split);
  out += blockIdx.y * part_stride;

  const bool mine = g == wave;
  // buffer resources over this split's part of each key-side stream
  const uint32_t nsteps = (uint32_t)max(0, s_end - s_begin);
  const auto rk = make_rsrc(reinterpret_cast<const char*>(ks) + (int64_t)s_begin * KCH * 1024,
                            nsteps * KCH * 1024);
  const auto rv = make_rsrc(reinterpret_cast<const char*>(vt) + (int64_t)s_begin * CT * 1024,
                            nsteps * CT * 1024);
  const auto rsc = make_rsrc(scal + (int64_t)s_begin * kScalarFloats, nsteps * kScalarFloats * 4);
  const uint32_t lds0 = lds_address(lds);
  auto issue = [&](int s, int stage) {
    if (!mine) return;
    const uint32_t base = lds0 + stage * STAGE;
    const uint32_t ls = (uint32_t)(s - s_begin);
#pragma unroll
    for (int c = 0; c < KCH; ++c) dma_x4(rk, (ls * KCH + c) * 1024, base + c * 1024, dlane);
#pragma unroll
    for (int c = 0; c < CT; ++c) dma_x4(rv, (ls * CT + c) * 1024, base + (KCH + c) * 1024, dlane);
    // at D > 128 with one value tile the scalar row's lane offset is formed
    // again in every step (kept live across the loop it was spilled)
    dma_x1(rsc, ls * kScalarFloats * 4, base + NCH * 1024,
           4 * (DP == 8 && CT == 1 ? opaque_lane() : lane));
  };

  uint4 qreg[QT][DP];
  float bq[QT], off[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    load_k_tile<DP>(qs, q0 / 16 + qt, j, g, qreg[qt]);
    bq[qt] = tau2 * nhq[q0 + 16 * qt + j];
    off[qt] = 0.0f;
  }
  // range of the wave's kernel values: plain [0, 1], shifted by 2^kSigma, or
  // exact row maxima as offsets, from the per-row levels k_row_check wrote
  // (its coarse sample decides exactly as needs_shift would, so the forward
  // skips that check: 6 % of a 16384 x 16384, D = C = 128 pass)
  (void)samp_rt;
  const int level = wave_shift_level<QT>(row_flags(samp_nh), q0, j);
  if (level == 1) {
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      off[qt] = -kSigma;
      bq[qt] += kSigma;
    }
  }
  const bool shifted = level == 1;
  // level 2: the row maxima are tracked while streaming (running offset
  // off = exponent of the largest value seen so far, -inf before the first
  // step), instead of an exact pass over the keys first
  if (level == 2) {
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) off[qt] = -__builtin_inff();
  }

  settle(qreg);
  settle(bq);
  floatx4 O[QT][CT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) O[qt][ct] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

  // one key loop per range mode, so that each keeps the register budget of
  // a single loop body
  // Online offsets (level 2): before the exponentials of a query tile, the
  // wave checks that no exponent y (relative to the current offset) exceeds
  // kSigma; if one does, the offsets move up to the rows' largest exponent
  // so far (exact, across the four key groups of each row) and the row's
  // accumulators are rescaled by 2^(old - new).  Values are then at most
  // 2^kSigma (fp16 holds them) and the largest of a row within 2^-kSigma of
  // its maximum, as good as the exact offset for fp16 precision.  The check
  // triggers only when a row's maximum grows by more than kSigma, a few
  // times per row.
  auto online_check = [&](int qt, const floatx4 (&a)[2]) {
    float ymax = -__builtin_inff();
    const float be = bq[qt] - off[qt];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) ymax = fmaxf(ymax, fmaf(a[kt][r], tau2, be));
    if (__any(ymax > kSigma)) {
      float raw = -__builtin_inff();
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) raw = fmaxf(raw, fmaf(a[kt][r], tau2, bq[qt]));
      const float nw = fmaxf(off[qt], wave_max_over_g(raw));
      const float f = nw > off[qt] ? exp2f(off[qt] - nw) : 1.0f;
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int r = 0; r < 4; ++r) O[qt][ct][r] *= f;
      off[qt] = nw;
    }
    return bq[qt] - off[qt];
  };
  auto compute = [&](int stage, auto mode_c) {
    constexpr int MODE = decltype(mode_c)::value;
    constexpr bool SH = MODE == 1;
    const char* base = lds + stage * STAGE;
    const uint4* kb = reinterpret_cast<const uint4*>(base);
    const float* sc = reinterpret_cast<const float*>(base + NCH * 1024);
    floatx4 cin[2];
    uint4 kr[2][DP];
    // D > 128 with eight or more value tiles: all score MFMAs (each K read
    // feeding every query tile), then the exponentials, then the value
    // contractions, every LDS operand read as it is used.  Held for the step
    // the operands spilled at C = 128; M = N = 32768, D = 256: C = 128
    // 0.82 -> 0.76 ms, C = 256 1.51 -> 0.99 ms (two query tiles, which now
    // fit in 249 registers); C = 32 and 64 measured 1 - 3 % slower this way.
    // At every D with C > 128: two query tiles instead of one this way
    // (C = 256, M = N = 32768: D = 128 1.17 -> 0.78 ms, D = 64 1.53 -> 0.70,
    // D = 32 1.42 -> 0.66); at 64 < D <= 128 with C <= 128 (no spill, two
    // tiles either way) it measured 3 % slower.  D <= 64 with C = 65 - 128
    // fits four query tiles instead of two this way (C = 128: D = 64
    // 0.45 -> 0.38 ms, D = 32 0.45 -> 0.34 ms).
    constexpr bool LAZY = (DP == 8 && CT >= 8) || CT >= 16 || (DP <= 2 && CT == 8);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      cin[kt] = *reinterpret_cast<const floatx4*>(sc + 16 * kt + 4 * g);
      if constexpr (!LAZY) load_k_tile_lds<DP>(kb, kt, j, g, kr[kt]);
    }
    uint4 vr[CT];
    const uint4* vb = reinterpret_cast<const uint4*>(base + KCH * 1024);
    if constexpr (LAZY) {
      const int cl = lds_col(j, g);
      floatx4 acc[QT][2];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) acc[qt][kt] = cin[kt];
#pragma unroll
      for (int dc = 0; dc < DP; ++dc) {
        const uint4 a0 = kb[(dc * 16 + j) * 4 + cl];
        const uint4 a1 = kb[((DP + dc) * 16 + j) * 4 + cl];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          acc[qt][0] = mfma_qk<T>(a0, qreg[qt][dc], acc[qt][0]);
          acc[qt][1] = mfma_qk<T>(a1, qreg[qt][dc], acc[qt][1]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      uint4 b[QT];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        float p[2][4];
        if constexpr (MODE == 2) {
          const float be = online_check(qt, acc[qt]);
#pragma unroll
          for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int r = 0; r < 4; ++r) p[kt][r] = __builtin_amdgcn_exp2f(fmaf(acc[qt][kt][r], tau2, be));
        } else {
#pragma unroll
          for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float y = fmaf(acc[qt][kt][r], tau2, bq[qt]);
              p[kt][r] = SH ? exp2_shifted(y) : exp2_clamped(y);
            }
        }
        b[qt] = pack_tile_pair(p);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        const uint4 a = vb[(16 * ct + j) * 4 + cl];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) O[qt][ct] = mfma_f16(a, b[qt], O[qt][ct]);
      }
      return;
    }
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) vr[ct] = vb[(16 * ct + j) * 4 + lds_col(j, g)];
    if constexpr (DP == 1 && CT == 1 && MODE != 2) {
      // one 32-wide chunk and one value tile: all score MFMAs of the step,
      // then the exponentials, then the value contractions, kept apart by
      // scheduling barriers (3 % faster than tile by tile at D = 32 although
      // the accumulators cost one wave per SIMD)
      floatx4 acc[QT][2];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) acc[qt][kt] = score_tile<T, DP>(kr[kt], qreg[qt], cin[kt]);
      __builtin_amdgcn_sched_barrier(0);
      uint4 b[QT];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        float p[2][4];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float y = fmaf(acc[qt][kt][r], tau2, bq[qt]);
            p[kt][r] = SH ? exp2_shifted(y) : exp2_clamped(y);
          }
        b[qt] = pack_tile_pair(p);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) O[qt][0] = mfma_f16(vr[0], b[qt], O[qt][0]);
      return;
    }
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float p[2][4];
      if constexpr (MODE == 2) {
        floatx4 acc[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) acc[kt] = score_tile<T, DP>(kr[kt], qreg[qt], cin[kt]);
        const float be = online_check(qt, acc);
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) p[kt][r] = __builtin_amdgcn_exp2f(fmaf(acc[kt][r], tau2, be));
      } else {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          const floatx4 acc = score_tile<T, DP>(kr[kt], qreg[qt], cin[kt]);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float y = fmaf(acc[r], tau2, bq[qt]);
            p[kt][r] = SH ? exp2_shifted(y) : exp2_clamped(y);
          }
        }
      }
      const uint4 b = pack_tile_pair(p);
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) O[qt][ct] = mfma_f16(vr[ct], b, O[qt][ct]);
    }
  };
  auto stream = [&](auto cmp) {
    // eight waves and four stages: one barrier per two steps (not at
    // D = 256, where the two steps' code spills in the loop)
    if constexpr (WIDE && NS == 4 && DP <= 4)
      key_stream_pairs<NCH + 1>(s_begin, s_end, issue, cmp);
    else
      key_stream<NS, NCH + 1>(s_begin, s_end, issue, cmp);
  };
  if (level == 2)
    stream([&](int st) { compute(st, std::integral_constant<int, 2>{}); });
  else if (shifted)
    stream([&](int st) { compute(st, std::integral_constant<int, 1>{}); });
  else
    stream([&](int st) { compute(st, std::integral_constant<int, 0>{}); });

  const int ev = scale_exponent(*vslot) - (ONE ? 1 : 0);
  const bool v4 = vec4_rows(out, C);
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int64_t m = q0 + 16 * qt + j;
    if (m >= M) continue;
    const float f = exp2f(off[qt]);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
      store_row4(out + m * C, 16 * ct + 4 * g, C, v4, ldexpf(O[qt][ct][0] * f, -ev),
                 ldexpf(O[qt][ct][1] * f, -ev), ldexpf(O[qt][ct][2] * f, -ev), ldexpf(O[qt][ct][3] * f, -ev));
  }
}

// ---------------------------------------------------------------- gradient
//
// CW = 0 selects the single-channel form (C = 1): w_mn = g_m v_n.  |v_n|
// enters the exponent through the step scalars (as in k_fwd), sign(v_n) is
// folded into the KS copy of the keys, so P' = |Phi v_n| needs no multiply and
// no W contraction; the row sums take the signs from the step scalars, and
// g_m (exact, from the caller's array) multiplies the epilogue.  Row sums
// sum_n P use v_dot2_f32_f16 on the same fp16 values the dQ MFMA consumes.

//
// FCT > 0 fuses the forward sum into the same pass (the Sec. 3 observation
// that the query gradient is one more kernel sum over the same pairs): with
// C = 1 the forward output is the row sum sum_n Phi v_n the gradient already
// forms; with C > 1 the kernel values Phi (before the multiplication by w) go
// through one more MFMA against the FCT 16-row tiles of V^T streamed with
// the keys.  The forward result goes to out_s (M x C, split partials at
// part_stride_s), exactly as k_fwd would produce it.
// Two waves per SIMD (at most 256 VGPRs) wherever LDS allows two workgroups
// per CU: the large-D / large-C instances would otherwise take a few more
// registers and run one wave per SIMD, which costs far more than the spill
// of a few values outside the key loop.
//
// SV (with CW = 0): the SVGD direction of Sec. 3 in one pass.  Unit weights
// (P = Phi, no value magnitudes in the step scalars, no signs in the key
// copy), the FCT 16-row tiles of V^T hold the scores (C = D), and the
// epilogue writes out = sum_n Phi score_n - tau sum_n Phi (k_n - q_m) (the
// forward sum minus the query gradient with unit weights), or its split
// partial.
template <typename T, int DP, int CW, int QT, int FCT, bool BZ, int WPB, bool SV = false>
__global__ __launch_bounds__(kWave * WPB) __attribute__((amdgpu_waves_per_eu(2))) void k_dq(
    const uint4* __restrict__ qs, const float* __restrict__ nhq, const uint4* __restrict__ samp_rt,
    const float* __restrict__ samp_nh, const uint4* __restrict__ ks, const float* __restrict__ scal,
    const uint4* __restrict__ kt_ks, const uint32_t* __restrict__ kslot, const uint4* __restrict__ vs,
    const uint32_t* __restrict__ vslot, const uint4* __restrict__ gs,
    const uint32_t* __restrict__ gslot, const void* __restrict__ g1, int g1_dtype, float tau2,
    float tau, int64_t M, int D, int steps_total, int steps_per_split, float* __restrict__ out,
    int64_t part_stride, const uint4* __restrict__ vt, int C, float* __restrict__ out_s,
    int64_t part_stride_s, Bz bz) {
  if constexpr (BZ) {
    qs = zoff(qs, bz.ws);
    nhq = zoff(nhq, bz.ws);
    samp_rt = zoff(samp_rt, bz.ws);
    samp_nh = zoff(samp_nh, bz.ws);
    ks = zoff(ks, bz.ws);
    scal = zoff(scal, bz.ws);
    kt_ks = zoff(kt_ks, bz.ws);
    kslot = zoff(kslot, bz.ws);
    vs = zoff(vs, bz.ws);
    vslot = zoff(vslot, bz.ws);
    gs = zoff(gs, bz.ws);
    gslot = zoff(gslot, bz.ws);
    vt = zoff(vt, bz.ws);
    g1 = zoff(g1, bz.in2);
    out = zoff(out, bz.out);
    out_s = zoff(out_s, bz.out2);
  }
  constexpr int DT = 2 * DP;                // 16-row tiles of K^T (KS layout)
  constexpr int KCH = 2 * DP;               // chunks of K (RT) per step
  constexpr int VCH = 2 * CW;               // chunks of V (RT) per step
  // At D = 256 qreg (64) and dQ (128 registers) leave too few for the step's
  // operands when all of a tile's score operands are held across the query
  // tiles; in three phases with the operands read as they are used the pass
  // fits (and the fused forward costs a few per cent of the pass instead of
  // a pass of its own)
  constexpr bool PHASED = dq_phased(DP, CW);
  // the single-channel step and the SVGD mode at D > 128: every LDS operand
  // read as it is used.  Held for the whole step, the score operands and
  // the 16 K^T tiles (and the SVGD mode's 16 score tiles) spilled inside
  // the key loop: SVGD N = 16384, D = 256 1.84 -> 0.63 ms per call; the
  // single-channel gradient fits two query tiles in 244 registers this way
  // (D = 256, C = 1, M = 32768, N = 65536, forward and full gradient: two
  // tiles held 9.27 ms, one tile held 5.86 ms, two tiles read as used
  // 3.96 ms).  At 64 < D <= 128 the single-channel step read this way fits
  // four query tiles (two held: 4.39 ms, four read as used: 3.77 ms at
  // D = 128, C = 1, M = N = 65536); the SVGD mode there, where nothing
  // spills, measured 1 - 3 % slower this way.
  constexpr bool LAZY = (SV && DP == 8) || (CW == 0 && !SV && DP >= 4);
  // K^T operands read from the RT key tiles by transposing LDS reads (no KS
  // copy of the keys in the stream)
  constexpr bool TR = dq_transposed_keys(std::is_same<T, F16>::value, DP, CW);
  constexpr int TCH = TR ? 0 : DT;          // chunks of K^T (KS) per step: 32 DP rows x 64 B
  static_assert(!SV || CW == 0, "SVGD mode uses unit weights");
  constexpr int FCH = (CW > 0 || SV) ? FCT : 0;  // chunks of V^T (KS) per step, fused forward
  constexpr int NCH = KCH + VCH + TCH + FCH;
  constexpr int STAGE = NCH * 1024 + kScalarFloats * 4;
  // eight waves (one workgroup per CU): waves 0-3 copy every chunk, waves 4-7
  // none (splitting the copies between the two groups measured slower here)
  constexpr bool WIDE = WPB == 2 * kWavesPerBlock;
  constexpr int NS = WIDE ? wide_stages(STAGE, NCH + 1) : ring_stages(STAGE, NCH + 1);
  constexpr int GW = CW > 0 ? CW : 1;       // RT chunks of the upstream gradient
  __shared__ __attribute__((aligned(1024))) char lds[NS * STAGE];

  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t dlane = dma_lane_offset(lane);
  const int wave = threadIdx.x / kWave;
  const int j = lane & 15, g = lane >> 4;
  const int64_t q0 = ((int64_t)blockIdx.x * WPB + wave) * (16 * QT);
  const int s_begin = blockIdx.y * steps_per_split;
  const int s_end = min(steps_total, s_begin + steps_per_split);
  out += blockIdx.y * part_stride;
  if constexpr (FCT > 0) out_s += blockIdx.y * part_stride_s;

  const bool mine = g == wave;
  // buffer resources over this split's part of each key-side stream
  const uint32_t nsteps = (uint32_t)max(0, s_end - s_begin);
  const auto rk = make_rsrc(reinterpret_cast<const char*>(ks) + (int64_t)s_begin * KCH * 1024,
                            nsteps * KCH * 1024);
  const auto rv = make_rsrc(reinterpret_cast<const char*>(vs) + (int64_t)s_begin * VCH * 1024,
                            nsteps * VCH * 1024);
  const auto rt = make_rsrc(reinterpret_cast<const char*>(kt_ks) + (int64_t)s_begin * TCH * 1024,
                            nsteps * TCH * 1024);
  const auto rf = make_rsrc(reinterpret_cast<const char*>(vt) + (int64_t)s_begin * FCH * 1024,
                            nsteps * FCH * 1024);
  const auto rsc = make_rsrc(scal + (int64_t)s_begin * kScalarFloats, nsteps * kScalarFloats * 4);
  const uint32_t lds0 = lds_address(lds);
  auto issue = [&](int s, int stage) {
    if (!mine) return;
    const uint32_t base = lds0 + stage * STAGE;
    const uint32_t ls = (uint32_t)(s - s_begin);
#pragma unroll
    for (int c = 0; c < KCH; ++c) dma_x4(rk, (ls * KCH + c) * 1024, base + c * 1024, dlane);
#pragma unroll
    for (int c = 0; c < VCH; ++c) dma_x4(rv, (ls * VCH + c) * 1024, base + (KCH + c) * 1024, dlane);
#pragma unroll
    for (int c = 0; c < TCH; ++c)
      dma_x4(rt, (ls * TCH + c) * 1024, base + (KCH + VCH + c) * 1024, dlane);
#pragma unroll
    for (int c = 0; c < FCH; ++c)
      dma_x4(rf, (ls * FCH + c) * 1024, base + (KCH + VCH + TCH + c) * 1024, dlane);
    dma_x1(rsc, ls * kScalarFloats * 4, base + NCH * 1024, 4 * lane);
  };

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
  if constexpr (CW > 0) settle(greg);

  floatx4 dQ[QT][DT];
  float rs[QT];
  floatx4 O[QT][FCH > 0 ? FCH : 1];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    rs[qt] = 0.0f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) dQ[qt][dt] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int ct = 0; ct < FCH; ++ct) O[qt][ct] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
  }

  auto compute = [&](int stage) {
    const char* base = lds + stage * STAGE;
    const uint4* kb = reinterpret_cast<const uint4*>(base);
    const uint4* vb = reinterpret_cast<const uint4*>(base + KCH * 1024);
    const uint4* tb = reinterpret_cast<const uint4*>(base + (KCH + VCH) * 1024);
    const float* sc = reinterpret_cast<const float*>(base + NCH * 1024);
    // the lane's tile row and column group: in the SVGD mode formed again in
    // every step (kept live across the loop they pushed a spill into it)
    int jl = j, gl = g;
    if constexpr (SV) {
      const int ln = opaque_lane();
      jl = ln & 15;
      gl = ln >> 4;
    }
    floatx4 cin[2];
    uint4 kr[2][DP];
    uint4 vr[2][GW];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      cin[kt] = *reinterpret_cast<const floatx4*>(sc + 16 * kt + 4 * gl);
      if constexpr (!PHASED && !LAZY) load_k_tile_lds<DP>(kb, kt, jl, gl, kr[kt]);
      if constexpr (CW > 0) load_k_tile_lds<GW>(vb, kt, jl, gl, vr[kt]);
    }
    // per key slot of this lane's B operand: sign(v_n) (single channel) or 1
    const uint4 sg = (CW > 0 || SV) ? uint4{0x3C003C00u, 0x3C003C00u, 0x3C003C00u, 0x3C003C00u}
                                    : *reinterpret_cast<const uint4*>(sc + 32 + 4 * gl);
    const uint4* fb = reinterpret_cast<const uint4*>(base + (KCH + VCH + TCH) * 1024);
    if constexpr (PHASED) {
      // all score MFMAs (A operands read chunk by chunk, each feeding every
      // query tile), then the w contractions, exponentials and products, then
      // the contractions over keys, their A operands read two d-tiles ahead
      floatx4 acc[QT][2];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) acc[qt][kt] = cin[kt];
      const int col = lds_col(j, g);
#pragma unroll
      for (int dc = 0; dc < DP; ++dc) {
        const uint4 a0 = kb[(dc * 16 + j) * 4 + col];
        const uint4 a1 = kb[((DP + dc) * 16 + j) * 4 + col];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          acc[qt][0] = mfma_qk<T>(a0, qreg[qt][dc], acc[qt][0]);
          acc[qt][1] = mfma_qk<T>(a1, qreg[qt][dc], acc[qt][1]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      uint4 b[QT], bphi[QT];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        float p[2][4], phi[2][4];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          floatx4 w = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int cw = 0; cw < CW; ++cw) w = mfma_f16(vr[kt][cw], greg[qt][cw], w);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            phi[kt][r] = exp2_clamped(fmaf(acc[qt][kt][r], tau2, bq[qt]));
            p[kt][r] = phi[kt][r] * w[r];
          }
        }
        bphi[qt] = pack_tile_pair(phi);
        b[qt] = pack_tile_pair(p);
      }
      __builtin_amdgcn_sched_barrier(0);
      // the lane's transposing-read offsets, formed again in every step (kept
      // live across the loop they would cost registers)
      TrLane trl{0, 0};
      if constexpr (TR) {
        trl = tr_lane(opaque_lane());
        // the V^T tiles, then the K^T operands two d-tiles ahead of their
        // MFMAs (left to itself the compiler issued each pair of transposing
        // reads just before its MFMAs and waited for it)
        const uint32_t kb0 = lds_address(base);
        const uint32_t ae = kb0 + trl.even, ao = kb0 + trl.odd;
        const uint32_t af = kb0 + (KCH + VCH) * 1024 + (j * 4 + col) * 16;
        u32x4 f[FCH > 0 ? FCH : 1];
        u32x2 x0[DT], x1[DT];
        static_for<0, FCH>([&](auto ic) {
          constexpr int ct = decltype(ic)::value;
          f[ct] = ds_read_b128_asm<ct * 1024>(af);
        });
        auto rd = [&](auto ic) {
          constexpr int dt = decltype(ic)::value;
          const uint32_t a = (dt & 1) ? ao : ae;
          x0[dt] = ds_read_tr_b64_asm<(dt >> 1) * 1024>(a);
          x1[dt] = ds_read_tr_b64_asm<(dt >> 1) * 1024 + DP * 1024>(a);
        };
        rd(std::integral_constant<int, 0>{});
        if constexpr (DT > 1) rd(std::integral_constant<int, 1>{});
        static_for<0, FCH>([&](auto ic) {
          constexpr int ct = decltype(ic)::value;
          lgkm_fence<FCH - 1 - ct + 2 * (DT > 1 ? 2 : 1)>(f[ct]);
          const uint4 a = __builtin_bit_cast(uint4, f[ct]);
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) O[qt][ct] = mfma_f16(a, bphi[qt], O[qt][ct]);
        });
        static_for<0, DT>([&](auto ic) {
          constexpr int dt = decltype(ic)::value;
          if constexpr (dt + 2 < DT) rd(std::integral_constant<int, dt + 2>{});
          lgkm_fence<dt + 2 < DT ? 4 : dt + 1 < DT ? 2 : 0>(x0[dt], x1[dt]);
          const uint4 a = uint4{x0[dt].x, x0[dt].y, x1[dt].x, x1[dt].y};
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) dQ[qt][dt] = mfma_f16(a, b[qt], dQ[qt][dt]);
        });
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) rs[qt] = dot2_acc(b[qt], sg, rs[qt]);
        return;
      }
      // bf16 points: the V^T tiles, then the K^T operands from the KS copy,
      // also two d-tiles ahead of their MFMAs
      const uint32_t lo = lds_address(base) + (j * 4 + col) * 16;  // the lane's operand column
      u32x4 f[FCH > 0 ? FCH : 1], x[DT];
      static_for<0, FCH>([&](auto ic) {
        constexpr int ct = decltype(ic)::value;
        f[ct] = ds_read_b128_asm<(KCH + VCH + TCH + ct) * 1024>(lo);
      });
      auto rd = [&](auto ic) {
        constexpr int dt = decltype(ic)::value;
        x[dt] = ds_read_b128_asm<(KCH + VCH + dt) * 1024>(lo);
      };
      constexpr int LT = DT > 1 ? 2 : 1;
      static_for<0, LT>(rd);
      static_for<0, FCH>([&](auto ic) {
        constexpr int ct = decltype(ic)::value;
        lgkm_fence<FCH - 1 - ct + LT>(f[ct]);
        const uint4 a = __builtin_bit_cast(uint4, f[ct]);
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) O[qt][ct] = mfma_f16(a, bphi[qt], O[qt][ct]);
      });
      static_for<0, DT>([&](auto ic) {
        constexpr int dt = decltype(ic)::value;
        if constexpr (dt + LT < DT) rd(std::integral_constant<int, dt + LT>{});
        lgkm_fence<dt + LT < DT ? LT : DT - 1 - dt>(x[dt]);
        const uint4 a = __builtin_bit_cast(uint4, x[dt]);
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) dQ[qt][dt] = mfma_f16(a, b[qt], dQ[qt][dt]);
      });
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) rs[qt] = dot2_acc(b[qt], sg, rs[qt]);
      return;
    }
    if constexpr (LAZY) {
      const int cl = lds_col(jl, gl);
      floatx4 acc[QT][2];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) acc[qt][kt] = cin[kt];
#pragma unroll
      for (int dc = 0; dc < DP; ++dc) {
        const uint4 a0 = kb[(dc * 16 + jl) * 4 + cl];
        const uint4 a1 = kb[((DP + dc) * 16 + jl) * 4 + cl];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          acc[qt][0] = mfma_qk<T>(a0, qreg[qt][dc], acc[qt][0]);
          acc[qt][1] = mfma_qk<T>(a1, qreg[qt][dc], acc[qt][1]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      uint4 b[QT];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        float p[2][4];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) p[kt][r] = exp2_clamped(fmaf(acc[qt][kt][r], tau2, bq[qt]));
        b[qt] = pack_tile_pair(p);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const uint4 a = tb[(16 * dt + jl) * 4 + cl];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) dQ[qt][dt] = mfma_f16(a, b[qt], dQ[qt][dt]);
        if ((dt & 3) == 3) __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int ct = 0; ct < FCH; ++ct) {
        const uint4 a = fb[(16 * ct + jl) * 4 + cl];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) O[qt][ct] = mfma_f16(a, b[qt], O[qt][ct]);
        if ((ct & 3) == 3) __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) rs[qt] = dot2_acc(b[qt], sg, rs[qt]);
      return;
    }
    uint4 ktr[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) ktr[dt] = tb[(16 * dt + jl) * 4 + lds_col(jl, gl)];
    uint4 vtr[FCH > 0 ? FCH : 1];
#pragma unroll
    for (int ct = 0; ct < FCH; ++ct) vtr[ct] = fb[(16 * ct + jl) * 4 + lds_col(jl, gl)];
    if constexpr (CW == 0) {
      // single channel: the score MFMAs of all query tiles, then their
      // exponentials, then the contractions over keys, kept apart by
      // scheduling barriers (2 % faster than tile by tile).  The row-sum dot2
      // instructions go with the contractions for D > 32 (there they cost
      // nothing) and with the exponentials for D <= 32 (interleaved with the
      // few contraction MFMAs of a 32-wide step they cost 14 % of the pass,
      // in the exponential block 8 %)
      floatx4 acc[QT][2];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) acc[qt][kt] = score_tile<T, DP>(kr[kt], qreg[qt], cin[kt]);
      __builtin_amdgcn_sched_barrier(0);
      uint4 b[QT];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        float p[2][4];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) p[kt][r] = exp2_clamped(fmaf(acc[qt][kt][r], tau2, bq[qt]));
        b[qt] = pack_tile_pair(p);
        if constexpr (DP == 1) rs[qt] = dot2_acc(b[qt], sg, rs[qt]);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) dQ[qt][dt] = mfma_f16(ktr[dt], b[qt], dQ[qt][dt]);
        if constexpr (SV) {
#pragma unroll
          for (int ct = 0; ct < FCH; ++ct) O[qt][ct] = mfma_f16(vtr[ct], b[qt], O[qt][ct]);
        }
        if constexpr (DP > 1) rs[qt] = dot2_acc(b[qt], sg, rs[qt]);
      }
      return;
    }
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float p[2][4], phi[2][4];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const floatx4 acc = score_tile<T, DP>(kr[kt], qreg[qt], cin[kt]);
        if constexpr (CW > 0) {
          floatx4 w = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int cw = 0; cw < CW; ++cw) w = mfma_f16(vr[kt][cw], greg[qt][cw], w);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            phi[kt][r] = exp2_clamped(fmaf(acc[r], tau2, bq[qt]));
            p[kt][r] = phi[kt][r] * w[r];
          }
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) p[kt][r] = exp2_clamped(fmaf(acc[r], tau2, bq[qt]));
        }
      }
      if constexpr (FCH > 0) {
        const uint4 bphi = pack_tile_pair(phi);
#pragma unroll
        for (int ct = 0; ct < FCH; ++ct) O[qt][ct] = mfma_f16(vtr[ct], bphi, O[qt][ct]);
      }
      const uint4 b = pack_tile_pair(p);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) dQ[qt][dt] = mfma_f16(ktr[dt], b, dQ[qt][dt]);
      rs[qt] = dot2_acc(b, sg, rs[qt]);
    }
  };
  // three-phase eight-wave passes with four stages: one barrier per two
  // steps (1 % faster at D = 256, the same L2 hit rate)
  if constexpr (PHASED && WIDE && NS == 4)
    key_stream_pairs<NCH + 1>(s_begin, s_end, issue, compute);
  else
    key_stream<NS, NCH + 1>(s_begin, s_end, issue, compute);

  const int ek = kslot ? point_scale_exponent(*kslot) : 0;
  const uint16_t* q16 = reinterpret_cast<const uint16_t*>(qs);
  // rs holds this lane's 8-key partial sums; add the other three key groups
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    rs[qt] += __shfl_xor(rs[qt], 16, kWave);
    rs[qt] += __shfl_xor(rs[qt], 32, kWave);
  }
  if constexpr (SV) {
    // SVGD direction: the forward sum over the scores (scaled by 2^ev in their
    // copy) minus the unit-weight query gradient tau (sum_n Phi k_n - q_m sum_n Phi)
    const int ev = scale_exponent(*vslot);
    const bool v4d = vec4_rows(out, D);
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      const int64_t m = q0 + 16 * qt + j;
      if (m >= M) continue;
      const float fo = exp2f(off[qt]);
      const float fw = tau * fo;
      const float rm = rs[qt];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int d0 = 16 * dt + 4 * g;
        if (d0 >= D) continue;
        const uint2 qq = *reinterpret_cast<const uint2*>(q16 + rt_index(m, d0, 32 * DP));
        const float qv[4] = {T::to_float((uint16_t)qq.x), T::to_float((uint16_t)(qq.x >> 16)),
                             T::to_float((uint16_t)qq.y), T::to_float((uint16_t)(qq.y >> 16))};
        float o[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float fwd = dt < FCH ? ldexpf(O[qt][dt < FCH ? dt : 0][r], -ev) * fo : 0.0f;
          o[r] = fwd - (ldexpf(dQ[qt][dt][r], -ek) - qv[r] * rm) * fw;
        }
        store_row4(out + m * D, d0, D, v4d, o[0], o[1], o[2], o[3]);
      }
    }
    return;
  }
  if constexpr (FCT > 0) {
    // fused forward output: single channel from the signed row sums (values
    // scaled by 2^(ev-1)), several channels from the extra MFMA (2^ev)
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      const int64_t m = q0 + 16 * qt + j;
      if (m >= M) continue;
      const float f = exp2f(off[qt]);
      if constexpr (CW == 0) {
        if (g == 0) out_s[m] = ldexpf(rs[qt] * f, 1 - scale_exponent(*vslot));
      } else {
        const int ev = scale_exponent(*vslot);
        const bool v4 = vec4_rows(out_s, C);
#pragma unroll
        for (int ct = 0; ct < FCH; ++ct)
          store_row4(out_s + m * C, 16 * ct + 4 * g, C, v4, ldexpf(O[qt][ct][0] * f, -ev),
                     ldexpf(O[qt][ct][1] * f, -ev), ldexpf(O[qt][ct][2] * f, -ev),
                     ldexpf(O[qt][ct][3] * f, -ev));
      }
    }
  }
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int64_t m = q0 + 16 * qt + j;
    if (m >= M) continue;
    float f = tau * exp2f(off[qt]);
    int e;
    if constexpr (CW > 0) {
      e = -scale_exponent(*vslot) - scale_exponent(*gslot);
    } else {
      // single channel: w = g_m v_n with v_n 2^(ev-1) in the kernel values
      e = 1 - scale_exponent(*vslot);
      f *= load_any(g1, m, g1_dtype);
    }
    const float rm = rs[qt];
    const bool v4d = vec4_rows(out, D);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int d0 = 16 * dt + 4 * g;
      if (d0 >= D) continue;
      // q_m,d0 .. d0+3 from the RT copy: four consecutive halves (8 bytes)
      const uint2 qq = *reinterpret_cast<const uint2*>(q16 + rt_index(m, d0, 32 * DP));
      const float qv[4] = {T::to_float((uint16_t)qq.x), T::to_float((uint16_t)(qq.x >> 16)),
                           T::to_float((uint16_t)qq.y), T::to_float((uint16_t)(qq.y >> 16))};
      float o[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) o[r] = ldexpf((ldexpf(dQ[qt][dt][r], -ek) - qv[r] * rm) * f, e);
      store_row4(out + m * D, d0, D, v4d, o[0], o[1], o[2], o[3]);
    }
  }
}

}  // namespace gs
