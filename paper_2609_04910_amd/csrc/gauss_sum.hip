// gauss_sum.hip -- C ABI of the gfx950 Gauss-sum library: validation, launch
// planning, workspace carving and kernel dispatch.  Declarations and the
// contract of every entry point are in include/gauss_sum.h.
#include "../../include/gauss_sum.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>

#include "gs_common.h"
#include "gs_kernels.h"
#include "gs_prep.h"
#include "gs_f32.h"

namespace gs {
namespace {

constexpr size_t kAlign = 256;
constexpr int kMinStepsPerSplit = 4;     // 128 keys
constexpr int kSplitOverheadSteps = 8;   // per-workgroup fixed cost (prologue, epilogue), in key steps
// Most key steps one split may cover: every key-side stream moves at most
// 16 KiB per step, and a split's part of a stream is addressed through one
// buffer resource (32-bit byte count) with 32-bit step offsets.
constexpr int kMaxStepsPerSplit = 1 << 17;
// Largest M and N accepted: the main kernels launch one workgroup of 256
// threads per 64 QT rows, and a grid's x extent in threads must stay below
// 2^32 (QT >= 1).
constexpr int64_t kMaxRows = int64_t(1) << 30;
constexpr int kDefaultSlots = 512;       // resident workgroups assumed when no device can be queried

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
inline int64_t ceil_div(int64_t x, int64_t m) { return (x + m - 1) / m; }

inline int pow2_chunks(int64_t width, int unit, int max_chunks) {
  int c = 1;
  while (c * unit < width && c < max_chunks) c *= 2;
  return c;
}

// Shape parameters of the tiles (see gs_common.h for the layouts).
struct Dims {
  int DP;  // 32-wide chunks of D (1, 2, 4, 8): RT width W = 32 DP, KS rows = 32 DP
  int CW;  // 32-wide chunks of C (1, 2, 4, 8): RT width of values = 32 CW
  int CT;  // 16-row tiles of C (1, 2, 4, 8, 16): KS rows of values = 16 CT
  int W() const { return 32 * DP; }
  int Wv() const { return 32 * CW; }
  int Rv() const { return 16 * CT; }
};

inline Dims dims_of(int64_t D, int64_t C) {
  Dims d;
  d.DP = pow2_chunks(D, 32, 8);
  d.CW = pow2_chunks(C, 32, 8);
  d.CT = pow2_chunks(C, 16, 16);
  return d;
}

// Query tiles per wave.  Forward: 8 for D <= 64 with C <= 32 (the per-step
// barrier, loads and K-tile reads then cover twice the pairs: D = 64, C = 1
// 0.76 -> 0.71 ms), else the largest of 4, 2, 1 whose kernel (as compiled
// for gfx950) keeps the register count at or below 256 per lane (two waves
// per SIMD).  Gradient: for D > 64 two tiles even where that needs the
// occupancy hint on k_dq or (D = 256, whose LDS ring allows one workgroup per
// CU anyway) one wave per SIMD: a K tile read from LDS then feeds two MFMAs,
// and a single tile per wave is bound by LDS bandwidth; D > 128 with
// C > 64 keeps one tile (two spilled 27 values inside the key loop; the
// single channel keeps two with its operands read as they are used; at
// 64 < D <= 128 the single channel, read that way, takes four).  The
// D > 128 forward with C = 65 - 128 keeps two (one spilled value; 0.83 ms
// against 1.17 ms with one tile at M = N = 32768).
// (C > 128: two tiles at every D, and D <= 64 with C = 65 - 128: four,
// the operands read as they are used.)
constexpr int fwd_qt(int DP, int CT) {
  return CT >= 16 ? 2 : CT == 8 ? (DP <= 2 ? 4 : 2) : (DP == 8 && CT > 1) ? 2 : (DP <= 2 && CT <= 2) ? 8 : 4;
}
// Every workgroup's rows lie inside the padded row range.
static_assert(kRowPad % (kBlockThreads / 4 * 8) == 0 && kRowPad % 256 == 0, "row padding vs. query tiles");


// Waves per workgroup of the gradient and forward kernels: eight for D > 64,
// where a key step's operands take 12 to 34 KiB of LDS -- one workgroup per
// CU then holds a deeper ring (three or four stages) that feeds twice the
// queries of a four-wave workgroup, half the copies per pair (D = 256,
// C = 16: dq pass 378 -> 265 ms, forward 124 -> 107 ms; D = C = 128: 5 %);
// four for D <= 64 (no gain there).
constexpr int dq_wpb(int DP) { return DP >= 4 ? 2 * kWavesPerBlock : kWavesPerBlock; }
constexpr int fwd_wpb(int DP) { return DP >= 4 ? 2 * kWavesPerBlock : kWavesPerBlock; }

constexpr int dq_qt(int DP, int CW) {
  return DP >= 4 ? (DP == 8 && CW >= 4 ? 1 : DP == 4 && CW == 0 ? 4 : 2) : DP == 2 ? (CW == 0 ? 4 : 2) : CW >= 4 ? 2 : 4;
}

// Every workgroup of a main kernel covers at most kRowPad query rows (the
// padded row count of every operand copy is a multiple of kRowPad).
constexpr bool tiles_within_padding() {
  const int dps[4] = {1, 2, 4, 8}, cts[6] = {0, 1, 2, 4, 8, 16}, cws[5] = {0, 1, 2, 4, 8};
  for (int dp : dps) {
    for (int ct : cts)
      if (16 * fwd_qt(dp, ct) * fwd_wpb(dp) > kRowPad) return false;
    for (int cw : cws)
      if (16 * dq_qt(dp, cw) * dq_wpb(dp) > kRowPad) return false;
  }
  return true;
}
static_assert(tiles_within_padding(), "query rows of a workgroup exceed the row padding");

// ------------------------------------------------------------ dispatch tables

using FwdFn = void (*)(dim3, hipStream_t, const uint4*, const float*, const uint4*, const float*,
                       const uint4*, const float*, const uint4*, const uint32_t*, float, int64_t, int,
                       int, int, float*, int64_t, const Bz&);

// grid.z > 1: the batched instance (problem blockIdx.z at the strides of bz).
template <typename T, int DP, int CT, bool ONE>
void launch_fwd(dim3 grid, hipStream_t st, const uint4* qs, const float* nhq, const uint4* srt,
                const float* snh, const uint4* ks, const float* scal, const uint4* vt,
                const uint32_t* vslot, float tau2, int64_t M, int C, int steps, int sps, float* out,
                int64_t pstride, const Bz& bz) {
  if (grid.z > 1)
    hipLaunchKernelGGL((k_fwd<T, DP, CT, fwd_qt(DP, CT), ONE, true, fwd_wpb(DP)>), grid, dim3(kWave * fwd_wpb(DP)), 0, st,
                       qs, nhq, srt, snh, ks, scal, vt, vslot, tau2, M, C, steps, sps, out, pstride, bz);
  else
    hipLaunchKernelGGL((k_fwd<T, DP, CT, fwd_qt(DP, CT), ONE, false, fwd_wpb(DP)>), grid, dim3(kWave * fwd_wpb(DP)), 0, st,
                       qs, nhq, srt, snh, ks, scal, vt, vslot, tau2, M, C, steps, sps, out, pstride, bz);
}

// A launcher and the kernel it launches (for occupancy queries).
struct FwdK {
  FwdFn launch = nullptr;
  const void* kernel = nullptr;
};

template <typename T, int DP, int CT, bool ONE>
FwdK fwd_k() {
  return {&launch_fwd<T, DP, CT, ONE>,
          reinterpret_cast<const void*>(&k_fwd<T, DP, CT, fwd_qt(DP, CT), ONE, false, fwd_wpb(DP)>)};
}

// CT = 0 selects the single-channel form (one 16-row tile of signs).
template <typename T, int DP>
FwdK fwd_by_ct(int CT) {
  switch (CT) {
    case 0: return fwd_k<T, DP, 1, true>();
    case 1: return fwd_k<T, DP, 1, false>();
    case 2: return fwd_k<T, DP, 2, false>();
    case 4: return fwd_k<T, DP, 4, false>();
    case 8: return fwd_k<T, DP, 8, false>();
    case 16: return fwd_k<T, DP, 16, false>();
  }
  return {};
}

template <typename T>
FwdK fwd_fn(int DP, int CT) {
  switch (DP) {
    case 1: return fwd_by_ct<T, 1>(CT);
    case 2: return fwd_by_ct<T, 2>(CT);
    case 4: return fwd_by_ct<T, 4>(CT);
    case 8: return fwd_by_ct<T, 8>(CT);
  }
  return {};
}

using DqFn = void (*)(dim3, hipStream_t, const uint4*, const float*, const uint4*, const float*,
                      const uint4*, const float*, const uint4*, const uint32_t*, const uint4*,
                      const uint32_t*, const uint4*, const uint32_t*, const void*, int, float, float,
                      int64_t, int, int, int, float*, int64_t, const uint4*, int, float*, int64_t,
                      const Bz&);

template <typename T, int DP, int CW, int FCT>
void launch_dq(dim3 grid, hipStream_t st, const uint4* qs, const float* nhq, const uint4* srt,
               const float* snh, const uint4* ks, const float* scal, const uint4* kt,
               const uint32_t* kslot, const uint4* vs, const uint32_t* vslot, const uint4* gsr,
               const uint32_t* gslot, const void* g1, int g1_dtype, float tau2, float tau, int64_t M,
               int D, int steps, int sps, float* out, int64_t pstride, const uint4* vt, int C,
               float* out_s, int64_t pstride_s, const Bz& bz) {
  if (grid.z > 1)
    hipLaunchKernelGGL((k_dq<T, DP, CW, dq_qt(DP, CW), FCT, true, dq_wpb(DP)>), grid, dim3(kWave * dq_wpb(DP)), 0, st, qs,
                       nhq, srt, snh, ks, scal, kt, kslot, vs, vslot, gsr, gslot, g1, g1_dtype, tau2, tau,
                       M, D, steps, sps, out, pstride, vt, C, out_s, pstride_s, bz);
  else
    hipLaunchKernelGGL((k_dq<T, DP, CW, dq_qt(DP, CW), FCT, false, dq_wpb(DP)>), grid, dim3(kWave * dq_wpb(DP)), 0, st, qs,
                       nhq, srt, snh, ks, scal, kt, kslot, vs, vslot, gsr, gslot, g1, g1_dtype, tau2, tau,
                       M, D, steps, sps, out, pstride, vt, C, out_s, pstride_s, bz);
}

struct DqK {
  DqFn launch = nullptr;
  const void* kernel = nullptr;
};

template <typename T, int DP, int CW, int FCT>
DqK dq_k() {
  return {&launch_dq<T, DP, CW, FCT>,
          reinterpret_cast<const void*>(&k_dq<T, DP, CW, dq_qt(DP, CW), FCT, false, dq_wpb(DP)>)};
}

// fused: also produce the forward sum (one 16-row tile: C = 1 through the
// row sums, 1 < C <= kFuseMaxC through one V^T tile); wider values are never
// fused (see kFuseMaxC), so those instances do not exist.
template <typename T, int DP, int CW>
DqK dq_pick(bool fused) {
  return fused ? dq_k<T, DP, CW, 1>() : dq_k<T, DP, CW, 0>();
}

template <typename T, int DP>
DqK dq_by_cw(int CW, int CT, bool fused) {
  if (fused && CT > 1) return {};
  switch (CW) {
    case 0: return dq_pick<T, DP, 0>(fused);
    case 1: return dq_pick<T, DP, 1>(fused);
    case 2: return fused ? DqK{} : dq_k<T, DP, 2, 0>();
    case 4: return fused ? DqK{} : dq_k<T, DP, 4, 0>();
    case 8: return fused ? DqK{} : dq_k<T, DP, 8, 0>();
  }
  return {};
}

template <typename T>
DqK dq_fn(int DP, int CW, int CT, bool fused) {
  switch (DP) {
    case 1: return dq_by_cw<T, 1>(CW, CT, fused);
    case 2: return dq_by_cw<T, 2>(CW, CT, fused);
    case 4: return dq_by_cw<T, 4>(CW, CT, fused);
    case 8: return dq_by_cw<T, 8>(CW, CT, fused);
  }
  return {};
}

// SVGD direction in one pass (k_dq with SV = true, C = D): query tiles per
// wave so that the query operands, dQ and the forward accumulators stay
// within the register budget.
constexpr int sv_qt(int DP) { return DP == 8 ? 1 : DP == 4 ? 2 : 4; }

using SvFn = void (*)(dim3, hipStream_t, const uint4*, const float*, const uint4*, const float*,
                      const uint4*, const float*, const uint4*, const uint32_t*, const uint32_t*, float,
                      float, int64_t, int, int, int, float*, int64_t, const uint4*);

template <typename T, int DP, int CT>
void launch_sv(dim3 grid, hipStream_t st, const uint4* xs, const float* nh, const uint4* srt,
               const float* snh, const uint4* ks, const float* scal, const uint4* kt, const uint32_t* kslot,
               const uint32_t* vslot, float tau2, float tau, int64_t M, int D, int steps, int sps, float* out,
               int64_t pstride, const uint4* vt) {
  hipLaunchKernelGGL((k_dq<T, DP, 0, sv_qt(DP), CT, false, dq_wpb(DP), true>), grid, dim3(kWave * dq_wpb(DP)), 0,
                     st, xs, nh, srt, snh, ks, scal, kt, kslot, nullptr, vslot, nullptr, nullptr, nullptr, 0,
                     tau2, tau, M, D, steps, sps, out, pstride, vt, D, nullptr, 0, Bz{});
}

struct SvK {
  SvFn launch = nullptr;
  const void* kernel = nullptr;
};

template <typename T, int DP, int CT>
SvK sv_k() {
  return {&launch_sv<T, DP, CT>,
          reinterpret_cast<const void*>(&k_dq<T, DP, 0, sv_qt(DP), CT, false, dq_wpb(DP), true>)};
}

// The instance for D (CT = 16-row tiles of C = D).
template <typename T>
SvK sv_fn(int DP, int CT) {
  if (DP == 1 && CT == 1) return sv_k<T, 1, 1>();
  if (DP == 1 && CT == 2) return sv_k<T, 1, 2>();
  if (DP == 2 && CT == 4) return sv_k<T, 2, 4>();
  if (DP == 4 && CT == 8) return sv_k<T, 4, 8>();
  if (DP == 8 && CT == 16) return sv_k<T, 8, 16>();
  return {};
}

// fp32 tier (fp32 points, C = 1, forward): the kernel for D chunks DP.
const void* f32_kernel(int DP) {
  switch (DP) {
    case 1: return reinterpret_cast<const void*>(&k_fwd32<1>);
    case 2: return reinterpret_cast<const void*>(&k_fwd32<2>);
    case 4: return reinterpret_cast<const void*>(&k_fwd32<4>);
    case 8: return reinterpret_cast<const void*>(&k_fwd32<8>);
  }
  return nullptr;
}

// fp32 tier, several channels: channel tiles per launch (16 * CT channels)
// and the launcher of k_fwd32c.
inline int f32c_ct(int64_t C) {
  const int64_t cw = std::min<int64_t>(C, kF32MaxChannels);
  return cw <= 16 ? 1 : cw <= 32 ? 2 : 4;
}

using F32cFn = void (*)(dim3, hipStream_t, const uint4*, const uint4*, const float*, const uint4*,
                        const uint4*, const float*, const uint4*, const uint4*, int, const uint32_t*, int,
                        float, int64_t, int, int, int, int, float*, int64_t, const Bz&);

template <int DP, int CT>
void launch_f32c(dim3 grid, hipStream_t st, const uint4* qh, const uint4* ql, const float* nhq,
                 const uint4* kh, const uint4* kl, const float* scal, const uint4* vh, const uint4* vl,
                 int vstep, const uint32_t* slots, int kslot, float tau2, int64_t M, int C, int cw,
                 int steps, int sps, float* out, int64_t pstride, const Bz& bz) {
  hipLaunchKernelGGL((k_fwd32c<DP, CT>), grid, dim3(kBlockThreads), 0, st, qh, ql, nhq, kh, kl, scal, vh,
                     vl, vstep, slots, kslot, tau2, M, C, cw, steps, sps, out, pstride, bz);
}

struct F32cK {
  F32cFn launch = nullptr;
  const void* kernel = nullptr;
};

template <int DP, int CT>
F32cK f32c_k() {
  return {&launch_f32c<DP, CT>, reinterpret_cast<const void*>(&k_fwd32c<DP, CT>)};
}

template <int DP>
F32cK f32c_by_ct(int CT) {
  switch (CT) {
    case 1: return f32c_k<DP, 1>();
    case 2: return f32c_k<DP, 2>();
    case 4: return f32c_k<DP, 4>();
  }
  return {};
}

F32cK f32c_for(int DP, int CT) {
  switch (DP) {
    case 1: return f32c_by_ct<1>(CT);
    case 2: return f32c_by_ct<2>(CT);
    case 4: return f32c_by_ct<4>(CT);
    case 8: return f32c_by_ct<8>(CT);
  }
  return {};
}

// The fp32-tier forward kernel for this shape and its queries per wave.
const void* f32_pass_kernel(int64_t C, int DP) {
  return C == 1 ? f32_kernel(DP) : f32c_for(DP, f32c_ct(C)).kernel;
}
int f32_pass_qt(int64_t C, int DP) { return C == 1 ? f32_qt(DP) : f32c_qt(DP, f32c_ct(C)); }

// ------------------------------------------------------------ workspace plan

struct Carver {
  size_t off = 0;
  char* base = nullptr;
  template <typename P>
  P* take(size_t bytes) {
    size_t at = off;
    off = round_up((int64_t)(off + bytes), kAlign);
    return base ? reinterpret_cast<P*>(base + at) : nullptr;
  }
};

struct Side {  // one point set with the arrays derived from it
  uint16_t* rt = nullptr;       // RT copy (input dtype)
  float* nh = nullptr;          // -||x||^2/2 (padding rows: kPadBias)
  uint16_t* ks = nullptr;       // KS fp16 copy (operand of sum_n P k_n) as keys of a gradient pass
  uint16_t* samp_rt = nullptr;  // kSampleRows sampled rows, RT layout (coarse sample first)
  float* samp_nh = nullptr;     // their half norms
  uint16_t* lo = nullptr;       // fp32 tier: low fp16 part (rt then holds the high part)
};

struct Vals {  // one value set (v or dout)
  uint16_t* rt = nullptr;
  uint16_t* ks = nullptr;
};

// One problem's slice of the workspace (a batch puts G slices back to back,
// problem z at z * total bytes).
struct Plan {
  Dims dm;
  int64_t G = 1;               // problems sharing each launch (split counts are chosen for G)
  int64_t Mp = 0, Np = 0;
  bool alias = false;          // q and k are the same array
  uint32_t* slots = nullptr;   // [0] |v| max, [1] |dout| max, [2] |q| max, [3] |k| max
  Side q, k;
  Vals v, g;
  float* scal_kv = nullptr;    // per-step scalars, keys k with values v
  float* scal_qg = nullptr;    // per-step scalars, keys q with values dout
  float* part = nullptr;       // split partials of the running pass
  float* part_s = nullptr;     // split partials of a forward sum fused into the dq pass
  size_t total = 0;
};

struct PassShape {
  int blocks, splits, sps, steps;
};

// Workgroups of `kernel` resident on the current device at once (CUs times
// workgroups per CU), cached per kernel and device; kDefaultSlots when no
// device can be queried (workspace sizes asked for on a machine without one).
int device_slots(const void* kernel, int threads) {
  struct Entry {
    const void* kernel;
    int device, slots;
  };
  static Entry cache[512];
  static int used = 0;
  static std::mutex mu;
  int dev = 0;
  if (!kernel || hipGetDevice(&dev) != hipSuccess) return kDefaultSlots;
  std::lock_guard<std::mutex> lock(mu);
  for (int i = 0; i < used; ++i)
    if (cache[i].kernel == kernel && cache[i].device == dev) return cache[i].slots;
  int cus = 0, occ = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    return kDefaultSlots;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, threads, 0) != hipSuccess ||
      occ < 1)
    return kDefaultSlots;
  const int slots = cus * occ;
  if (used < 512) cache[used++] = Entry{kernel, dev, slots};
  return slots;
}

// Workgroups along the rows, and the split of the key steps into grid.y
// parts (partial sums combined afterwards): the split count that minimises
// (rounds of resident workgroups) x (steps per split + fixed cost), searched
// from the smallest count that fills the device once up to four times that.
// `group` problems run side by side on grid.z.
PassShape pass_shape(int64_t rows, int64_t keys, int QT, const void* kernel, int64_t group,
                     int wpb = kWavesPerBlock) {
  PassShape ps;
  ps.blocks = (int)ceil_div(rows, 16 * QT * wpb);
  ps.steps = (int)ceil_div(keys, kStep);
  const int64_t slots = device_slots(kernel, kWave * wpb);
  const int64_t wide = (int64_t)std::max(1, ps.blocks) * std::max<int64_t>(1, group);
  const int cap = std::max(1, ps.steps / kMinStepsPerSplit);
  const int need = (int)std::max<int64_t>(1, ceil_div(ps.steps, kMaxStepsPerSplit));
  const int lo = std::max(need, (int)std::min<int64_t>(cap, std::max<int64_t>(1, ceil_div(slots, wide))));
  const int hi = std::max(lo, std::min(cap, 4 * lo));
  auto cost = [&](int sp) {
    return ceil_div(wide * sp, slots) * (ceil_div(ps.steps, sp) + kSplitOverheadSteps);
  };
  int splits = lo;
  int64_t best = cost(lo);
  for (int sp = lo + 1; sp <= hi; ++sp) {
    const int64_t c = cost(sp);
    if (c * 50 < best * 49) {  // at least 2 % better
      best = c;
      splits = sp;
    }
  }
  ps.sps = (int)ceil_div(ps.steps, splits);
  ps.splits = ps.steps ? (int)ceil_div(ps.steps, ps.sps) : 1;
  return ps;
}

// When the forward sum rides along in the dq pass.  C = 1 always (it is the
// row sum the gradient forms anyway).  Otherwise only while it needs a single
// 16-row tile of V^T: beyond that the extra contraction and its registers
// cost more than a separate forward pass (C = 128, D = 128: 0.52 ms fused
// against 0.17 + 0.25 ms).  At D = 256, C = 16 the fused passes take 276 +
// 264 ms against 105 + 265 + 252 + 106 ms for the four separate ones.
constexpr int64_t kFuseMaxC = 16;

struct Want {
  bool fwd = false, dq = false, dk = false, dv = false;
  bool fuse = false;  // set by want_for (kFuseMaxC)
  bool fused() const { return fwd && dq && fuse; }  // forward computed inside the dq pass
  // dv computed inside the dk pass: with the roles of (q, dout) and (k, v)
  // exchanged, dv_n = sum_m Phi g_m is that pass's forward sum
  bool fused_kv() const { return dk && dv && fuse; }
};

Want want_for(const gs_problem& p, bool fwd, bool dq, bool dk, bool dv) {
  Want w;
  w.fwd = fwd;
  w.dq = dq;
  w.dk = dk;
  w.dv = dv;
  w.fuse = p.C <= kFuseMaxC;
  return w;
}

inline int dq_cw(const gs_problem& p, const Dims& dm) { return p.C == 1 ? 0 : dm.CW; }

FwdK fwd_for(const gs_problem& p, const Dims& dm) {
  const int ct = p.C == 1 ? 0 : dm.CT;
  return p.qk_dtype == GS_F16 ? fwd_fn<F16>(dm.DP, ct) : fwd_fn<BF16>(dm.DP, ct);
}
DqK dq_for(const gs_problem& p, const Dims& dm, bool fused) {
  const int cw = dq_cw(p, dm);
  return p.qk_dtype == GS_F16 ? dq_fn<F16>(dm.DP, cw, dm.CT, fused) : dq_fn<BF16>(dm.DP, cw, dm.CT, fused);
}
const void* fwd_kernel(const gs_problem& p, const Dims& dm) { return fwd_for(p, dm).kernel; }
const void* dq_kernel(const gs_problem& p, const Dims& dm, bool fused) { return dq_for(p, dm, fused).kernel; }

// Small forward problems: the preparation in one launch (k_prep_fwd_small)
// and a row check that reads its key sample from the key copy, instead of
// nine dependent launches.  Bounds: every workgroup of the preparation
// reduces all N C values itself, and the point copies stay small.
constexpr int64_t kSmallValues = 8192;        // N * C
constexpr int64_t kSmallPointHalves = 1 << 18; // padded rows x RT width, per point set

bool small_forward(const gs_problem& p, const Want& w, const Plan& pl, int64_t G) {
  return w.fwd && !w.dq && !w.dk && !w.dv && G == 1 && p.N * p.C <= kSmallValues &&
         pl.Mp * pl.dm.W() <= kSmallPointHalves && pl.Np * pl.dm.W() <= kSmallPointHalves;
}

// Lays out every buffer the requested passes need for one problem of a group
// of G; with ws == nullptr only computes the size.
void make_plan(const gs_problem& p, const Want& w, bool alias, void* ws, Plan& pl, int64_t G) {
  pl.dm = dims_of(p.D, p.C);
  pl.G = G;
  pl.Mp = round_up(std::max<int64_t>(p.M, 1), kRowPad);
  pl.Np = round_up(std::max<int64_t>(p.N, 1), kRowPad);
  pl.alias = alias;
  const int W = pl.dm.W(), Wv = pl.dm.Wv(), Rv = pl.dm.Rv();
  Carver cv;
  cv.base = static_cast<char*>(ws);
  pl.slots = cv.take<uint32_t>(64);
  if (p.qk_dtype == GS_F32) {
    // fp32 tier (forward): split copies, half norms, step scalars, and for
    // several channels the split values (KS layout)
    auto split = [&](Side& s, int64_t n_pad) {
      s.rt = cv.take<uint16_t>(n_pad * W * 2);
      s.lo = cv.take<uint16_t>(n_pad * W * 2);
      s.nh = cv.take<float>(n_pad * 4);
    };
    split(pl.q, pl.Mp);
    if (alias)
      pl.k = pl.q;
    else
      split(pl.k, pl.Np);
    pl.scal_kv = cv.take<float>(pl.Np * 2 * 4);
    if (p.C > 1) {
      pl.v.ks = cv.take<uint16_t>(pl.Np * Rv * 2);  // high parts
      pl.v.rt = cv.take<uint16_t>(pl.Np * Rv * 2);  // low parts (same KS layout)
    }
    const PassShape ps = pass_shape(p.M, p.N, f32_pass_qt(p.C, pl.dm.DP), f32_pass_kernel(p.C, pl.dm.DP), G);
    pl.part = ps.splits > 1 ? cv.take<float>((size_t)ps.splits * p.M * p.C * 4) : nullptr;
    pl.total = cv.off;
    return;
  }
  const bool keys_k = w.fwd || w.dq;  // passes whose keys are k
  const bool keys_q = w.dk || w.dv;   // passes whose keys are q
  // KS copies of the points: keys of a gradient pass, unless that pass reads
  // its K^T operands from the RT tiles (dq_transposed_keys)
  const bool f16 = p.qk_dtype == GS_F16;
  const int cw = dq_cw(p, pl.dm);
  const bool need_k_ks = w.dq && !dq_transposed_keys(f16, pl.dm.DP, cw);
  const bool need_q_ks = w.dk && !dq_transposed_keys(f16, pl.dm.DP, cw);
  // sample of a key side: its half norms are followed by the row-bound flags
  // of the rows queried against it (the other side's padded row count)
  auto side = [&](Side& s, int64_t n_pad, bool ks, bool sample, int64_t other_pad) {
    s.rt = cv.take<uint16_t>(n_pad * W * 2);
    s.nh = cv.take<float>(n_pad * 4);
    if (ks) s.ks = cv.take<uint16_t>(n_pad * W * 2);
    if (sample) {
      s.samp_rt = cv.take<uint16_t>(kSampleRows * W * 2);
      s.samp_nh = cv.take<float>(kSampleRows * 4 + other_pad * 4);
    }
  };
  if (alias) {
    // single channel: the KS copies carry the signs of v (dq) or dout (dk)
    const bool two = p.C == 1 && need_q_ks && need_k_ks;
    side(pl.q, pl.Mp, need_q_ks || need_k_ks, true, pl.Mp);
    pl.k = pl.q;
    if (two) pl.k.ks = cv.take<uint16_t>(pl.Mp * W * 2);
  } else {
    side(pl.q, pl.Mp, need_q_ks, keys_q, pl.Np);
    side(pl.k, pl.Np, need_k_ks, keys_k, pl.Mp);
  }
  if (keys_k) pl.scal_kv = cv.take<float>(pl.Np * 2 * 4);
  if (keys_q) pl.scal_qg = cv.take<float>(pl.Mp * 2 * 4);
  // RT value copies feed the <g, v> contraction of several channels only
  // (single-channel gradients fold v into the exponent and the signs)
  const bool wc = (w.dq || w.dk) && p.C > 1;
  if (wc) pl.v.rt = cv.take<uint16_t>(pl.Np * Wv * 2);
  if (w.fwd && !(w.fused() && p.C == 1)) pl.v.ks = cv.take<uint16_t>(pl.Np * Rv * 2);
  if (wc) pl.g.rt = cv.take<uint16_t>(pl.Mp * Wv * 2);
  if (w.dv && !(w.fused_kv() && p.C == 1)) pl.g.ks = cv.take<uint16_t>(pl.Mp * Rv * 2);

  // Partial-sum buffer for split passes (reused by every pass in turn).
  size_t part = 0, part_s = 0;
  auto consider = [&](int64_t rows, int64_t keys, int QT, int64_t width, const void* kernel,
                      int wpb = kWavesPerBlock) {
    PassShape ps = pass_shape(rows, keys, QT, kernel, G, wpb);
    if (ps.splits > 1) part = std::max(part, (size_t)ps.splits * rows * width * 4);
    return ps.splits;
  };
  const int qf = fwd_qt(pl.dm.DP, pl.dm.CT), qd = dq_qt(pl.dm.DP, dq_cw(p, pl.dm));
  const void* kf = fwd_kernel(p, pl.dm);
  if (w.fwd && !w.fused()) consider(p.M, p.N, qf, p.C, kf, fwd_wpb(pl.dm.DP));
  if (w.dq) {
    const int sp = consider(p.M, p.N, qd, p.D, dq_kernel(p, pl.dm, w.fused()), dq_wpb(pl.dm.DP));
    if (w.fused() && sp > 1) part_s = (size_t)sp * p.M * p.C * 4;
  }
  if (w.dk) {
    const int sp = consider(p.N, p.M, qd, p.D, dq_kernel(p, pl.dm, w.fused_kv()), dq_wpb(pl.dm.DP));
    if (w.fused_kv() && sp > 1) part_s = std::max(part_s, (size_t)sp * p.N * p.C * 4);
  }
  if (w.dv && !w.fused_kv()) consider(p.N, p.M, qf, p.C, kf, fwd_wpb(pl.dm.DP));
  pl.part = part ? cv.take<float>(part) : nullptr;
  pl.part_s = part_s ? cv.take<float>(part_s) : nullptr;
  pl.total = cv.off;
}

// ------------------------------------------------------------ timing hook

struct Profiler {
  hipEvent_t* ev = nullptr;
  int capacity = 0, used = 0, kind = 0;
};
Profiler g_prof;

enum { kKindFwd = 1, kKindGrad = 2 };

inline void prof_before(int kind, hipStream_t st) {
  if (g_prof.ev && (g_prof.kind & kind) && g_prof.used < g_prof.capacity)
    (void)hipEventRecord(g_prof.ev[2 * g_prof.used], st);
}
inline void prof_after(int kind, hipStream_t st) {
  if (g_prof.ev && (g_prof.kind & kind) && g_prof.used < g_prof.capacity) {
    (void)hipEventRecord(g_prof.ev[2 * g_prof.used + 1], st);
    ++g_prof.used;
  }
}

void prof_release() {
  if (!g_prof.ev) return;
  for (int i = 0; i < 2 * g_prof.capacity; ++i)
    if (g_prof.ev[i]) (void)hipEventDestroy(g_prof.ev[i]);
  delete[] g_prof.ev;
  g_prof = Profiler();
}

// ------------------------------------------------------------ launches

inline unsigned grid1(int64_t n, int threads = 256) {
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>(ceil_div(n, threads), 1 << 20));
}
// Reductions: at most 512 workgroups (grid-stride), one atomic each.
inline unsigned grid_reduce(int64_t n) { return std::min(grid1(n), 128u); }

// A launch group: G problems on grid.z, each with a workspace slice of
// `slice` bytes (pl describes the first one).
struct Ctx {
  hipStream_t st;
  const gs_problem* p;
  Plan* pl;
  float tau, tau2;
  unsigned G;
  int64_t slice;
};

inline Bz bz_ws(const Ctx& c) {
  Bz b;
  b.ws = c.slice;
  return b;
}
inline dim3 grid_g(const Ctx& c, unsigned x, unsigned y = 1) { return dim3(x, y, c.G); }

// xs: byte stride of x between problems.  sgn / sgn_dt / sgns: for
// single-channel problems, the values whose signs the KS copy of these points
// (as keys of a gradient pass) carries, and their stride; else NULL.
template <typename T>
void prep_points_t(const Ctx& c, const uint16_t* x16, int64_t xs, int64_t n, int64_t n_pad, Side& s,
                   uint32_t* slot, const void* sgn, int sgn_dt, int64_t sgns) {
  const gs_problem& p = *c.p;
  const int W = c.pl->dm.W();
  Bz bz = bz_ws(c);
  bz.in = xs;
  bz.in2 = sgns;
  // 16-byte row loads when every problem's rows start on 16-byte boundaries
  const int vec = (p.D % 8 == 0) && ((reinterpret_cast<uintptr_t>(x16) | (uintptr_t)xs) % 16 == 0);
  hipLaunchKernelGGL(k_points_rt_norm<T>, grid_g(c, grid1(n_pad * (W / 8))), dim3(256), 0, c.st, x16, n,
                     (int)p.D, n_pad, W, s.rt, s.nh, vec, bz);
  if (s.samp_rt)
    hipLaunchKernelGGL(k_sample, grid_g(c, grid1(kSampleRows * W)), dim3(256), 0, c.st, x16, n, (int)p.D,
                       W, (const float*)s.nh, s.samp_rt, s.samp_nh, bz);
  if (s.ks) {
    const uint32_t* sl = nullptr;
    if (p.qk_dtype == GS_BF16) {
      hipLaunchKernelGGL(k_absmax, grid_g(c, grid_reduce(n * p.D)), dim3(256), 0, c.st,
                         static_cast<const void*>(x16), n * p.D, 2, slot, bz);
      sl = slot;
    }
    hipLaunchKernelGGL(k_points_ks<T>, grid_g(c, grid1(n_pad / 8 * W)), dim3(256), 0, c.st, x16, n,
                       (int)p.D, n_pad, W, sl, sgn, (int)sgn_dt, s.ks, bz);
  }
}

void prep_points(const Ctx& c, const void* x, int64_t xs, int64_t n, int64_t n_pad, Side& s,
                 uint32_t* slot, const void* sgn = nullptr, int sgn_dt = GS_F32, int64_t sgns = 0) {
  const uint16_t* x16 = static_cast<const uint16_t*>(x);
  if (c.p->qk_dtype == GS_F16)
    prep_points_t<F16>(c, x16, xs, n, n_pad, s, slot, sgn, sgn_dt, sgns);
  else
    prep_points_t<BF16>(c, x16, xs, n, n_pad, s, slot, sgn, sgn_dt, sgns);
}

// KS copy only (the second, differently signed copy of aliased points).
void prep_points_ks(const Ctx& c, const void* x, int64_t xs, int64_t n, int64_t n_pad, uint16_t* ks,
                    uint32_t* slot, const void* sgn, int sgn_dt, int64_t sgns) {
  const gs_problem& p = *c.p;
  const int W = c.pl->dm.W();
  const uint16_t* x16 = static_cast<const uint16_t*>(x);
  const uint32_t* sl = p.qk_dtype == GS_BF16 ? slot : nullptr;
  Bz bz = bz_ws(c);
  bz.in = xs;
  bz.in2 = sgns;
  if (p.qk_dtype == GS_F16)
    hipLaunchKernelGGL(k_points_ks<F16>, grid_g(c, grid1(n_pad / 8 * W)), dim3(256), 0, c.st, x16, n,
                       (int)p.D, n_pad, W, sl, sgn, (int)sgn_dt, ks, bz);
  else
    hipLaunchKernelGGL(k_points_ks<BF16>, grid_g(c, grid1(n_pad / 8 * W)), dim3(256), 0, c.st, x16, n,
                       (int)p.D, n_pad, W, sl, sgn, (int)sgn_dt, ks, bz);
}

void prep_values(const Ctx& c, const void* x, int dt, int64_t xs, int64_t n, int64_t n_pad,
                 Vals& s, uint32_t* slot) {
  const gs_problem& p = *c.p;
  const int Wv = c.pl->dm.Wv(), Rv = c.pl->dm.Rv();
  Bz bz = bz_ws(c);
  bz.in = xs;
  if (n > 0)
    hipLaunchKernelGGL(k_absmax, grid_g(c, grid_reduce(n * p.C)), dim3(256), 0, c.st, x, n * p.C, (int)dt,
                       slot, bz);
  if (s.rt)
    hipLaunchKernelGGL(k_values_rt, grid_g(c, grid1(n_pad * Wv)), dim3(256), 0, c.st, x, (int)dt, n,
                       (int)p.C, n_pad, Wv, (const uint32_t*)slot, s.rt, bz);
  if (s.ks)
    hipLaunchKernelGGL(k_values_ks, grid_g(c, grid1(n_pad / 8 * Rv)), dim3(256), 0, c.st, x, (int)dt, n,
                       (int)p.C, n_pad, Rv, (const uint32_t*)slot, (int)(p.C == 1), s.ks, bz);
}

// Per-step key scalars of key side `s` paired with values x (byte stride xs,
// slot = their absolute maximum): single-channel problems fold log2|v| and
// sign(v) in, otherwise half norms only.
void prep_scalars(const Ctx& c, const Side& s, const void* x, int dt, int64_t xs, int64_t n,
                  int64_t n_pad, const uint32_t* slot, float* out) {
  const bool vals = c.p->C == 1 && x != nullptr;
  Bz bz = bz_ws(c);
  bz.in = vals ? xs : 0;
  hipLaunchKernelGGL(k_step_scalars, grid_g(c, grid1(n_pad * 2)), dim3(256), 0, c.st, (const float*)s.nh,
                     vals ? x : nullptr, (int)dt, n, n_pad, slot, c.tau2, out, bz);
}

// Row-bound flags of the rows of `qs` (n rows, n_pad padded) against the
// sampled keys of `ks`, stored after the sample's half norms.
template <typename T, bool GATHER>
void row_check_t(const Ctx& c, const Side& qs, int64_t n, int64_t n_pad, const Side& ks, int64_t nk) {
  uint32_t* shift = reinterpret_cast<uint32_t*>(ks.samp_nh + kSampleRows);
  const dim3 grid = grid_g(c, (unsigned)(n_pad / 256)), block(kBlockThreads);
  const uint4* q = (const uint4*)qs.rt;
  // the copied sample, or (GATHER) the key set's own RT copy and half norms
  const uint4* s = (const uint4*)(GATHER ? ks.rt : ks.samp_rt);
  const float* snh = GATHER ? ks.nh : ks.samp_nh;
  const Bz bz = bz_ws(c);
  switch (c.pl->dm.DP) {
    case 1: hipLaunchKernelGGL((k_row_check<T, 1, GATHER>), grid, block, 0, c.st, q, qs.nh, s, snh, c.tau2, n, shift, bz, nk); break;
    case 2: hipLaunchKernelGGL((k_row_check<T, 2, GATHER>), grid, block, 0, c.st, q, qs.nh, s, snh, c.tau2, n, shift, bz, nk); break;
    case 4: hipLaunchKernelGGL((k_row_check<T, 4, GATHER>), grid, block, 0, c.st, q, qs.nh, s, snh, c.tau2, n, shift, bz, nk); break;
    case 8: hipLaunchKernelGGL((k_row_check<T, 8, GATHER>), grid, block, 0, c.st, q, qs.nh, s, snh, c.tau2, n, shift, bz, nk); break;
  }
}

// Row-bound flags of the rows of qs against the key sample of ks; gather:
// read the sampled keys from ks's own RT copy (nk keys) instead of a copy.
void row_check(const Ctx& c, const Side& qs, int64_t n, int64_t n_pad, const Side& ks, bool gather = false,
               int64_t nk = 0) {
  if (c.p->qk_dtype == GS_F16) {
    if (gather)
      row_check_t<F16, true>(c, qs, n, n_pad, ks, nk);
    else
      row_check_t<F16, false>(c, qs, n, n_pad, ks, nk);
  } else {
    if (gather)
      row_check_t<BF16, true>(c, qs, n, n_pad, ks, nk);
    else
      row_check_t<BF16, false>(c, qs, n, n_pad, ks, nk);
  }
}

void prep_fwd_small(const Ctx& c, const void* q, const void* k, const void* v, bool alias) {
  const gs_problem& p = *c.p;
  Plan& pl = *c.pl;
  const int W = pl.dm.W(), R = pl.dm.Rv();
  const int64_t items = pl.Mp * (W / 8) + (alias ? 0 : pl.Np * (W / 8)) + (pl.Np / 32) * R * 4 + pl.Np;
  const unsigned blocks = (unsigned)std::min<int64_t>(ceil_div(items, 256), 1024);
  auto vec = [&](const void* x) {
    return (int)((p.D % 8 == 0) && (reinterpret_cast<uintptr_t>(x) % 16 == 0));
  };
  const uint16_t* q16 = static_cast<const uint16_t*>(q);
  const uint16_t* k16 = static_cast<const uint16_t*>(k);
  if (p.qk_dtype == GS_F16)
    hipLaunchKernelGGL(k_prep_fwd_small<F16>, dim3(blocks), dim3(256), 0, c.st, q16, k16, (int)alias, v,
                       (int)p.v_dtype, p.M, p.N, (int)p.D, (int)p.C, pl.Mp, pl.Np, W, R, vec(q), vec(k), c.tau2,
                       pl.q.rt, pl.q.nh, pl.k.rt, pl.k.nh, pl.v.ks, pl.scal_kv, pl.slots);
  else
    hipLaunchKernelGGL(k_prep_fwd_small<BF16>, dim3(blocks), dim3(256), 0, c.st, q16, k16, (int)alias, v,
                       (int)p.v_dtype, p.M, p.N, (int)p.D, (int)p.C, pl.Mp, pl.Np, W, R, vec(q), vec(k), c.tau2,
                       pl.q.rt, pl.q.nh, pl.k.rt, pl.k.nh, pl.v.ks, pl.scal_kv, pl.slots);
}

// Split partials (in the workspace slices) -> out (byte stride out_stride).
void combine(const Ctx& c, const PassShape& ps, const float* part, int64_t count, float* out,
             int64_t out_stride) {
  if (ps.splits <= 1) return;
  Bz bz = bz_ws(c);
  bz.out = out_stride;
  hipLaunchKernelGGL(k_combine, grid_g(c, grid1(count)), dim3(256), 0, c.st, part, ps.splits, count, out,
                     bz);
}

// Forward-type pass: out[m, :] = sum_n Phi(x_m, y_n) val_n for x = qside rows
// (out: byte stride os between problems).
void pass_fwd(const Ctx& c, const Side& qs, int64_t nq, const Side& ks, int64_t nk, const float* scal,
              const uint16_t* vks, const uint32_t* vslot, float* out, int64_t os) {
  const gs_problem& p = *c.p;
  const Dims& dm = c.pl->dm;
  const FwdK fk = fwd_for(p, dm);
  PassShape ps = pass_shape(nq, nk, fwd_qt(dm.DP, dm.CT), fk.kernel, c.pl->G, fwd_wpb(dm.DP));
  const bool split = ps.splits > 1;
  float* dst = split ? c.pl->part : out;
  Bz bz = bz_ws(c);
  bz.out = split ? c.slice : os;
  prof_before(kKindFwd, c.st);
  fk.launch(grid_g(c, ps.blocks, ps.splits), c.st, (const uint4*)qs.rt, qs.nh, (const uint4*)ks.samp_rt,
            ks.samp_nh, (const uint4*)ks.rt, scal, (const uint4*)vks, vslot, c.tau2, nq, (int)p.C,
            ps.steps, ps.sps, dst, split ? nq * p.C : 0, bz);
  prof_after(kKindFwd, c.st);
  combine(c, ps, c.pl->part, nq * p.C, out, os);
}

// dq-type pass: out[m, :] = tau sum_n Phi(x_m, y_n) <gx_m, vy_n> (y_n - x_m).
// g1 / g1_dt / g1s: the caller's single-channel upstream gradient of the
// query rows (C = 1), read exactly in the epilogue, and its byte stride.
// With out_s != NULL the forward sum over the same pairs is produced by the
// same kernel (values vks: V^T in KS layout, unused for C = 1).  os / os_s:
// byte strides of out / out_s between problems.
void pass_dq(const Ctx& c, const Side& qs, int64_t nq, const Side& ks, int64_t nk, const float* scal,
             const uint32_t* kslot, const uint16_t* vrt, const uint32_t* vslot, const uint16_t* grt,
             const uint32_t* gslot, const void* g1, int g1_dt, int64_t g1s, float* out, int64_t os,
             const uint16_t* vks = nullptr, float* out_s = nullptr, int64_t os_s = 0) {
  const gs_problem& p = *c.p;
  const Dims& dm = c.pl->dm;
  const bool fused = out_s != nullptr;
  const DqK dk = dq_for(p, dm, fused);
  PassShape ps = pass_shape(nq, nk, dq_qt(dm.DP, dq_cw(p, dm)), dk.kernel, c.pl->G, dq_wpb(dm.DP));
  const bool split = ps.splits > 1;
  float* dst = split ? c.pl->part : out;
  float* dst_s = fused ? (split ? c.pl->part_s : out_s) : nullptr;
  Bz bz = bz_ws(c);
  bz.in2 = g1s;
  bz.out = split ? c.slice : os;
  bz.out2 = split ? c.slice : os_s;
  prof_before(kKindGrad, c.st);
  dk.launch(grid_g(c, ps.blocks, ps.splits), c.st, (const uint4*)qs.rt, qs.nh, (const uint4*)ks.samp_rt,
            ks.samp_nh, (const uint4*)ks.rt, scal, (const uint4*)ks.ks,
            p.qk_dtype == GS_BF16 ? kslot : nullptr, (const uint4*)vrt, vslot, (const uint4*)grt, gslot,
            g1, (int)g1_dt, c.tau2, c.tau, nq, (int)p.D, ps.steps, ps.sps, dst, split ? nq * p.D : 0,
            (const uint4*)vks, (int)p.C, dst_s, split ? nq * p.C : 0, bz);
  prof_after(kKindGrad, c.st);
  combine(c, ps, c.pl->part, nq * p.D, out, os);
  if (fused) combine(c, ps, c.pl->part_s, nq * p.C, out_s, os_s);
}

// fp32 tier: prep (maxima, split copies, step scalars) and the forward pass
// of one launch group.  xs / ks / vst / os: byte strides between problems.
void run_f32(const Ctx& c, const void* q, int64_t qs, const void* k, int64_t ks, const void* v,
             int64_t vst, float* out, int64_t os) {
  const gs_problem& p = *c.p;
  Plan& pl = *c.pl;
  const int W = pl.dm.W(), DP = pl.dm.DP;
  const int64_t M = p.M, N = p.N;
  Bz bz = bz_ws(c);
  hipLaunchKernelGGL(k_fill_u32, grid_g(c, 1), dim3(64), 0, c.st, pl.slots, 16, 0u, bz);
  auto points = [&](const void* x, int64_t xs, int64_t n, int64_t n_pad, Side& sd, uint32_t* slot) {
    Bz b = bz_ws(c);
    b.in = xs;
    hipLaunchKernelGGL(k_absmax, grid_g(c, grid_reduce(n * p.D)), dim3(256), 0, c.st, x, n * p.D, 0, slot, b);
    hipLaunchKernelGGL(k_points_split, grid_g(c, grid1(n_pad * (W / 8))), dim3(256), 0, c.st,
                       static_cast<const float*>(x), n, (int)p.D, n_pad, W, (const uint32_t*)slot, sd.rt,
                       sd.lo, sd.nh, b);
  };
  points(q, qs, M, pl.Mp, pl.q, pl.slots + 2);
  if (!pl.alias) points(k, ks, N, pl.Np, pl.k, pl.slots + 3);
  const int kslot = pl.alias ? 2 : 3;
  Bz bv = bz_ws(c);
  bv.in = vst;
  const int64_t C = p.C;
  hipLaunchKernelGGL(k_absmax, grid_g(c, grid_reduce(N * C)), dim3(256), 0, c.st, v, N * C, (int)p.v_dtype,
                     pl.slots + 0, bv);
  if (C > 1) {
    const int Rv = pl.dm.Rv();
    hipLaunchKernelGGL(k_values_ks_split, grid_g(c, grid1(pl.Np / 8 * Rv)), dim3(256), 0, c.st, v,
                       (int)p.v_dtype, N, (int)C, pl.Np, Rv, (const uint32_t*)pl.slots + 0, pl.v.ks, pl.v.rt,
                       bv);
  }
  hipLaunchKernelGGL(k_step_scalars32, grid_g(c, grid1(pl.Np * 2)), dim3(256), 0, c.st,
                     (const float*)pl.k.nh, C == 1 ? v : nullptr, (int)p.v_dtype, N, pl.Np,
                     (const uint32_t*)pl.slots + 0, (const uint32_t*)pl.slots + 2,
                     (const uint32_t*)pl.slots + kslot, c.tau2, pl.scal_kv, bv);
  if (C > 1) {
    // several channels: launches of up to kF32MaxChannels channels each
    const int CT = f32c_ct(C);
    const F32cK fk = f32c_for(DP, CT);
    const PassShape ps = pass_shape(M, N, f32c_qt(DP, CT), fk.kernel, pl.G);
    const bool split = ps.splits > 1;
    Bz bk = bz_ws(c);
    bk.out = split ? c.slice : os;
    const int Rv = pl.dm.Rv();
    prof_before(kKindFwd, c.st);
    for (int64_t c0 = 0; c0 < C; c0 += kF32MaxChannels) {
      const int cw = (int)std::min<int64_t>(C - c0, kF32MaxChannels);
      float* dst = (split ? pl.part : out) + c0;
      fk.launch(grid_g(c, ps.blocks, ps.splits), c.st, (const uint4*)pl.q.rt, (const uint4*)pl.q.lo,
                (const float*)pl.q.nh, (const uint4*)pl.k.rt, (const uint4*)pl.k.lo, (const float*)pl.scal_kv,
                (const uint4*)(pl.v.ks + c0 * 32), (const uint4*)(pl.v.rt + c0 * 32), Rv * 64,
                (const uint32_t*)pl.slots, kslot, c.tau2, M, (int)C, cw, ps.steps, ps.sps, dst,
                split ? M * C : 0, bk);
    }
    prof_after(kKindFwd, c.st);
    combine(c, ps, pl.part, M * C, out, os);
    return;
  }
  const PassShape ps = pass_shape(M, N, f32_qt(DP), f32_kernel(DP), pl.G);
  const bool split = ps.splits > 1;
  float* dst = split ? pl.part : out;
  Bz bk = bz_ws(c);
  bk.out = split ? c.slice : os;
  const dim3 grid = grid_g(c, ps.blocks, ps.splits), block(kBlockThreads);
  const uint4 *qh = (const uint4*)pl.q.rt, *ql = (const uint4*)pl.q.lo;
  const uint4 *kh = (const uint4*)pl.k.rt, *kl = (const uint4*)pl.k.lo;
  const int64_t pst = split ? M : 0;
  prof_before(kKindFwd, c.st);
  switch (DP) {
    case 1: hipLaunchKernelGGL(k_fwd32<1>, grid, block, 0, c.st, qh, ql, (const float*)pl.q.nh, kh, kl, (const float*)pl.scal_kv, (const uint32_t*)pl.slots, kslot, c.tau2, M, ps.steps, ps.sps, dst, pst, bk); break;
    case 2: hipLaunchKernelGGL(k_fwd32<2>, grid, block, 0, c.st, qh, ql, (const float*)pl.q.nh, kh, kl, (const float*)pl.scal_kv, (const uint32_t*)pl.slots, kslot, c.tau2, M, ps.steps, ps.sps, dst, pst, bk); break;
    case 4: hipLaunchKernelGGL(k_fwd32<4>, grid, block, 0, c.st, qh, ql, (const float*)pl.q.nh, kh, kl, (const float*)pl.scal_kv, (const uint32_t*)pl.slots, kslot, c.tau2, M, ps.steps, ps.sps, dst, pst, bk); break;
    case 8: hipLaunchKernelGGL(k_fwd32<8>, grid, block, 0, c.st, qh, ql, (const float*)pl.q.nh, kh, kl, (const float*)pl.scal_kv, (const uint32_t*)pl.slots, kslot, c.tau2, M, ps.steps, ps.sps, dst, pst, bk); break;
  }
  prof_after(kKindFwd, c.st);
  combine(c, ps, pl.part, M, out, os);
}

void fill_zero(hipStream_t st, float* p, int64_t n) {
  if (p && n > 0) hipLaunchKernelGGL(k_fill_f32, dim3(grid1(n)), dim3(256), 0, st, p, n, 0.0f);
}

// ------------------------------------------------------------ validation

size_t dsize(int t) { return t == GS_F32 ? 4 : 2; }

bool valid_dtype(int t) { return t == GS_F32 || t == GS_F16 || t == GS_BF16; }

gs_status check_problem(const gs_problem* p) {
  if (!p) return GS_ERR_NULL_POINTER;
  if (p->M < 0 || p->N < 0 || p->D < 1 || p->D > GAUSS_SUM_MAX_DIM || p->C < 1 ||
      p->C > GAUSS_SUM_MAX_DIM)
    return GS_ERR_BAD_SHAPE;
  if (p->M > kMaxRows || p->N > kMaxRows) return GS_ERR_BAD_SHAPE;
  if (!valid_dtype(p->qk_dtype)) return GS_ERR_UNSUPPORTED;
  if (!valid_dtype(p->v_dtype)) return GS_ERR_UNSUPPORTED;
  return GS_SUCCESS;
}

// The fp32 tier (fp32 points) computes the forward sum only.
gs_status check_tier(const gs_problem* p, bool grads) {
  if (p->qk_dtype == GS_F32 && grads) return GS_ERR_UNSUPPORTED;
  return GS_SUCCESS;
}

gs_status check_tau(float tau) {
  if (!(tau > 0.0f) || !std::isfinite(tau)) return GS_ERR_BAD_TAU;
  return GS_SUCCESS;
}

bool aligned(const void* ptr, size_t a) { return (reinterpret_cast<uintptr_t>(ptr) % a) == 0; }

struct Range {
  uintptr_t lo, hi;
};
Range range_of(const void* ptr, int64_t bytes) {
  uintptr_t a = reinterpret_cast<uintptr_t>(ptr);
  return Range{a, a + (uintptr_t)std::max<int64_t>(bytes, 0)};
}
bool overlap(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi && a.hi > a.lo && b.hi > b.lo; }

gs_status check_workspace(void* ws, size_t have, size_t need) {
  if (need == 0) return GS_SUCCESS;
  if (!ws) return GS_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return GS_ERR_MISALIGNED;
  if (have < need) return GS_ERR_WORKSPACE;
  return GS_SUCCESS;
}

gs_status launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? GS_SUCCESS : GS_ERR_HIP;
}

}  // namespace
}  // namespace gs

using namespace gs;

namespace {
constexpr int kDotBlocks = 256;

// Leading workspace of gauss_sum_mmd_flow: all-ones upstream gradient (n
// fp32), the forward sum when the caller does not want it (n fp32), the
// reduction partials; the gradient pass's own workspace follows.
size_t flow_extra(int64_t n) {
  const int64_t a = gs::round_up(std::max<int64_t>(n, 1) * 4, 256);
  return (size_t)(2 * a + gs::round_up(kDotBlocks * 8, 256));
}
}  // namespace

extern "C" {

int gauss_sum_abi_version(void) { return GAUSS_SUM_ABI_VERSION; }


const char* gauss_sum_status_string(int status) {
  // an int, not gs_status: a C caller may pass any code, and an enumeration
  // object holding a value outside its range is undefined in C++
  switch (status) {
    case GS_SUCCESS: return "success";
    case GS_ERR_NULL_POINTER: return "a required pointer is NULL or no output was requested";
    case GS_ERR_BAD_SHAPE: return "bad shape: need M, N >= 0 and 1 <= D, C <= 256";
    case GS_ERR_BAD_TAU: return "tau must be finite and > 0";
    case GS_ERR_UNSUPPORTED: return "unsupported dtype combination";
    case GS_ERR_MISALIGNED: return "pointer not aligned (elements to their size, workspace to 256 bytes)";
    case GS_ERR_WORKSPACE: return "workspace missing or smaller than required";
    case GS_ERR_HIP: return "HIP runtime error";
    case GS_ERR_INTERNAL: return "internal error";
    case GS_ERR_ALIAS: return "an output overlaps an input or another output";
    case GS_ERR_SCRATCH_LIMIT: return "problem needs more scratch than the no-allocation entry point holds";
  }
  return "unknown status";
}

gs_status gauss_sum_profile_start(int capacity, int kind) {
  if (capacity < 1 || kind < 1 || kind > 3) return GS_ERR_BAD_SHAPE;
  prof_release();
  g_prof.ev = new (std::nothrow) hipEvent_t[2 * (size_t)capacity]();
  if (!g_prof.ev) return GS_ERR_INTERNAL;
  g_prof.capacity = capacity;
  g_prof.kind = kind;
  for (int i = 0; i < 2 * capacity; ++i) {
    if (hipEventCreate(&g_prof.ev[i]) != hipSuccess) {
      prof_release();
      return GS_ERR_HIP;
    }
  }
  return GS_SUCCESS;
}

int gauss_sum_profile_stop(float* ms, int max) {
  if (!g_prof.ev) return 0;
  int n = g_prof.used, rc = n;
  for (int i = 0; i < n; ++i) {
    if (hipEventSynchronize(g_prof.ev[2 * i + 1]) != hipSuccess) { rc = -1; break; }
    float t = 0.0f;
    if (hipEventElapsedTime(&t, g_prof.ev[2 * i], g_prof.ev[2 * i + 1]) != hipSuccess) {
      rc = -1;
      break;
    }
    if (ms && i < max) ms[i] = t;
  }
  prof_release();
  return rc;
}

}  // extern "C"

namespace gs {

// Workspace of gauss_sum_fwd_noalloc: a file-scope device array (one copy
// per GPU, held until the process ends).  Host code never uses the symbol
// itself as an address: its device address on the current GPU comes from
// hipGetSymbolAddress, once per device.
constexpr size_t kScratchBytes = GAUSS_SUM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void* g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

// Device address of `scratch` on the current GPU (looked up on the first
// call per device, with that device current).
gs_status scratch_address(void** ptr) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return GS_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return GS_ERR_UNSUPPORTED;
  std::call_once(g_scratch_once[dev], [dev] {
    void* p = nullptr;
    g_scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch_ptr[dev] = p;
  });
  if (g_scratch_err[dev] != hipSuccess || !g_scratch_ptr[dev]) return GS_ERR_HIP;
  *ptr = g_scratch_ptr[dev];
  return GS_SUCCESS;
}

// Problems per launch group at most (grid.z).
constexpr int64_t kMaxGroup = 65535;

// Workspace for `count` problems of shape p in one launch group (count
// capped at kMaxGroup); 0 when nothing would be computed.
size_t workspace_for(const gs_problem* p, bool fwd, int want_dq, int want_dk, int want_dv,
                     int64_t count = 1) {
  if (check_problem(p) != GS_SUCCESS) return 0;
  if (check_tier(p, want_dq || want_dk || want_dv) != GS_SUCCESS) return 0;
  if (p->M == 0 || p->N == 0 || count < 1) return 0;
  Want w = want_for(*p, fwd, want_dq != 0, want_dk != 0, want_dv != 0);
  if (!w.fwd && !w.dq && !w.dk && !w.dv) return 0;
  const int64_t G = std::min(count, kMaxGroup);
  Plan pl;
  make_plan(*p, w, false, nullptr, pl, G);
  // the plan with q and k aliased never needs more than the separate one
  return (size_t)G * pl.total;
}

// Problems per launch group for `cnt` problems and the workspace given (at
// least one problem's slice, checked by the caller): the most that fit,
// then evened out over the groups that takes.  pl: the plan for that size.
int64_t group_size(const gs_problem& p, const Want& w, bool alias, int64_t cnt, size_t bytes, Plan& pl) {
  int64_t G = std::min(cnt, kMaxGroup);
  for (;;) {
    make_plan(p, w, alias, nullptr, pl, G);
    if (G == 1 || (size_t)G * pl.total <= bytes) break;
    G = std::max<int64_t>(1, std::min<int64_t>(G - 1, (int64_t)(bytes / pl.total)));
  }
  const int64_t even = ceil_div(cnt, ceil_div(cnt, G));
  if (even < G) {
    Plan pe;
    make_plan(p, w, alias, nullptr, pe, even);
    if ((size_t)even * pe.total <= bytes) {
      pl = pe;
      return even;
    }
  }
  return G;
}

// Common body of the compute entry points.  b == NULL: one problem; else a
// batch of b->count problems at the element strides of b.  Validates
// everything (every problem's operand spans against each other and the
// workspace) before anything is enqueued, then runs the problems in launch
// groups: prep kernels and passes for the requested outputs (out: forward
// sum, dq / dk / dv: gradients; NULL = not requested), each launch covering a
// whole group on grid.z.
gs_status run(const gs_problem* p, const gs_batch* b, const void* q, const void* k, const void* v,
              float tau, const void* dout, int dout_dtype, float* out, float* dq, float* dk,
              float* dv, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  gs_status st = check_problem(p);
  if (st != GS_SUCCESS) return st;
  if ((st = check_tau(tau)) != GS_SUCCESS) return st;
  const int64_t M = p->M, N = p->N, D = p->D, C = p->C;
  const bool grads = dq || dk || dv;
  if ((st = check_tier(p, grads)) != GS_SUCCESS) return st;
  const int64_t ps = (int64_t)dsize(p->qk_dtype);  // bytes per point coordinate
  gs_batch one{};
  one.count = 1;
  if (b) {
    if (b->count < 0 || b->q_stride < 0 || b->k_stride < 0 || b->v_stride < 0 || b->dout_stride < 0 ||
        b->out_stride < 0 || b->dq_stride < 0 || b->dk_stride < 0 || b->dv_stride < 0)
      return GS_ERR_BAD_SHAPE;
    if (b->count == 0) return GS_SUCCESS;  // nothing to compute, no pointer is used
    if (!out && !grads) return GS_ERR_NULL_POINTER;
  }
  const gs_batch& bt = b ? *b : one;
  const int64_t cnt = bt.count;
  if (grads && !valid_dtype(dout_dtype)) return GS_ERR_UNSUPPORTED;
  if (!out && !grads) return M == 0 && N == 0 ? GS_SUCCESS : GS_ERR_NULL_POINTER;
  if (cnt > 1 && ((out && bt.out_stride < M * C) || (dq && bt.dq_stride < M * D) ||
                  (dk && bt.dk_stride < N * D) || (dv && bt.dv_stride < N * C)))
    return GS_ERR_BAD_SHAPE;
  if ((M > 0 && (!q || (grads && !dout))) || (N > 0 && (!k || !v))) return GS_ERR_NULL_POINTER;
  const int64_t vs = (int64_t)dsize(p->v_dtype), gsz = (int64_t)dsize(dout_dtype);
  // (strides count elements, so every problem's pointers keep the alignment
  // of the first one's)
  if ((M > 0 && (!aligned(q, ps) || (grads && !aligned(dout, gsz)))) ||
      (N > 0 && (!aligned(k, ps) || !aligned(v, vs))) || (out && !aligned(out, 4)) ||
      (dq && !aligned(dq, 4)) || (dk && !aligned(dk, 4)) || (dv && !aligned(dv, 4)))
    return GS_ERR_MISALIGNED;
  // operand spans over the whole batch
  auto span = [&](const void* base, int64_t stride, int64_t esize, int64_t elems) {
    return range_of(base, base ? ((cnt - 1) * stride + elems) * esize : 0);
  };
  const Range in[4] = {span(q, bt.q_stride, ps, M * D), span(k, bt.k_stride, ps, N * D),
                       span(v, bt.v_stride, vs, N * C),
                       span(grads ? dout : nullptr, bt.dout_stride, gsz, M * C)};
  const Range outs[4] = {span(out, bt.out_stride, 4, out ? M * C : 0),
                         span(dq, bt.dq_stride, 4, dq ? M * D : 0),
                         span(dk, bt.dk_stride, 4, dk ? N * D : 0),
                         span(dv, bt.dv_stride, 4, dv ? N * C : 0)};
  for (int a = 0; a < 4; ++a) {
    for (int c = 0; c < 4; ++c)
      if (overlap(outs[a], in[c])) return GS_ERR_ALIAS;
    for (int c = a + 1; c < 4; ++c)
      if (overlap(outs[a], outs[c])) return GS_ERR_ALIAS;
  }
  auto at_w = [](float* base, int64_t i, int64_t stride) -> float* {
    return base ? base + i * stride : nullptr;
  };
  if (M == 0 || N == 0) {
    // Empty sums: every requested output is zero.
    for (int64_t i = 0; i < cnt; ++i) {
      if (M > 0) {
        fill_zero(stream, at_w(out, i, bt.out_stride), M * C);
        fill_zero(stream, at_w(dq, i, bt.dq_stride), M * D);
      }
      if (N > 0) {
        fill_zero(stream, at_w(dk, i, bt.dk_stride), N * D);
        fill_zero(stream, at_w(dv, i, bt.dv_stride), N * C);
      }
    }
    return launch_status();
  }
  // the same array for q and k in every problem
  const bool alias = (q == k) && (M == N) && (cnt == 1 || bt.q_stride == bt.k_stride);
  Want w = want_for(*p, out != nullptr, dq != nullptr, dk != nullptr, dv != nullptr);
  if (p->qk_dtype == GS_F32) {
    if (!f32_pass_kernel(C, dims_of(D, C).DP)) return GS_ERR_INTERNAL;
  } else {
    // every kernel the passes below launch must exist for this shape
    const Dims dm = dims_of(D, C);
    if (((w.fwd && !w.fused()) || (w.dv && !w.fused_kv())) && !fwd_for(*p, dm).launch)
      return GS_ERR_INTERNAL;
    if (w.dq && !dq_for(*p, dm, w.fused()).launch) return GS_ERR_INTERNAL;
    if (w.dk && !dq_for(*p, dm, w.fused_kv()).launch) return GS_ERR_INTERNAL;
  }
  Plan pl;
  make_plan(*p, w, alias, nullptr, pl, 1);
  if ((st = check_workspace(workspace, workspace_bytes, pl.total)) != GS_SUCCESS) return st;
  const int64_t G = cnt > 1 ? group_size(*p, w, alias, cnt, workspace_bytes, pl) : 1;
  const Range rw = range_of(workspace, G * (int64_t)pl.total);
  for (int a = 0; a < 4; ++a)
    if (overlap(outs[a], rw) || overlap(in[a], rw)) return GS_ERR_ALIAS;
  make_plan(*p, w, alias, workspace, pl, G);

  // byte strides between problems
  const int64_t qs = bt.q_stride * ps, ks = bt.k_stride * ps, vst = bt.v_stride * vs,
                gst = bt.dout_stride * gsz, os = bt.out_stride * 4, dqs = bt.dq_stride * 4,
                dks = bt.dk_stride * 4, dvs = bt.dv_stride * 4;
  auto at = [](const void* base, int64_t i, int64_t bytes) -> const char* {
    return base ? static_cast<const char*>(base) + i * bytes : nullptr;
  };
  auto at_o = [](float* base, int64_t i, int64_t bytes) -> float* {
    return base ? reinterpret_cast<float*>(reinterpret_cast<char*>(base) + i * bytes) : nullptr;
  };
  const bool one_c = C == 1;
  const float tau2 = (float)(tau * 1.4426950408889634);
  for (int64_t g0 = 0; g0 < cnt; g0 += G) {
    Ctx c{stream, p, &pl, tau, tau2, (unsigned)std::min(G, cnt - g0), (int64_t)pl.total};
    const void* q_ = at(q, g0, qs);
    const void* k_ = at(k, g0, ks);
    const void* v_ = at(v, g0, vst);
    const void* g_ = grads ? at(dout, g0, gst) : nullptr;
    float* out_ = at_o(out, g0, os);
    float* dq_ = at_o(dq, g0, dqs);
    float* dk_ = at_o(dk, g0, dks);
    float* dv_ = at_o(dv, g0, dvs);
    if (p->qk_dtype == GS_F32) {
      run_f32(c, q_, qs, k_, ks, v_, vst, out_, os);
      continue;
    }
    if (small_forward(*p, w, pl, G)) {
      prep_fwd_small(c, q_, k_, v_, alias);
      row_check(c, pl.q, M, pl.Mp, pl.k, true, N);
      pass_fwd(c, pl.q, M, pl.k, N, pl.scal_kv, pl.v.ks, pl.slots + 0, out_, os);
      continue;
    }
    hipLaunchKernelGGL(k_fill_u32, grid_g(c, 1), dim3(64), 0, stream, pl.slots, 16, 0u, bz_ws(c));
    if (alias) {
      // q.ks serves dk (keys q, signs of dout) unless only dq wants a KS copy
      const bool q_for_dk = w.dk;
      prep_points(c, q_, qs, M, pl.Mp, pl.q, pl.slots + 2, one_c ? (q_for_dk ? g_ : v_) : nullptr,
                  q_for_dk ? dout_dtype : p->v_dtype, q_for_dk ? gst : vst);
      if (pl.k.ks != pl.q.ks)
        prep_points_ks(c, k_, ks, N, pl.Np, pl.k.ks, pl.slots + 2, v_, p->v_dtype, vst);
    } else {
      prep_points(c, q_, qs, M, pl.Mp, pl.q, pl.slots + 2, one_c && grads ? g_ : nullptr, dout_dtype, gst);
      prep_points(c, k_, ks, N, pl.Np, pl.k, pl.slots + 3, one_c ? v_ : nullptr, p->v_dtype, vst);
    }
    if (w.fwd || w.dq || w.dk) prep_values(c, v_, p->v_dtype, vst, N, pl.Np, pl.v, pl.slots + 0);
    // dout: its maximum scales the RT / KS copies (several channels, dv) and
    // enters the key scalars of passes keyed by q (dk, dv); a single-channel
    // dq reads dout exactly in its epilogue and needs none of it
    if (grads && (C > 1 || w.dk || w.dv)) prep_values(c, g_, dout_dtype, gst, M, pl.Mp, pl.g, pl.slots + 1);
    if (pl.scal_kv) prep_scalars(c, pl.k, v_, p->v_dtype, vst, N, pl.Np, pl.slots + 0, pl.scal_kv);
    if (pl.scal_qg) prep_scalars(c, pl.q, g_, dout_dtype, gst, M, pl.Mp, pl.slots + 1, pl.scal_qg);
    const uint32_t* kslot = alias ? pl.slots + 2 : pl.slots + 3;
    // full-sample row-bound flags for the forward-kernel passes (fwd, dv)
    if (w.fwd && !w.fused()) row_check(c, pl.q, M, pl.Mp, pl.k);
    if (w.dv && !w.fused_kv() && !(alias && w.fwd && !w.fused())) row_check(c, pl.k, N, pl.Np, pl.q);
    if (w.fwd && !w.fused()) pass_fwd(c, pl.q, M, pl.k, N, pl.scal_kv, pl.v.ks, pl.slots + 0, out_, os);
    if (w.dq)
      pass_dq(c, pl.q, M, pl.k, N, pl.scal_kv, kslot, pl.v.rt, pl.slots + 0, pl.g.rt, pl.slots + 1, g_,
              dout_dtype, gst, dq_, dqs, pl.v.ks, w.fused() ? out_ : nullptr, os);
    if (w.dk)
      pass_dq(c, pl.k, N, pl.q, M, pl.scal_qg, pl.slots + 2, pl.g.rt, pl.slots + 1, pl.v.rt,
              pl.slots + 0, v_, p->v_dtype, vst, dk_, dks, pl.g.ks, w.fused_kv() ? dv_ : nullptr, dvs);
    if (w.dv && !w.fused_kv()) pass_fwd(c, pl.k, N, pl.q, M, pl.scal_qg, pl.g.ks, pl.slots + 1, dv_, dvs);
  }
  return launch_status();
}

}  // namespace
}  // namespace gs

extern "C" {

size_t gauss_sum_fwd_workspace_size(const gs_problem* p) { return workspace_for(p, true, 0, 0, 0); }

gs_status gauss_sum_fwd_noalloc(const gs_problem* p, const void* q, const void* k, const void* v,
                                float tau, float* out, hipStream_t stream) {
  gs_status st = check_problem(p);
  if (st != GS_SUCCESS || (st = check_tau(tau)) != GS_SUCCESS) return st;
  const size_t need = workspace_for(p, true, 0, 0, 0);
  if (need > kScratchBytes) return GS_ERR_SCRATCH_LIMIT;
  void* ws = nullptr;
  if (need > 0 && (st = scratch_address(&ws)) != GS_SUCCESS) return st;
  return run(p, nullptr, q, k, v, tau, nullptr, GS_F32, out, nullptr, nullptr, nullptr, ws,
             need > 0 ? kScratchBytes : 0, stream);
}

size_t gauss_sum_bwd_workspace_size(const gs_problem* p, int want_dq, int want_dk, int want_dv) {
  if (!want_dq && !want_dk && !want_dv) return 0;
  return workspace_for(p, false, want_dq, want_dk, want_dv);
}

size_t gauss_sum_fwd_bwd_workspace_size(const gs_problem* p, int want_dq, int want_dk, int want_dv) {
  return workspace_for(p, true, want_dq, want_dk, want_dv);
}

gs_status gauss_sum_fwd(const gs_problem* p, const void* q, const void* k, const void* v, float tau,
                        float* out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  try {
    if (p && check_problem(p) == GS_SUCCESS && check_tau(tau) == GS_SUCCESS && p->M == 0)
      return GS_SUCCESS;
    if (!out && p) return GS_ERR_NULL_POINTER;
    return run(p, nullptr, q, k, v, tau, nullptr, GS_F32, out, nullptr, nullptr, nullptr, workspace,
               workspace_bytes, stream);
  } catch (...) {
    return GS_ERR_INTERNAL;
  }
}

gs_status gauss_sum_bwd(const gs_problem* p, const void* q, const void* k, const void* v, float tau,
                        const void* dout, int dout_dtype, float* dq, float* dk, float* dv,
                        void* workspace, size_t workspace_bytes, hipStream_t stream) {
  try {
    if (!dq && !dk && !dv) {
      gs_status st = check_problem(p);
      if (st != GS_SUCCESS) return st;
      if ((st = check_tau(tau)) != GS_SUCCESS) return st;
      return GS_ERR_NULL_POINTER;
    }
    return run(p, nullptr, q, k, v, tau, dout, dout_dtype, nullptr, dq, dk, dv, workspace,
               workspace_bytes, stream);
  } catch (...) {
    return GS_ERR_INTERNAL;
  }
}

gs_status gauss_sum_fwd_bwd(const gs_problem* p, const void* q, const void* k, const void* v,
                            float tau, const void* dout, int dout_dtype, float* out, float* dq,
                            float* dk, float* dv, void* workspace, size_t workspace_bytes,
                            hipStream_t stream) {
  try {
    if (!out) {
      gs_status st = check_problem(p);
      if (st != GS_SUCCESS) return st;
      if ((st = check_tau(tau)) != GS_SUCCESS) return st;
      return GS_ERR_NULL_POINTER;
    }
    return run(p, nullptr, q, k, v, tau, dout, dout_dtype, out, dq, dk, dv, workspace,
               workspace_bytes, stream);
  } catch (...) {
    return GS_ERR_INTERNAL;
  }
}

// SVGD: workspace = unit weights (N floats) and the query-gradient buffer
// (N x D floats), then room for the larger of the two passes.
}  // extern "C"

namespace gs {
namespace {

// Workspace of gauss_sum_svgd: the point-side arrays of a unit-weight dq
// pass (RT copy, half norms, KS copy, sample, key scalars), the KS copy of
// the scores, and the split partials of the one SVGD pass.
struct SvPlan {
  gs_problem p1;  // the problem with C = 1 (unit weights) whose plan holds the point side
  Plan pl;
  Dims dm;        // tiles for C = D
  SvK k;
  PassShape ps;
  uint16_t* score_ks = nullptr;
  float* part = nullptr;
  size_t total = 0;
};

void svgd_plan(const gs_problem& p, void* ws, SvPlan& sp) {
  sp.p1 = p;
  sp.p1.C = 1;
  sp.p1.v_dtype = GS_F32;
  make_plan(sp.p1, want_for(sp.p1, false, true, false, false), true, ws, sp.pl, 1);
  Carver cv;
  cv.base = static_cast<char*>(ws);
  cv.off = sp.pl.total;
  sp.dm = dims_of(p.D, p.D);
  sp.k = p.qk_dtype == GS_F16 ? sv_fn<F16>(sp.dm.DP, sp.dm.CT) : sv_fn<BF16>(sp.dm.DP, sp.dm.CT);
  sp.score_ks = cv.take<uint16_t>(sp.pl.Np * sp.dm.Rv() * 2);
  sp.ps = pass_shape(p.N, p.N, sv_qt(sp.dm.DP), sp.k.kernel, 1, dq_wpb(sp.dm.DP));
  sp.part = sp.ps.splits > 1 ? cv.take<float>((size_t)sp.ps.splits * p.N * p.D * 4) : nullptr;
  sp.total = cv.off;
}

}  // namespace
}  // namespace gs

extern "C" {

size_t gauss_sum_svgd_workspace_size(const gs_problem* p) {
  if (!p || gs::check_problem(p) != GS_SUCCESS || p->M != p->N || p->C != p->D ||
      p->qk_dtype == GS_F32 || p->N == 0)
    return 0;
  gs::SvPlan sp;
  gs::svgd_plan(*p, nullptr, sp);
  return sp.total;
}

// One pass over the pairs: k_dq in its SVGD mode forms the kernel values
// once and accumulates both the score sum (values = scores) and the unit-
// weight query gradient, and writes their difference.
gs_status gauss_sum_svgd(const gs_problem* p, const void* x, const void* score, float tau, float* phi,
                         void* workspace, size_t workspace_bytes, hipStream_t stream) {
  using namespace gs;
  try {
    gs_status st = check_problem(p);
    if (st != GS_SUCCESS) return st;
    if ((st = check_tau(tau)) != GS_SUCCESS) return st;
    if (p->M != p->N || p->C != p->D) return GS_ERR_BAD_SHAPE;
    if (p->qk_dtype == GS_F32) return GS_ERR_UNSUPPORTED;
    if (!phi) return GS_ERR_NULL_POINTER;
    const int64_t n = p->N, D = p->D;
    if (n > 0 && (!x || !score)) return GS_ERR_NULL_POINTER;
    if (!aligned(phi, 4) || (n > 0 && (!aligned(x, 2) || !aligned(score, dsize(p->v_dtype)))))
      return GS_ERR_MISALIGNED;
    if (n == 0) return GS_SUCCESS;
    SvPlan sp;
    svgd_plan(*p, nullptr, sp);
    if (!sp.k.launch) return GS_ERR_INTERNAL;
    if ((st = check_workspace(workspace, workspace_bytes, sp.total)) != GS_SUCCESS) return st;
    const Range in[3] = {range_of(x, n * D * 2), range_of(score, n * D * (int64_t)dsize(p->v_dtype)),
                         range_of(workspace, (int64_t)sp.total)};
    for (int b = 0; b < 3; ++b)
      if (overlap(range_of(phi, n * D * 4), in[b])) return GS_ERR_ALIAS;
    svgd_plan(*p, workspace, sp);
    Plan& pl = sp.pl;
    const float tau2 = (float)(tau * 1.4426950408889634);
    Ctx c{stream, &sp.p1, &pl, tau, tau2, 1u, (int64_t)pl.total};
    hipLaunchKernelGGL(k_fill_u32, dim3(1), dim3(64), 0, stream, pl.slots, 16, 0u, Bz{});
    // points: RT copy, half norms, sample, KS copy (plain: unit weights)
    prep_points(c, x, 0, n, pl.Mp, pl.q, pl.slots + 2);
    // scores: |max| and the KS copy (the values of the forward sum)
    hipLaunchKernelGGL(k_absmax, dim3(grid_reduce(n * D)), dim3(256), 0, stream, score, n * D,
                       (int)p->v_dtype, pl.slots + 0, Bz{});
    hipLaunchKernelGGL(k_values_ks, dim3(grid1(pl.Np / 8 * sp.dm.Rv())), dim3(256), 0, stream, score,
                       (int)p->v_dtype, n, (int)D, pl.Np, sp.dm.Rv(), (const uint32_t*)pl.slots + 0, 0,
                       sp.score_ks, Bz{});
    // key scalars: half norms only (unit weights)
    prep_scalars(c, pl.q, nullptr, GS_F32, 0, n, pl.Np, pl.slots + 0, pl.scal_kv);
    const PassShape& ps = sp.ps;
    const bool split = ps.splits > 1;
    prof_before(kKindGrad, stream);
    sp.k.launch(dim3(ps.blocks, ps.splits), stream, (const uint4*)pl.q.rt, pl.q.nh, (const uint4*)pl.q.samp_rt,
                pl.q.samp_nh, (const uint4*)pl.q.rt, pl.scal_kv, (const uint4*)pl.q.ks,
                p->qk_dtype == GS_BF16 ? pl.slots + 2 : nullptr, pl.slots + 0, tau2, tau, n, (int)D, ps.steps,
                ps.sps, split ? sp.part : phi, split ? n * D : 0, (const uint4*)sp.score_ks);
    prof_after(kKindGrad, stream);
    combine(c, ps, sp.part, n * D, phi, 0);
    return launch_status();
  } catch (...) {
    return GS_ERR_INTERNAL;
  }
}
size_t gauss_sum_mmd_flow_workspace_size(const gs_problem* p) {
  if (!p || gs::check_problem(p) != GS_SUCCESS || p->M != p->N || p->C != 1 || p->qk_dtype == GS_F32)
    return 0;
  return flow_extra(p->N) + gs::workspace_for(p, true, 1, 0, 0);
}

gs_status gauss_sum_mmd_flow(const gs_problem* p, const void* x, const void* v, float tau, float* s,
                             float* grad, double* mmd2, void* workspace, size_t workspace_bytes,
                             hipStream_t stream) {
  using namespace gs;
  try {
    gs_status st = check_problem(p);
    if (st != GS_SUCCESS) return st;
    if ((st = check_tau(tau)) != GS_SUCCESS) return st;
    if (p->M != p->N) return GS_ERR_BAD_SHAPE;
    if (p->C != 1 || p->qk_dtype == GS_F32) return GS_ERR_UNSUPPORTED;
    if (!s && !grad && !mmd2) return GS_ERR_NULL_POINTER;
    const int64_t n = p->N, D = p->D;
    if (n > 0 && (!x || !v)) return GS_ERR_NULL_POINTER;
    if (!aligned(mmd2, 8) || !aligned(s, 4) || !aligned(grad, 4)) return GS_ERR_MISALIGNED;
    const size_t need = gauss_sum_mmd_flow_workspace_size(p);
    if ((st = check_workspace(workspace, workspace_bytes, need)) != GS_SUCCESS) return st;
    // outputs overlap neither the inputs, the workspace nor each other (all
    // checked before anything is enqueued)
    const Range in[3] = {range_of(x, n * D * 2), range_of(v, n * (int64_t)dsize(p->v_dtype)),
                         range_of(workspace, (int64_t)need)};
    const Range outs[3] = {range_of(s, s ? n * 4 : 0), range_of(grad, grad ? n * D * 4 : 0),
                           range_of(mmd2, mmd2 ? 8 : 0)};
    for (int a = 0; a < 3; ++a) {
      for (int b = 0; b < 3; ++b)
        if (overlap(outs[a], in[b])) return GS_ERR_ALIAS;
      for (int b = a + 1; b < 3; ++b)
        if (overlap(outs[a], outs[b])) return GS_ERR_ALIAS;
    }
    char* base = static_cast<char*>(workspace);
    const int64_t a = round_up(std::max<int64_t>(n, 1) * 4, 256);
    float* ones = reinterpret_cast<float*>(base);
    float* sbuf = reinterpret_cast<float*>(base + a);
    double* parts = reinterpret_cast<double*>(base + 2 * a);
    const size_t extra = flow_extra(n);
    float* s_out = s ? s : (mmd2 ? sbuf : nullptr);
    if (n > 0) {
      if (grad) hipLaunchKernelGGL(k_fill_f32, dim3(grid1(n)), dim3(256), 0, stream, ones, n, 1.0f);
      st = run(p, nullptr, x, x, v, tau, grad ? ones : nullptr, GS_F32, s_out, grad, nullptr, nullptr,
               base + extra, workspace_bytes - extra, stream);
      if (st != GS_SUCCESS) return st;
    }
    if (mmd2) {
      hipLaunchKernelGGL(k_dot_partial, dim3(kDotBlocks), dim3(256), 0, stream, v, (int)p->v_dtype,
                         (const float*)s_out, n, parts);
      hipLaunchKernelGGL(k_dot_final, dim3(1), dim3(64), 0, stream, (const double*)parts, kDotBlocks,
                         mmd2);
    }
    return launch_status();
  } catch (...) {
    return GS_ERR_INTERNAL;
  }
}
size_t gauss_sum_fwd_batched_workspace_size(const gs_problem* p, int64_t count) {
  try {
    return workspace_for(p, true, 0, 0, 0, count);
  } catch (...) {
    return 0;
  }
}

size_t gauss_sum_bwd_batched_workspace_size(const gs_problem* p, int64_t count, int want_dq,
                                            int want_dk, int want_dv) {
  if (!want_dq && !want_dk && !want_dv) return 0;
  try {
    return workspace_for(p, false, want_dq, want_dk, want_dv, count);
  } catch (...) {
    return 0;
  }
}

gs_status gauss_sum_fwd_batched(const gs_problem* p, const gs_batch* batch, const void* q,
                                const void* k, const void* v, float tau, float* out,
                                void* workspace, size_t workspace_bytes, hipStream_t stream) {
  try {
    if (!batch) {
      gs_status st = check_problem(p);
      if (st != GS_SUCCESS) return st;
      if ((st = check_tau(tau)) != GS_SUCCESS) return st;
      return GS_ERR_NULL_POINTER;
    }
    return run(p, batch, q, k, v, tau, nullptr, GS_F32, out, nullptr, nullptr, nullptr, workspace,
               workspace_bytes, stream);
  } catch (...) {
    return GS_ERR_INTERNAL;
  }
}

gs_status gauss_sum_bwd_batched(const gs_problem* p, const gs_batch* batch, const void* q,
                                const void* k, const void* v, float tau, const void* dout,
                                int dout_dtype, float* dq, float* dk, float* dv,
                                void* workspace, size_t workspace_bytes, hipStream_t stream) {
  try {
    if (!batch) {
      gs_status st = check_problem(p);
      if (st != GS_SUCCESS) return st;
      if ((st = check_tau(tau)) != GS_SUCCESS) return st;
      return GS_ERR_NULL_POINTER;
    }
    return run(p, batch, q, k, v, tau, dout, dout_dtype, nullptr, dq, dk, dv, workspace,
               workspace_bytes, stream);
  } catch (...) {
    return GS_ERR_INTERNAL;
  }
}

size_t gauss_sum_fwd_bwd_batched_workspace_size(const gs_problem* p, int64_t count, int want_dq,
                                                int want_dk, int want_dv) {
  try {
    return workspace_for(p, true, want_dq, want_dk, want_dv, count);
  } catch (...) {
    return 0;
  }
}
gs_status gauss_sum_fwd_bwd_batched(const gs_problem* p, const gs_batch* batch, const void* q,
                                    const void* k, const void* v, float tau, const void* dout,
                                    int dout_dtype, float* out, float* dq, float* dk, float* dv,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream) {
  try {
    if (!batch || (!out && batch->count > 0)) {
      gs_status st = check_problem(p);
      if (st != GS_SUCCESS) return st;
      if ((st = check_tau(tau)) != GS_SUCCESS) return st;
      return GS_ERR_NULL_POINTER;
    }
    return run(p, batch, q, k, v, tau, dout, dout_dtype, out, dq, dk, dv, workspace,
               workspace_bytes, stream);
  } catch (...) {
    return GS_ERR_INTERNAL;
  }
}
}  // extern "C"
