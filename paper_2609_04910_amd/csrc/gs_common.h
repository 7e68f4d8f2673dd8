// gs_common.h -- types, MFMA wrappers and the operand layouts shared by the
// Gauss-sum kernels (gfx950 / CDNA4).
//
// Every kernel works in the transposed tile orientation S^T[n][m] = k_n . q_m
// (keys on the MFMA row index, queries on the column index), so that the
// 16x16 fp32 result tile of one v_mfma_f32_16x16x32 already has the register
// layout of the B operand of the next contraction over keys.  Lane l of a
// wave64 holds, for the 16x16x32 MFMA:
//     A operand: A[i = l%16][k = 8*(l/16) .. +7]      (8 x 16-bit)
//     B operand: B[k = 8*(l/16) .. +7][j = l%16]      (8 x 16-bit)
//     result   : D[i = 4*(l/16) + r][j = l%16], r = 0..3 (4 x fp32)
//
// Operand storage in the workspace (all 16-byte loads, fully coalesced):
//
//   Row-tile layout "RT" for a matrix X (rows x W, W padded to a multiple of
//   32): element (r, w) lives at half-index
//       ((r/16 * (W/32) + w/32) * 16 + r%16) * 32 + w%32 ,
//   so the 16 x 32 block needed by one MFMA operand is one contiguous 1 KiB
//   run, and lane (i = l%16, g = l/16) reads 16 bytes at
//       (((t * W/32 + c) * 16 + i) * 4 + g)   in 16-byte units,
//   for row tile t and column chunk c.  Used for the contraction over D
//   (points) and over C (values, upstream gradient).
//
//   Key-slot layout "KS" for a matrix Y (keys x R, R padded to 16): used as
//   the A operand of a contraction over keys (V^T for P.V, K^T for P.K).  A
//   32-key step s holds R rows of 32 halves; row w, slot z stores key
//       s*32 + 16*((z%8)/4) + 4*(z/8) + z%4
//   which is exactly the key the B operand (built from two S^T result tiles)
//   carries in k-slot z.  Lane (i, g) reads 16 bytes at ((s*R + w0 + i)*4 + g).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gs {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kBlockThreads = kWave * kWavesPerBlock;
constexpr int kStep = 32;      // keys per inner step
constexpr int kRowPad = 512;   // row padding of every point / value array (one workgroup of 8-tile waves)
constexpr float kPadBias = -1.0e30f;  // -||k||^2/2 of a padding row: Phi = 0
constexpr int kSampleCoarse = 64;     // keys of the first row-bound check
constexpr int kSampleRows = 1024;     // keys of the second (and all sampled rows)

struct F16 {
  typedef _Float16 storage;
  static __device__ __forceinline__ float to_float(uint16_t b) {
    return (float)__builtin_bit_cast(_Float16, b);
  }
};
struct BF16 {
  typedef __bf16 storage;
  static __device__ __forceinline__ float to_float(uint16_t b) {
    return __builtin_bit_cast(float, (uint32_t)b << 16);
  }
};

template <typename T>
__device__ __forceinline__ floatx4 mfma_qk(uint4 a, uint4 b, floatx4 c);
template <>
__device__ __forceinline__ floatx4 mfma_qk<F16>(uint4 a, uint4 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8, a),
                                                __builtin_bit_cast(half8, b), c, 0, 0, 0);
}
template <>
__device__ __forceinline__ floatx4 mfma_qk<BF16>(uint4 a, uint4 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ floatx4 mfma_f16(uint4 a, uint4 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8, a),
                                                __builtin_bit_cast(half8, b), c, 0, 0, 0);
}

// exp2 of the exponent, clamped to [0, 1] (folds into v_exp_f32 ... clamp):
// the clamp is the "exponent <= 0" guarantee, so fp32 cancellation in the
// expanded exponent can never produce a kernel value above 1.
__device__ __forceinline__ float exp2_clamped(float x) {
  return __builtin_amdgcn_fmed3f(__builtin_amdgcn_exp2f(x), 0.0f, 1.0f);
}

typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef _Float16 halfx2 __attribute__((ext_vector_type(2)));

// Two fp32 -> one dword of two fp16, round to nearest even (one v_cvt_pk_f16_f32).
__device__ __forceinline__ uint32_t pack_f16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{lo, hi}, halfx2));
}

// Register fences for operands loaded from global memory before a key loop.
// The direct HBM -> LDS copies of the loops are inline assembly, which the
// compiler does not count in its memory-counter bookkeeping: if the first
// use of a prologue load sits inside the loop, the compiler's wait for it
// there ("at most n loads outstanding", n counting only its own loads)
// executes on every step and also waits for most of the step's own
// prefetch.  An empty assembly statement that reads and writes the register
// is such a use, placed before the loop, so the wait happens there once.
__device__ __forceinline__ void settle(float& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void settle(uint4& x) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  u32x4 t = __builtin_bit_cast(u32x4, x);
  asm volatile("" : "+v"(t));
  x = __builtin_bit_cast(uint4, t);
}
template <typename T, int A, int B>
__device__ __forceinline__ void settle(T (&x)[A][B]) {
#pragma unroll
  for (int a = 0; a < A; ++a)
#pragma unroll
    for (int b = 0; b < B; ++b) settle(x[a][b]);
}
template <typename T, int A>
__device__ __forceinline__ void settle(T (&x)[A]) {
#pragma unroll
  for (int a = 0; a < A; ++a) settle(x[a]);
}

// Element i of an fp32 / fp16 / bf16 array (dtype codes of gs_dtype: 0, 1, 2).
__device__ __forceinline__ float load_any(const void* p, int64_t i, int dtype) {
  if (dtype == 0) return static_cast<const float*>(p)[i];
  uint16_t b = static_cast<const uint16_t*>(p)[i];
  return dtype == 1 ? F16::to_float(b) : BF16::to_float(b);
}

// Power-of-two scale exponent e with max * 2^e in [1, 2); 0 for max = 0, Inf or NaN.
__device__ __forceinline__ int scale_exponent(uint32_t max_bits) {
  float mx = __builtin_bit_cast(float, max_bits);
  if (!(mx > 0.0f) || !(mx < __builtin_inff())) return 0;
  int e;
  (void)frexpf(mx, &e);  // mx = f * 2^e, f in [0.5, 1)
  return 1 - e;
}

// Exponent of the scale of the fp16 KS copy of bf16 points (the operand of
// the gradient contraction): the largest magnitude lands in [2^14, 2^15), so
// coordinates down to 2^-28 of it keep fp16's full 11 bits.  Scaled to
// [1, 2), as the values are, coordinates below 2^-14 of the largest fell
// into fp16 subnormals, and where such a coordinate of q nearly equals the
// same coordinate of k the difference q - k, which the gradient sums, lost
// its leading bits.
constexpr int kPointScaleHeadroom = 14;
__device__ __forceinline__ int point_scale_exponent(uint32_t max_bits) {
  return scale_exponent(max_bits) + kPointScaleHeadroom;
}

// Per-problem byte strides of a launch over a batch of problems: problem
// blockIdx.z finds each operand at its base + blockIdx.z * stride.  One
// problem: all zero, gridDim.z = 1.
struct Bz {
  int64_t ws = 0;    // the problem's workspace slice (every derived operand)
  int64_t in = 0;    // the caller's input array the kernel reads
  int64_t in2 = 0;   // a second caller input (sign source of a KS copy, exact upstream gradient)
  int64_t out = 0;   // output: the caller's array, or the partial sums in the workspace
  int64_t out2 = 0;  // second output (forward sum of a fused gradient pass)
};

// p advanced to problem blockIdx.z (NULL stays NULL).
template <typename P>
__device__ __forceinline__ const P* zoff(const P* p, int64_t stride) {
  return p ? reinterpret_cast<const P*>(reinterpret_cast<const char*>(p) + (int64_t)blockIdx.z * stride)
           : p;
}
template <typename P>
__device__ __forceinline__ P* zoff(P* p, int64_t stride) {
  return p ? reinterpret_cast<P*>(reinterpret_cast<char*>(p) + (int64_t)blockIdx.z * stride) : p;
}

// RT-layout half index of element (r, w) for a matrix with W (multiple of 32) columns.
__host__ __device__ __forceinline__ int64_t rt_index(int64_t r, int w, int W) {
  return (((r >> 4) * (W >> 5) + (w >> 5)) * 16 + (r & 15)) * 32 + (w & 31);
}
// KS-layout half index of element (key r, row w) for R (multiple of 16) rows.
__host__ __device__ __forceinline__ int64_t ks_index(int64_t r, int w, int R) {
  int o = (int)(r & 31);
  int z = 8 * ((o & 15) >> 2) + 4 * (o >> 4) + (o & 3);
  return ((r >> 5) * R + w) * 32 + z;
}

}  // namespace gs
