// favor_common.hpp - device building blocks shared by the FAVOR kernels.
//
// Matrix-core conventions (CDNA3/CDNA4 16x16 MFMA tiles, wave64):
//   A operand [16 rows x K]:  lane l holds row (l % 16)
//   B operand [K x 16 cols]:  lane l holds col (l % 16)
//   C/D       [16 x 16] fp32: lane l holds col (l % 16), rows 4*(l/16) + j, j = 0..3
// A "k32 fragment" is one lane's share of a 32-deep slice of K: 8 values. The
// eight k positions a lane holds are paired with the same eight positions of
// the other operand, so any bijection between (lane group g = l/16, slot i)
// and the 32 logical k indices is valid as long as both operands use it.
//
// Two bijections are used:
//   loaded   slot i of group g  <->  k = 8 g + i          (16 contiguous bytes)
//   chained  slot i of group g  <->  k = 16 (i / 4) + 4 g + (i % 4)
// "Chained" is the k order in which two vertically adjacent 16x16 accumulator
// tiles already sit in a lane (rows 4g+j of tile 0, then of tile 1), so an MFMA
// result can feed the next MFMA as its k operand without moving data across
// lanes. Tables written for an operand that meets a chained one (the value
// tile C~, the state, Buf1) are stored in chained order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace favor {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;
constexpr float kInv2Pi = 0.15915494309189535f;

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// Policy for the matrix-core element type T (the type of Q, K, V).
template <typename T> struct Mma;

// bf16 inputs: v_mfma_f32_16x16x32_bf16, bf16 features, hardware cosine.
template <> struct Mma<bf16> {
  using frag = bf16x8;
  static constexpr int kFragBytes = 16;
  __device__ __forceinline__ static f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  __device__ __forceinline__ static frag pack(f32x4 lo, f32x4 hi) {
    frag r;
    r[0] = (bf16)lo[0]; r[1] = (bf16)lo[1]; r[2] = (bf16)lo[2]; r[3] = (bf16)lo[3];
    r[4] = (bf16)hi[0]; r[5] = (bf16)hi[1]; r[6] = (bf16)hi[2]; r[7] = (bf16)hi[3];
    return r;
  }
  __device__ __forceinline__ static frag from_f32(const float *v, float s) {
    frag r;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = (bf16)(v[i] * s);
    return r;
  }
  __device__ __forceinline__ static frag splat(float v) {
    frag r;
    bf16 h = (bf16)v;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = h;
    return r;
  }
  // cos(2 pi x), sin(2 pi x): v_cos_f32 / v_sin_f32 take revolutions.
  __device__ __forceinline__ static float cos_rev(float x) { return __builtin_amdgcn_cosf(x); }
  __device__ __forceinline__ static float sin_rev(float x) { return __builtin_amdgcn_sinf(x); }
};

// fp32 inputs: eight v_mfma_f32_16x16x4_f32 per k32 fragment (slot i = k-step i),
// fp32 features, accurately rounded cosine.
template <> struct Mma<float> {
  using frag = f32x8;
  static constexpr int kFragBytes = 32;
  __device__ __forceinline__ static f32x4 mma(frag a, frag b, f32x4 c) {
#pragma unroll
    for (int i = 0; i < 8; ++i) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[i], c, 0, 0, 0);
    return c;
  }
  __device__ __forceinline__ static frag pack(f32x4 lo, f32x4 hi) {
    frag r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
  }
  __device__ __forceinline__ static frag from_f32(const float *v, float s) {
    frag r;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = v[i] * s;
    return r;
  }
  __device__ __forceinline__ static frag splat(float v) {
    frag r;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = v;
    return r;
  }
  __device__ __forceinline__ static float cos_rev(float x) { return cospif(2.0f * x); }
  __device__ __forceinline__ static float sin_rev(float x) { return sinpif(2.0f * x); }
};

// ---- element conversions ---------------------------------------------------
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }
__device__ __forceinline__ float to_f32(float v) { return v; }

// Sum of squares of the 16 values of two fragments (a lane's share of a row):
// bf16 pairs go through the dot2 instruction (two exact products and an fp32
// sum per instruction, no conversions); fp32 values through fused multiply-adds.
__device__ __forceinline__ float sq_sum16(const bf16x8 (&f)[2]) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  struct Pairs { bf16x2 p[4]; };
  float n = 0.f;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const Pairs q = __builtin_bit_cast(Pairs, f[k]);
#pragma unroll
    for (int i = 0; i < 4; ++i) n = __builtin_amdgcn_fdot2_f32_bf16(q.p[i], q.p[i], n, false);
  }
  return n;
}
__device__ __forceinline__ float sq_sum16(const f32x8 (&f)[2]) {
  float n = 0.f;
#pragma unroll
  for (int k = 0; k < 2; ++k)
#pragma unroll
    for (int i = 0; i < 8; ++i) n = fmaf(f[k][i], f[k][i], n);
  return n;
}
template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }

// Load 8 consecutive elements starting at p as a fragment (16 B bf16, 32 B fp32).
template <typename T>
__device__ __forceinline__ typename Mma<T>::frag load_frag(const T *p) {
  return *reinterpret_cast<const typename Mma<T>::frag *>(p);
}
template <typename T>
__device__ __forceinline__ void store_frag(T *p, typename Mma<T>::frag v) {
  *reinterpret_cast<typename Mma<T>::frag *>(p) = v;
}

// Load 8 consecutive elements and widen to fp32.
__device__ __forceinline__ void load8_f32(const bf16 *p, float *v) {
  bf16x8 x = *reinterpret_cast<const bf16x8 *>(p);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (float)x[i];
}
__device__ __forceinline__ void load8_f32(const float *p, float *v) {
  f32x4 a = *reinterpret_cast<const f32x4 *>(p);
  f32x4 b = *reinterpret_cast<const f32x4 *>(p + 4);
  v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
  v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
}

// Store 4 consecutive output elements from fp32 values.
__device__ __forceinline__ void store4(bf16 *p, f32x4 v) {
  bf16x4 r;
  r[0] = (bf16)v[0]; r[1] = (bf16)v[1]; r[2] = (bf16)v[2]; r[3] = (bf16)v[3];
  *reinterpret_cast<bf16x4 *>(p) = r;
}
__device__ __forceinline__ void store4(float *p, f32x4 v) { *reinterpret_cast<f32x4 *>(p) = v; }

// Eight consecutive output elements from two fp32 quadruples.
__device__ __forceinline__ void store8(bf16 *p, f32x4 a, f32x4 b) {
  bf16x8 r;
  r[0] = (bf16)a[0]; r[1] = (bf16)a[1]; r[2] = (bf16)a[2]; r[3] = (bf16)a[3];
  r[4] = (bf16)b[0]; r[5] = (bf16)b[1]; r[6] = (bf16)b[2]; r[7] = (bf16)b[3];
  *reinterpret_cast<bf16x8 *>(p) = r;
}
__device__ __forceinline__ void store8(float *p, f32x4 a, f32x4 b) {
  *reinterpret_cast<f32x4 *>(p) = a;
  *reinterpret_cast<f32x4 *>(p + 4) = b;
}

// Feature kernels (Sec. 2.2, Eq. interesting): the epilogue applied to a
// projection p = W'' x + b'' whose accumulator was seeded with the row's b''.
// kCos: cos(2 pi p) (W'' and b'' carry 1/2 pi; the D_X sqrt(2/M) factor is
// applied, or cancelled, outside). kRelu: ReLU(W'' x) + kernel_eps, computed as
// max(p, b'') with b'' = kernel_eps (W'' carries s / sqrt(M), no D_X factor).
//
// Rows past the M features drawn (the kernels work on 64, 128 or 256 rows) have
// W'' = 0 and the seed seed_row gives them: a quarter revolution for cos
// features (cos(pi/2), zero up to the hardware cosine's error, which enters the
// products only squared) and 0 for ReLU features (max(0, 0) = 0 exactly), so
// they add nothing to any aggregate.
constexpr int kCos = 0;
constexpr int kRelu = 1;
template <int KN, typename P>
__device__ __forceinline__ float feature(float p, float seed) {
  if constexpr (KN == kRelu) {
    return fmaxf(p, seed);
  } else {
    return P::cos_rev(p);
  }
}

// Derivative factor of a feature with respect to its projection, up to the
// constant the caller folds in: kCos: sin(2 pi p) (d cos / d theta = -sin);
// kRelu: the step [W'' x > 0] = [p > seed] (0 at W'' x = 0).
template <int KN, typename P>
__device__ __forceinline__ float feature_slope(float p, float seed) {
  if constexpr (KN == kRelu) {
    return p > seed ? 1.f : 0.f;
  } else {
    return P::sin_rev(p);
  }
}

// b'' of feature row m of M_r drawn rows: the phase b_m bs (cos) or kernel_eps
// (ReLU); rows m >= M_r are padding (see above).
template <int KN>
__device__ __forceinline__ float seed_row(int m, int Mr, const float *__restrict__ b, float bs,
                                          float keps) {
  if (m >= Mr) return KN == kRelu ? 0.f : 0.25f;
  return KN == kRelu ? keps : b[m] * bs;
}

// Value-column order of the output-side operands (Buf1^T fragments, the causal
// value tiles and state): row r of 16-column block nb is value column
//   pi(nb, r) = 32 (nb / 2) + 8 (r / 4) + 4 (nb % 2) + r % 4,
// so that a lane holding rows 4 g .. 4 g + 3 of output blocks 2 p and 2 p + 1
// holds the eight consecutive columns 32 p + 8 g .. 32 p + 8 g + 7 (one 16-byte
// store in bf16).
__device__ __forceinline__ int perm_col(int nb, int r) {
  return 32 * (nb >> 1) + 8 * (r >> 2) + 4 * (nb & 1) + (r & 3);
}

// Chained slot of logical k index r in [0, 32): k = 16 h + 4 g + i'  ->  (g, slot 4h + i').
__device__ __forceinline__ int chained_group(int r) { return (r & 15) >> 2; }
__device__ __forceinline__ int chained_slot(int r) { return ((r >> 4) << 2) | (r & 3); }

}  // namespace favor
