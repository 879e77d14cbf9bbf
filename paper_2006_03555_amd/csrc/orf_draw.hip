// orf_draw.hip - orthogonal random features (Sec. 2.4, R-ORFs) drawn on the GPU.
//
// One workgroup per (d x d block, head). Random numbers come from Philox4x64-10
// (Salmon, Moraes, Dror, Shaw, SC'11) with key (seed, 0) and counter
// (index, head, purpose, 0); each call gives eight 32-bit words (low then high
// half of each 64-bit output), u = (x + 0.5) 2^-32, and Gaussians by the
// Box-Muller transform of consecutive uniform pairs.
//
// Four threads own one row of the block, 16 consecutive elements each, held in
// fp64 registers from the Gaussian draw to the final store. The rows are
// orthogonalised in order by modified Gram-Schmidt: when row j is final, its
// owners publish it into its own LDS slot and raise a ready flag; every later
// row then removes its component along row j (quad-local dot products; the
// readers also form ||row j||^2 from the same loads). Waves wait on the flags of the rows they need
// rather than on workgroup barriers, so the work of rows far from the next
// pivot overlaps the chain of pivots. A wave waits only for rows owned by
// itself (published earlier in its own program order) or by lower waves, so
// every flag is raised and every wave finishes; a bounded spin makes that hold
// even if it did not. Rows stay unnormalised during the sweep and are
// normalised at the store. The triangular factor of row Gram-Schmidt has a
// positive diagonal, so the result is the unique orthogonal factor. Rows are
// then scaled by chi_d norms (independent Gaussian vectors) or sqrt(d) and
// rounded to fp32.
#include <type_traits>

#include "favor_common.hpp"
#include "kernels.hpp"

namespace favor {

namespace {
constexpr uint64_t kPhM0 = 0xD2E7470EE14C6C93ull;
constexpr uint64_t kPhM1 = 0xCA5A826395121157ull;
constexpr uint64_t kPhW0 = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kPhW1 = 0xBB67AE8584CAA73Bull;
constexpr int kOrfD = 64;
}  // namespace

__device__ __forceinline__ void philox4x64_10(uint64_t c[4], uint64_t k0, uint64_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t hi0 = __umul64hi(kPhM0, c[0]);
    const uint64_t lo0 = kPhM0 * c[0];
    const uint64_t hi1 = __umul64hi(kPhM1, c[2]);
    const uint64_t lo1 = kPhM1 * c[2];
    const uint64_t n0 = hi1 ^ c[1] ^ k0;
    const uint64_t n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
    if (r < 9) {
      k0 += kPhW0;
      k1 += kPhW1;
    }
  }
}

// Eight uniforms of call `idx` of stream (seed, head, purpose).
__device__ __forceinline__ void uniforms8(uint64_t seed, uint32_t head, uint32_t purpose,
                                          uint64_t idx, float u[8]) {
  uint64_t c[4] = {idx, head, purpose, 0};
  philox4x64_10(c, seed, 0);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t lo = (uint32_t)c[j];
    const uint32_t hi = (uint32_t)(c[j] >> 32);
    u[2 * j] = fmaf((float)lo, 0x1p-32f, 0x1p-33f);
    u[2 * j + 1] = fmaf((float)hi, 0x1p-32f, 0x1p-33f);
  }
}

__device__ __forceinline__ void gaussians8(uint64_t seed, uint32_t head, uint32_t purpose,
                                           uint64_t idx, float z[8]) {
  float u[8];
  uniforms8(seed, head, purpose, idx, u);
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const float r = sqrtf(-2.0f * logf(u[2 * p]));
    float sn, cs;
    sincospif(2.0f * u[2 * p + 1], &sn, &cs);
    z[2 * p] = r * cs;
    z[2 * p + 1] = r * sn;
  }
}

// Sum over the four lanes of an aligned quad (DPP quad permutes, no LDS traffic).
__device__ __forceinline__ double quad_sum(double v) {
  auto perm = [](double x, auto ctrl_tag) {
    constexpr int ctrl = decltype(ctrl_tag)::value;
    const long long b = __double_as_longlong(x);
    const int lo = __builtin_amdgcn_mov_dpp((int)b, ctrl, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_mov_dpp((int)(b >> 32), ctrl, 0xF, 0xF, false);
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
  };
  v += perm(v, std::integral_constant<int, 0xB1>{});   // quad_perm(1,0,3,2): lane ^ 1
  v += perm(v, std::integral_constant<int, 0x4E>{});   // quad_perm(2,3,0,1): lane ^ 2
  return v;
}

__global__ __launch_bounds__(256) void k_orf_draw(uint64_t seed, int M, int kind,
                                                  float *__restrict__ W, float *__restrict__ b) {
  constexpr int D = kOrfD;             // 64 rows of 64; thread = (row, quarter)
  __shared__ double pub[D][D];         // finished rows, one slot each
  __shared__ int ready[D];             // row j published

  const int blk = blockIdx.x;
  const int h = blockIdx.y;
  const int tid = threadIdx.x;
  const int r = tid >> 2;              // row within the block
  const int p = tid & 3;               // elements 16 p .. 16 p + 15 of the row
  const uint64_t m = (uint64_t)blk * D + r;   // feature index of the row
  if (tid < D) ready[tid] = 0;

  // Gaussian block: element (blk D + r) D + c comes from call ((blk D + r) D + c) / 8
  double x[16];
  {
    float z[8];
    gaussians8(seed, h, 0, m * (D / 8) + 2 * p, z);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = (double)z[i];
    gaussians8(seed, h, 0, m * (D / 8) + 2 * p + 1, z);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[8 + i] = (double)z[i];
  }
  // chi_d norm of row m: elements m D .. m D + D - 1 (calls m D / 8 + q, q < 8)
  double rho = 8.0;                    // sqrt(64) for the fixed-norm kind
  if (kind == 0) {
    double ss = 0.0;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      float z[8];
      gaussians8(seed, h, 1, m * (D / 8) + 2 * p + q, z);
#pragma unroll
      for (int i = 0; i < 8; ++i) ss = fma((double)z[i], (double)z[i], ss);
    }
    rho = sqrt(quad_sum(ss));
  }
  // phases: element m = blk D + i
  if (tid < D / 8) {
    float u[8];
    uniforms8(seed, h, 2, (uint64_t)blk * (D / 8) + tid, u);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int mm = blk * D + tid * 8 + i;
      if (mm < M) b[(size_t)h * M + mm] = 6.283185307179586f * u[i];
    }
  }

  double scale = 1.0;
  __syncthreads();                     // flags cleared
  if (kind != 2) {
    // owners of row j publish it (data, then the flag); readers form its squared
    // norm themselves from the same loads, which keeps the norm and its
    // reciprocal off the owner's side of the chain
    auto publish = [&](int j) {
      double *dst = &pub[j][16 * p];
#pragma unroll
      for (int i = 0; i < 16; i += 2) *(double2 *)(dst + i) = make_double2(x[i], x[i + 1]);
      if (p == 0)
        __hip_atomic_store(&ready[j], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    };
    if (r == 0) publish(0);
    // a wave holds rows 16 w .. 16 w + 15; the last step that changes one of them is
    // j = 16 w + 14
    const int last = (tid >> 6) * 16 + 15;
    for (int j = 0; j < last; ++j) {
      for (int spin = 0; spin < (1 << 22); ++spin)
        if (__hip_atomic_load(&ready[j], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP)) break;
      const double *src = &pub[j][16 * p];
      double q[16];
#pragma unroll
      for (int i = 0; i < 16; i += 2) {
        const double2 v = *(const double2 *)(src + i);
        q[i] = v.x;
        q[i + 1] = v.y;
      }
      double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
      double n0 = 0.0, n1 = 0.0, n2 = 0.0, n3 = 0.0;
#pragma unroll
      for (int i = 0; i < 16; i += 4) {
        a0 = fma(x[i], q[i], a0);
        a1 = fma(x[i + 1], q[i + 1], a1);
        a2 = fma(x[i + 2], q[i + 2], a2);
        a3 = fma(x[i + 3], q[i + 3], a3);
        n0 = fma(q[i], q[i], n0);
        n1 = fma(q[i + 1], q[i + 1], n1);
        n2 = fma(q[i + 2], q[i + 2], n2);
        n3 = fma(q[i + 3], q[i + 3], n3);
      }
      const double dot = quad_sum((a0 + a1) + (a2 + a3));
      const double nq = quad_sum((n0 + n1) + (n2 + n3));
      // 1 / ||row j||^2: hardware reciprocal refined by two Newton steps
      double inv = __builtin_amdgcn_rcp(nq);
      inv = inv * fma(-nq, inv, 2.0);
      inv = inv * fma(-nq, inv, 2.0);
      const double c = (r > j) ? dot * inv : 0.0;   // rows up to j are final
#pragma unroll
      for (int i = 0; i < 16; ++i) x[i] = fma(-c, q[i], x[i]);
      if (r == j + 1) publish(j + 1);
    }
    double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
#pragma unroll
    for (int i = 0; i < 16; i += 4) {
      s0 = fma(x[i], x[i], s0);
      s1 = fma(x[i + 1], x[i + 1], s1);
      s2 = fma(x[i + 2], x[i + 2], s2);
      s3 = fma(x[i + 3], x[i + 3], s3);
    }
    const double nrm2 = quad_sum((s0 + s1) + (s2 + s3));
    scale = rho / sqrt(nrm2);
  }

  if ((int)m < M) {
    float4* dst = (float4 *)(W + ((size_t)h * M + m) * D + 16 * p);
#pragma unroll
    for (int i = 0; i < 16; i += 4)
      dst[i / 4] = make_float4((float)(x[i] * scale), (float)(x[i + 1] * scale),
                               (float)(x[i + 2] * scale), (float)(x[i + 3] * scale));
  }
}

hipError_t launch_orf_draw(uint64_t seed, int n_heads, int M, int kind, float *W, float *b,
                           hipStream_t st) {
  dim3 grid((M + kOrfD - 1) / kOrfD, n_heads);
  hipLaunchKernelGGL(k_orf_draw, grid, dim3(256), 0, st, seed, M, kind, W, b);
  return hipGetLastError();
}

}  // namespace favor
