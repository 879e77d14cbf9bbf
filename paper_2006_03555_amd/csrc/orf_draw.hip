// orf_draw.hip - orthogonal random features (Sec. 2.4, R-ORFs) drawn on the GPU.
//
// One workgroup per (d x d block, head). Random numbers come from Philox4x64-10
// (Salmon, Moraes, Dror, Shaw, SC'11) with key (seed, 0) and counter
// (index, head, purpose, 0); each call gives eight 32-bit words (low then high
// half of each 64-bit output), u = (x + 0.5) 2^-32, and Gaussians by the
// Box-Muller transform of consecutive uniform pairs. The Gaussian block is
// orthonormalised row by row with classical Gram-Schmidt applied twice per row
// ("twice is enough", which keeps fp32 rows orthogonal to rounding level);
// the triangular factor of row Gram-Schmidt has a positive diagonal, so the
// result is the unique orthogonal factor. Rows are then scaled by chi_d norms
// (independent Gaussian vectors) or sqrt(d).
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

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__global__ __launch_bounds__(256) void k_orf_draw(uint64_t seed, int M, int kind,
                                                  float *__restrict__ W, float *__restrict__ b) {
  constexpr int D = kOrfD;
  __shared__ float G[D][D + 1];
  __shared__ float Qm[D][D + 1];
  __shared__ float rho[D];
  __shared__ float r[D];
  __shared__ float coef[D];

  const int blk = blockIdx.x;
  const int h = blockIdx.y;
  const int tid = threadIdx.x;

  // Gaussian block: element n = (blk D + row) D + col, call n / 8
  for (int ci = tid; ci < D * D / 8; ci += 256) {
    float z[8];
    gaussians8(seed, h, 0, (uint64_t)blk * (D * D / 8) + ci, z);
    const int n0 = ci * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) G[n0 / D][n0 % D + i] = z[i];
  }
  // chi_d norms: row m = blk D + rr uses elements m D .. m D + D - 1 (8 calls)
  for (int ci = tid; ci < D * D / 8; ci += 256) {
    const int rr = ci >> 3;
    const int q = ci & 7;
    const uint64_t m = (uint64_t)blk * D + rr;
    float z[8];
    gaussians8(seed, h, 1, m * (D / 8) + q, z);
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) ss = fmaf(z[i], z[i], ss);
    ss += __shfl_xor(ss, 1);
    ss += __shfl_xor(ss, 2);
    ss += __shfl_xor(ss, 4);
    if (q == 0) rho[rr] = sqrtf(ss);
  }
  // phases: element m = blk D + rr
  if (tid < D / 8) {
    float u[8];
    uniforms8(seed, h, 2, (uint64_t)blk * (D / 8) + tid, u);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int m = blk * D + tid * 8 + i;
      if (m < M) b[(size_t)h * M + m] = 6.283185307179586f * u[i];
    }
  }
  __syncthreads();

  if (kind == 2) {  // IID: raw Gaussian rows
    for (int idx = tid; idx < D * D; idx += 256) {
      const int rr = idx / D;
      const int m = blk * D + rr;
      if (m < M) W[((size_t)h * M + m) * D + idx % D] = G[rr][idx % D];
    }
    return;
  }

  for (int i = 0; i < D; ++i) {
    if (tid < D) r[tid] = G[i][tid];
    __syncthreads();
    for (int pass = 0; pass < 2; ++pass) {
      {  // coef_j = q_j . r, four threads per j
        const int j = tid >> 2;
        const int part = tid & 3;
        float acc = 0.f;
        if (j < i) {
#pragma unroll
          for (int cc = 0; cc < 16; ++cc) acc = fmaf(Qm[j][part * 16 + cc], r[part * 16 + cc], acc);
        }
        acc += __shfl_xor(acc, 1);
        acc += __shfl_xor(acc, 2);
        if (part == 0) coef[j] = acc;
      }
      __syncthreads();
      {  // r_c -= sum_{j < i} coef_j q_j[c], four threads per c
        const int c = tid >> 2;
        const int part = tid & 3;
        float acc = 0.f;
        for (int j = part; j < i; j += 4) acc = fmaf(coef[j], Qm[j][c], acc);
        acc += __shfl_xor(acc, 1);
        acc += __shfl_xor(acc, 2);
        if (part == 0) r[c] -= acc;
      }
      __syncthreads();
    }
    if (tid < D) {
      const float v = r[tid];
      const float n2 = wave_sum(v * v);
      Qm[i][tid] = v / sqrtf(n2);
    }
    __syncthreads();
  }

  for (int idx = tid; idx < D * D; idx += 256) {
    const int rr = idx / D;
    const int m = blk * D + rr;
    if (m < M) {
      const float sc = (kind == 0) ? rho[rr] : 8.0f;  // sqrt(64)
      W[((size_t)h * M + m) * D + idx % D] = Qm[rr][idx % D] * sc;
    }
  }
}

hipError_t launch_orf_draw(uint64_t seed, int n_heads, int M, int kind, float *W, float *b,
                           hipStream_t st) {
  dim3 grid((M + kOrfD - 1) / kOrfD, n_heads);
  hipLaunchKernelGGL(k_orf_draw, grid, dim3(256), 0, st, seed, M, kind, W, b);
  return hipGetLastError();
}

}  // namespace favor
