// orf_draw.hip - orthogonal random features (Sec. 2.4, R-ORFs) drawn on the GPU.
//
// One workgroup per (d x d block, head). Random numbers come from Philox4x64-10
// (Salmon, Moraes, Dror, Shaw, SC'11) with key (seed, 0) and counter
// (index, head, purpose, 0); each call gives eight 32-bit words (low then high
// half of each 64-bit output), u = (x + 0.5) 2^-32, and Gaussians by the
// Box-Muller transform of consecutive uniform pairs. The Gaussian block is
// orthogonalised row by row with classical Gram-Schmidt in fp64: one pass per
// row suffices there (the loss of orthogonality grows like cond^2 * 1e-16),
// and rows are kept unnormalised during the sweep (coefficients divide by the
// squared norms, each formed by the threads that project onto that row next),
// so that each row costs two barrier-separated phases with quad-local sums;
// all rows are normalised at the end. The triangular factor of row
// Gram-Schmidt has a positive diagonal, so the result is the unique orthogonal
// factor. Rows are then scaled by chi_d norms (independent Gaussian vectors) or
// sqrt(d) and rounded to fp32.
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
  constexpr int D = kOrfD;
  constexpr int RS = D + 2;            // fp64 row stride (16-byte aligned rows; 2-way banks)
  __shared__ double R[D][RS];          // rows: Gaussian block, orthogonalised in place
  __shared__ double RT[D][RS];         // the same block column-major, for column sums
  __shared__ double dots[D];           // <R_j, R_i> / ||R_j||^2 for the current row i
  __shared__ double nrm2[D];           // ||R_j||^2 of finished rows
  __shared__ float rho[D];

  const int blk = blockIdx.x;
  const int h = blockIdx.y;
  const int tid = threadIdx.x;

  // Gaussian block: element n = (blk D + row) D + col, call n / 8
  for (int ci = tid; ci < D * D / 8; ci += 256) {
    float z[8];
    gaussians8(seed, h, 0, (uint64_t)blk * (D * D / 8) + ci, z);
    const int n0 = ci * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      R[n0 / D][n0 % D + i] = (double)z[i];
      RT[n0 % D + i][n0 / D] = (double)z[i];
    }
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
      if (m < M) W[((size_t)h * M + m) * D + idx % D] = (float)R[rr][idx % D];
    }
    return;
  }

  const int q4 = tid >> 2;    // row (phase 1) or column (phase 2) owned by 4 threads
  const int part = tid & 3;   // quarter of the 64-long sum
  for (int i = 0; i <= D; ++i) {
    // phase 1: coefficients <R_j, R_i> / ||R_j||^2 for the finished rows j < i. The four
    // threads of row i - 1 also form ||R_{i-1}||^2 (its last use of the previous step).
    // Loads are unconditional and in bounds so that they issue together.
    if (q4 < i) {
      const int ic = min(i, D - 1);
      double a0 = 0.0, a1 = 0.0, n0 = 0.0, n1 = 0.0;
#pragma unroll
      for (int cc = 0; cc < 16; cc += 2) {
        const double x0 = R[q4][part * 16 + cc];
        const double x1 = R[q4][part * 16 + cc + 1];
        a0 = fma(x0, R[ic][part * 16 + cc], a0);
        a1 = fma(x1, R[ic][part * 16 + cc + 1], a1);
        n0 = fma(x0, x0, n0);
        n1 = fma(x1, x1, n1);
      }
      const double a = quad_sum(a0 + a1);
      const double nn = quad_sum(n0 + n1);
      if (part == 0) {
        // 1 / ||R_j||^2: hardware reciprocal refined by two Newton steps
        double r = __builtin_amdgcn_rcp(nn);
        r = r * fma(-nn, r, 2.0);
        r = r * fma(-nn, r, 2.0);
        if (q4 == i - 1) nrm2[q4] = nn;
        dots[q4] = a * r;
      }
    }
    __syncthreads();
    if (i == D) break;
    // phase 2: R_i[c] -= sum_{j < i} coef_j * R_j[c] for column c = q4;
    // thread part p sums j in [16 p, 16 p + 16) (coefficients of rows j >= i masked)
    {
      double a0 = 0.0, a1 = 0.0;
      const int j0 = part * 16;
#pragma unroll
      for (int jj = 0; jj < 16; jj += 2) {
        const int j = j0 + jj;
        const double c0 = (j < i) ? dots[j] : 0.0;
        const double c1 = (j + 1 < i) ? dots[j + 1] : 0.0;
        a0 = fma(c0, RT[q4][j], a0);
        a1 = fma(c1, RT[q4][j + 1], a1);
      }
      const double a = quad_sum(a0 + a1);
      if (part == 0) {
        const double v = R[i][q4] - a;
        R[i][q4] = v;
        RT[q4][i] = v;
      }
    }
    __syncthreads();
  }

  for (int idx = tid; idx < D * D; idx += 256) {
    const int rr = idx / D;
    const int m = blk * D + rr;
    if (m < M) {
      const double sc = (kind == 0 ? (double)rho[rr] : 8.0) / sqrt(nrm2[rr]);  // 8 = sqrt(64)
      W[((size_t)h * M + m) * D + idx % D] = (float)(R[rr][idx % D] * sc);
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
