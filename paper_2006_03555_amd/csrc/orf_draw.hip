// orf_draw.hip - orthogonal random features (Sec. 2.4: R-ORFs, and the
// Hadamard / Givens H/G-ORFs at the end of the file) drawn on the GPU.
//
// One workgroup per (d x d block, head). Random numbers come from Philox4x64-10
// (Salmon, Moraes, Dror, Shaw, SC'11) with key (seed, 0) and counter
// (index, head, purpose, 0); each call gives eight 32-bit words (low then high
// half of each 64-bit output), u = (x + 0.5) 2^-32, and Gaussians by the
// Box-Muller transform of consecutive uniform pairs.
//
// Eight threads own one row of the block, 8 consecutive elements each (one
// generator call), held in fp64 registers from the Gaussian draw to the final
// store; wave w holds the panel of rows 8 w .. 8 w + 7. The rows are
// orthogonalised in order by modified Gram-Schmidt. Inside a panel the pivot
// chain stays in its wave: the owners of the final row j write it to its LDS
// slot and the wave reads it back (no flag: a wavefront-scope fence orders the
// stores before the loads and one wave's LDS accesses complete in order), then
// removes its component from its later rows. Each row is also published
// to the later waves by a ready flag; they remove the earlier panels' rows two
// at a time as the flags come up. Removing two orthogonal rows at once is the
// same projection as removing them one after the other. Dot products and norms
// are 8-lane sums on the DPP network. A wave waits only for flags of lower
// waves, so every flag is raised and every wave finishes; a bounded spin makes
// that hold even if it did not. Rows stay unnormalised during the sweep and
// are normalised at the store. The triangular factor of row Gram-Schmidt has
// a positive diagonal, so the result is the unique orthogonal factor. Rows are
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

// Sum over the eight lanes of an aligned group (DPP: swap within pairs, within
// quads, then mirror within the half-row; no LDS traffic).
__device__ __forceinline__ double sum8(double v) {
  auto perm = [](double x, auto ctrl_tag) {
    constexpr int ctrl = decltype(ctrl_tag)::value;
    const long long b = __double_as_longlong(x);
    const int lo = __builtin_amdgcn_mov_dpp((int)b, ctrl, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_mov_dpp((int)(b >> 32), ctrl, 0xF, 0xF, false);
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
  };
  v += perm(v, std::integral_constant<int, 0xB1>{});    // quad_perm(1,0,3,2): lane ^ 1
  v += perm(v, std::integral_constant<int, 0x4E>{});    // quad_perm(2,3,0,1): lane ^ 2
  v += perm(v, std::integral_constant<int, 0x141>{});   // row_half_mirror: lane 7 - i
  return v;
}

// Row j's eight doubles of lane part p, from its LDS slot.
__device__ __forceinline__ void read_row(const double *src, double (&q)[8]) {
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const double2 v = *(const double2 *)(src + i);
    q[i] = v.x;
    q[i + 1] = v.y;
  }
}

// x . q and q . q over a row held by an aligned group of eight lanes.
__device__ __forceinline__ void dot_and_norm(const double (&x)[8], const double (&q)[8],
                                             double &dot, double &nq) {
  double a0 = 0.0, a1 = 0.0, n0 = 0.0, n1 = 0.0;
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    a0 = fma(x[i], q[i], a0);
    a1 = fma(x[i + 1], q[i + 1], a1);
    n0 = fma(q[i], q[i], n0);
    n1 = fma(q[i + 1], q[i + 1], n1);
  }
  dot = sum8(a0 + a1);
  nq = sum8(n0 + n1);
}

// 1 / v: hardware reciprocal refined by two Newton steps.
__device__ __forceinline__ double recip(double v) {
  double inv = __builtin_amdgcn_rcp(v);
  inv = inv * fma(-v, inv, 2.0);
  return inv * fma(-v, inv, 2.0);
}

// Orders this wave's LDS stores before its later LDS loads across lanes (a
// wavefront-scope release/acquire pair around a wave barrier: no instructions,
// but the compiler may not move another lane's load above the store).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ bool flag_set(const int *f) {
  return __hip_atomic_load(f, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) != 0;
}
// Bounded wait for a row's flag: true once it is set. The bound only keeps a
// wave from spinning forever should a flag never come up; the caller then
// poisons its row (NaN), so such a failure shows in W instead of passing.
__device__ __forceinline__ bool wait_flag(const int *f) {
  for (int spin = 0; spin < (1 << 22); ++spin)
    if (flag_set(f)) return true;
  return false;
}

__global__ __launch_bounds__(512) void k_orf_draw(uint64_t seed, int M, int kind,
                                                  float *__restrict__ W, float *__restrict__ b) {
  constexpr int D = kOrfD;             // 64 rows of 64; thread = (row, eighth)
  constexpr int RW = 8;                // rows per wave (one panel)
  __shared__ double pub[D][D];         // finished rows, one slot each
  __shared__ int ready[D];             // row j published

  const int blk = blockIdx.x;
  const int h = blockIdx.y;
  const int tid = threadIdx.x;
  const int w = tid >> 6;              // wave = panel of rows 8 w .. 8 w + 7
  const int r = tid >> 3;              // row within the block
  const int p = tid & 7;               // elements 8 p .. 8 p + 7 of the row
  const uint64_t m = (uint64_t)blk * D + r;   // feature index of the row
  constexpr int kLastWave = D / RW - 1;
  if (tid < D) ready[tid] = 0;
  __syncthreads();                     // flags cleared before any wave publishes

  // Gaussian block: element (blk D + r) D + c comes from call ((blk D + r) D + c) / 8,
  // so the eight elements of this lane are exactly call m D / 8 + p
  double x[8];
  {
    float z[8];
    gaussians8(seed, h, 0, m * (D / 8) + p, z);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = (double)z[i];
  }
  // chi_d norm of row m (elements m D .. m D + D - 1, calls m D / 8 + p) and
  // the phases (element m = blk D + i): work off the pivot chain, done by the
  // last panel's wave while it waits for the earlier panels and by the others
  // after their own panel.
  double rho = 8.0;                    // sqrt(64) for the fixed-norm kind
  auto side_work = [&]() __attribute__((always_inline)) {
    if (kind == 0) {
      float z[8];
      gaussians8(seed, h, 1, m * (D / 8) + p, z);
      double ss = 0.0;
#pragma unroll
      for (int i = 0; i < 8; ++i) ss = fma((double)z[i], (double)z[i], ss);
      rho = sqrt(sum8(ss));
    }
    if (w == kLastWave && (tid & 63) < D / 8) {
      const int k = tid & 63;
      float u[8];
      uniforms8(seed, h, 2, (uint64_t)blk * (D / 8) + k, u);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int mm = blk * D + k * 8 + i;
        if (mm < M) b[(size_t)h * M + mm] = 6.283185307179586f * u[i];
      }
    }
  };

  double scale = 1.0;
  if (kind == 2) {
    side_work();
  } else {
    if (w == kLastWave) side_work();
    // Earlier panels' rows, two at a time as their owners publish them (each
    // owner raises its flags in order, each after its row's data, so the second
    // flag covers both rows). The two rows are orthogonal, so removing both
    // components at once is the same projection (modified Gram-Schmidt in
    // blocks of two).
    bool published = true;
    for (int j0 = 0; j0 < RW * w; j0 += 2) {
      published = wait_flag(&ready[j0 + 1]) && published;
      double q0[8], q1[8];
      read_row(&pub[j0][8 * p], q0);
      read_row(&pub[j0 + 1][8 * p], q1);
      double d0, n0, d1, n1;
      dot_and_norm(x, q0, d0, n0);
      dot_and_norm(x, q1, d1, n1);
      const double c0 = d0 * recip(n0);
      const double c1 = d1 * recip(n1);
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = fma(-c1, q1[i], fma(-c0, q0[i], x[i]));
    }
    // This wave's panel: row j is final once rows up to j - 1 are removed. Its
    // owners write it to its slot and the whole wave reads it back (ordered by a
    // wavefront-scope fence; no flag is needed inside the wave); the flag for
    // the later panels is raised after the read is issued.
    for (int jj = 0; jj < RW; ++jj) {
      const int j = RW * w + jj;
      double *slot = &pub[j][8 * p];
      if (r == j) {
#pragma unroll
        for (int i = 0; i < 8; i += 2) *(double2 *)(slot + i) = make_double2(x[i], x[i + 1]);
      }
      if (jj == RW - 1) {
        if (r == j && p == 0)
          __hip_atomic_store(&ready[j], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        break;
      }
      wave_sync();   // the owners' stores before every lane's loads
      double q[8];
      read_row(slot, q);
      if (r == j && p == 0)
        __hip_atomic_store(&ready[j], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
      double dot, nq;
      dot_and_norm(x, q, dot, nq);
      const double cj = (r > j) ? dot * recip(nq) : 0.0;   // rows up to j are final
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = fma(-cj, q[i], x[i]);
    }
    if (w != kLastWave) side_work();
    double s0 = 0.0, s1 = 0.0;
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
      s0 = fma(x[i], x[i], s0);
      s1 = fma(x[i + 1], x[i + 1], s1);
    }
    scale = rho / sqrt(sum8(s0 + s1));
    if (!published) scale = __builtin_nan("");
  }

  if ((int)m < M) {
    float4 *dst = (float4 *)(W + ((size_t)h * M + m) * D + 8 * p);
    dst[0] = make_float4((float)(x[0] * scale), (float)(x[1] * scale), (float)(x[2] * scale),
                         (float)(x[3] * scale));
    dst[1] = make_float4((float)(x[4] * scale), (float)(x[5] * scale), (float)(x[6] * scale),
                         (float)(x[7] * scale));
  }
}

// ---------------------------------------------------------------------------
// Structured orthogonal blocks (Sec. 2.4 (2)). Rows have norm sqrt(d); the
// phases are drawn as for the other kinds.

// The eight 32-bit words of call idx of stream (seed, head, purpose).
__device__ __forceinline__ void words8(uint64_t seed, uint32_t head, uint32_t purpose,
                                       uint64_t idx, uint32_t x[8]) {
  uint64_t c[4] = {idx, head, purpose, 0};
  philox4x64_10(c, seed, 0);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    x[2 * j] = (uint32_t)c[j];
    x[2 * j + 1] = (uint32_t)(c[j] >> 32);
  }
}

__device__ __forceinline__ void store_phases(uint64_t seed, int h, int blk, int M,
                                             float *__restrict__ b) {
  const int k = threadIdx.x;   // 8 threads, 8 phases each
  float u[8];
  uniforms8(seed, h, 2, (uint64_t)blk * (kOrfD / 8) + k, u);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int mm = blk * kOrfD + k * 8 + i;
    if (mm < M) b[(size_t)h * M + mm] = 6.283185307179586f * u[i];
  }
}

// Unnormalised Walsh-Hadamard transform of a 64-vector held by an aligned group
// of eight lanes (lane p: elements 8 p .. 8 p + 7), natural (Sylvester) order.
__device__ __forceinline__ void fwht64(double (&v)[8], int p) {
#pragma unroll
  for (int s = 1; s < 8; s <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if ((e & s) == 0) {
        const double a = v[e], c = v[e + s];
        v[e] = a + c;
        v[e + s] = a - c;
      }
#pragma unroll
  for (int m = 1; m < 8; m <<= 1) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const double o = __shfl_xor(v[e], m);
      v[e] = (p & m) ? o - v[e] : v[e] + o;
    }
  }
}

// H-ORF: row r of block blk is sqrt(d) e_r^T H D3 H D2 H D1 (normalised
// Sylvester-Hadamard H, Rademacher diagonals from stream 3: element
// (3 blk + t) d + c is +1 when its word is below 2^31). 512 threads: eight per row.
__global__ __launch_bounds__(512) void k_orf_hadamard(uint64_t seed, int M,
                                                      float *__restrict__ W,
                                                      float *__restrict__ b) {
  constexpr int D = kOrfD;
  const int blk = blockIdx.x;
  const int h = blockIdx.y;
  const int tid = threadIdx.x;
  const int r = tid >> 3;
  const int p = tid & 7;
  double sg[3][8];
#pragma unroll
  for (int t = 0; t < 3; ++t) {
    uint32_t x[8];
    words8(seed, h, 3, (uint64_t)(3 * blk + t) * (D / 8) + p, x);
#pragma unroll
    for (int e = 0; e < 8; ++e) sg[t][e] = x[e] < 0x80000000u ? 1.0 : -1.0;
  }
  double v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {   // (row r of H) o d3, H[r][c] = (-1)^popcount(r & c) / 8
    const int c = 8 * p + e;
    v[e] = ((__popc(r & c) & 1) ? -0.125 : 0.125) * sg[2][e];
  }
  fwht64(v, p);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] *= 0.125 * sg[1][e];
  fwht64(v, p);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] *= 0.125 * sg[0][e] * 8.0;   // times sqrt(d)
  const int m = blk * D + r;
  if (m < M) {
    float4 *dst = (float4 *)(W + ((size_t)h * M + m) * D + 8 * p);
    dst[0] = make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
    dst[1] = make_float4((float)v[4], (float)v[5], (float)v[6], (float)v[7]);
  }
  if (tid < D / 8) store_phases(seed, h, blk, M, b);
}

// G-ORF: block blk is sqrt(d) G_1 ... G_K, K = 2 d log2 d rotations; rotation t
// comes from call blk K + t of stream 4 (words x0, x1, x2): i = (x0 d) >> 32,
// j' = (x1 (d - 1)) >> 32, j = j' + [j' >= i], theta = 2 pi (x2 + 0.5) 2^-32, and
// acts on row vectors as v_i <- c v_i + s v_j, v_j <- -s v_i + c v_j. The
// parameters go to LDS first (all threads); then thread r rotates row r of the
// identity through the K rotations in order, in fp64 in LDS.
constexpr int kGivensK = 2 * kOrfD * 6;
__global__ __launch_bounds__(256) void k_orf_givens(uint64_t seed, int M, float *__restrict__ W,
                                                    float *__restrict__ b) {
  constexpr int D = kOrfD;
  constexpr int K = kGivensK;
  __shared__ double cs[K][2];
  __shared__ unsigned char pi[K], pj[K];
  __shared__ double rows[D][D + 1];
  const int blk = blockIdx.x;
  const int h = blockIdx.y;
  const int tid = threadIdx.x;
  for (int t = tid; t < K; t += blockDim.x) {
    uint32_t x[8];
    words8(seed, h, 4, (uint64_t)blk * K + t, x);
    const int i = (int)(((uint64_t)x[0] * D) >> 32);
    const int jp = (int)(((uint64_t)x[1] * (D - 1)) >> 32);
    const double th = 6.283185307179586 * (((double)x[2] + 0.5) * 0x1p-32);
    double sn, cn;
    sincos(th, &sn, &cn);
    pi[t] = (unsigned char)i;
    pj[t] = (unsigned char)(jp + (jp >= i ? 1 : 0));
    cs[t][0] = cn;
    cs[t][1] = sn;
  }
  for (int e = tid; e < D * D; e += blockDim.x) rows[e / D][e % D] = (e / D == e % D) ? 1.0 : 0.0;
  __syncthreads();
  if (tid < D) {
    double *v = rows[tid];
    for (int t = 0; t < K; ++t) {
      const int i = pi[t], j = pj[t];
      const double c = cs[t][0], s = cs[t][1];
      const double vi = v[i], vj = v[j];
      v[i] = fma(c, vi, s * vj);
      v[j] = fma(-s, vi, c * vj);
    }
  }
  __syncthreads();
  // rows * sqrt(d) -> W, 16-byte stores (thread = (row, eighth))
  for (int e = tid; e < D * 8; e += blockDim.x) {
    const int r = e >> 3, q = e & 7;
    const int m = blk * D + r;
    if (m < M) {
      const double *v = &rows[r][8 * q];
      float4 *dst = (float4 *)(W + ((size_t)h * M + m) * D + 8 * q);
      dst[0] = make_float4((float)(8.0 * v[0]), (float)(8.0 * v[1]), (float)(8.0 * v[2]),
                           (float)(8.0 * v[3]));
      dst[1] = make_float4((float)(8.0 * v[4]), (float)(8.0 * v[5]), (float)(8.0 * v[6]),
                           (float)(8.0 * v[7]));
    }
  }
  if (tid < D / 8) store_phases(seed, h, blk, M, b);
}

hipError_t launch_orf_draw(uint64_t seed, int n_heads, int M, int kind, float *W, float *b,
                           hipStream_t st) {
  dim3 grid((M + kOrfD - 1) / kOrfD, n_heads);
  if (kind == 3)
    hipLaunchKernelGGL(k_orf_hadamard, grid, dim3(512), 0, st, seed, M, W, b);
  else if (kind == 4)
    hipLaunchKernelGGL(k_orf_givens, grid, dim3(256), 0, st, seed, M, W, b);
  else
    hipLaunchKernelGGL(k_orf_draw, grid, dim3(512), 0, st, seed, M, kind, W, b);
  return hipGetLastError();
}

}  // namespace favor
