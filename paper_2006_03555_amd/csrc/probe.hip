// probe.hip - measurement probes for the roofline report: the rates this GPU
// reaches on the two compute resources the FAVOR kernels are bound by, the
// bf16 matrix cores (v_mfma_f32_16x16x32_bf16) and the transcendental unit
// (v_cos_f32), so that achieved figures can be read against measured peaks as
// well as the published ones. Not part of the method.
#include <hip/hip_runtime.h>

#include "../../include/favor.h"
#include "favor_common.hpp"
#include "kernels.hpp"

namespace favor {
namespace {

constexpr int kProbeThreads = 256;       // four waves per workgroup
constexpr int kProbeBlocksPerCu = 2;     // two waves per SIMD
constexpr int kProbeCus = 256;
constexpr int kMfmaChains = 8;           // independent accumulators per wave
constexpr int kCosChains = 8;            // independent cosine chains per lane

// Every wave issues iters x kMfmaChains independent 16x16x32 bf16 MFMAs.
__global__ __launch_bounds__(kProbeThreads) void k_probe_mfma(int iters, float *sink) {
  const int l = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (bf16)(1e-3f * (float)(l + i));
    b[i] = (bf16)(1e-3f * (float)(64 - l + i));
  }
  f32x4 c[kMfmaChains];
#pragma unroll
  for (int k = 0; k < kMfmaChains; ++k) c[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int k = 0; k < kMfmaChains; ++k) c[k] = Mma<bf16>::mma(a, b, c[k]);
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < kMfmaChains; ++k) s += c[k][0] + c[k][1] + c[k][2] + c[k][3];
  if (s == 1234.5f) sink[blockIdx.x] = s;   // keeps the work; never true for these inputs
}

// Every lane evaluates iters x kCosChains hardware cosines (revolutions), in
// independent chains whose arguments stay within a few revolutions.
__global__ __launch_bounds__(kProbeThreads) void k_probe_cos(int iters, float *sink) {
  float x[kCosChains];
#pragma unroll
  for (int k = 0; k < kCosChains; ++k) x[k] = 1e-3f * (float)(threadIdx.x + 7 * k);
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int k = 0; k < kCosChains; ++k) x[k] = __builtin_amdgcn_cosf(x[k]);
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < kCosChains; ++k) s += x[k];
  if (s == 1234.5f) sink[blockIdx.x] = s;
}

// The structured alternative to a dense projection for H-ORF features: every
// lane holds one token's 64-vector and applies, per 64-row block of M = 256,
// sqrt(d) H D3 H D2 H D1 (three unnormalised Walsh-Hadamard transforms of 64
// points, six butterfly stages each, and three sign diagonals) in registers,
// iters tokens per lane. The result is folded into a checksum: the probe times
// the arithmetic alone, without the feature epilogue or any memory traffic.
constexpr int kFwhtBlocks = 4;           // M / d for M = 256, d = 64
__device__ __forceinline__ void fwht64_lane(float (&v)[64]) {
#pragma unroll
  for (int h = 1; h < 64; h <<= 1)
#pragma unroll
    for (int i = 0; i < 64; ++i)
      if ((i & h) == 0) {
        const float a = v[i], c = v[i + h];
        v[i] = a + c;
        v[i + h] = a - c;
      }
}
__global__ __launch_bounds__(kProbeThreads) void k_probe_fwht(int iters, float *sink) {
  const uint32_t lane = threadIdx.x;
  float acc = 0.f;
  for (int it = 0; it < iters; ++it) {
    float x[64];
#pragma unroll
    for (int i = 0; i < 64; ++i) x[i] = 1e-3f * (float)((lane + 3 * i + it) & 255);
#pragma unroll 1
    for (int blk = 0; blk < kFwhtBlocks; ++blk) {
      float v[64];
#pragma unroll
      for (int i = 0; i < 64; ++i) v[i] = x[i];
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const uint32_t signs = 0x9E3779B9u * (uint32_t)(3 * blk + t + 1) ^ lane;
#pragma unroll
        for (int i = 0; i < 64; ++i) v[i] = ((signs >> (i & 31)) & 1u) ? -v[i] : v[i];
        fwht64_lane(v);
      }
#pragma unroll
      for (int i = 0; i < 64; ++i) acc += v[i];
    }
  }
  if (acc == 1234.5f) sink[blockIdx.x] = acc;
}

}  // namespace
}  // namespace favor

extern "C" {

FAVOR_API double favor_probe_work(int32_t kind, int32_t iters) {
  using namespace favor;
  const double waves = (double)kProbeCus * kProbeBlocksPerCu * (kProbeThreads / 64);
  if (iters <= 0) return 0.0;
  if (kind == 0) return waves * iters * kMfmaChains * (16.0 * 16.0 * 32.0 * 2.0);
  if (kind == 1) return waves * 64.0 * iters * kCosChains;
  if (kind == 2) return waves * 64.0 * iters;   // tokens projected onto M = 256 H-ORF rows
  return 0.0;
}

FAVOR_API favor_status favor_probe(int32_t kind, int32_t iters, float *sink,
                                   hipStream_t stream) {
  using namespace favor;
  if (kind < 0 || kind > 2 || iters <= 0 || !sink)
    return report(FAVOR_ERR_INVALID_ARGUMENT, "favor_probe: kind 0, 1 or 2, iters > 0, sink");
  const dim3 grid(kProbeCus * kProbeBlocksPerCu);
  if (kind == 0)
    hipLaunchKernelGGL(k_probe_mfma, grid, dim3(kProbeThreads), 0, stream, iters,
                       sink);
  else if (kind == 1)
    hipLaunchKernelGGL(k_probe_cos, grid, dim3(kProbeThreads), 0, stream, iters,
                       sink);
  else
    hipLaunchKernelGGL(k_probe_fwht, grid, dim3(kProbeThreads), 0, stream, iters, sink);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? FAVOR_OK : report(FAVOR_ERR_DEVICE, hipGetErrorString(e));
}

}  // extern "C"
