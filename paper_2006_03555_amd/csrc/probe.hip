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

}  // namespace
}  // namespace favor

extern "C" {

FAVOR_API double favor_probe_work(int32_t kind, int32_t iters) {
  using namespace favor;
  const double waves = (double)kProbeCus * kProbeBlocksPerCu * (kProbeThreads / 64);
  if (iters <= 0) return 0.0;
  if (kind == 0) return waves * iters * kMfmaChains * (16.0 * 16.0 * 32.0 * 2.0);
  if (kind == 1) return waves * 64.0 * iters * kCosChains;
  return 0.0;
}

FAVOR_API favor_status favor_probe(int32_t kind, int32_t iters, float *sink,
                                   hipStream_t stream) {
  using namespace favor;
  if ((kind != 0 && kind != 1) || iters <= 0 || !sink)
    return report(FAVOR_ERR_INVALID_ARGUMENT, "favor_probe: kind 0 or 1, iters > 0, sink");
  const dim3 grid(kProbeCus * kProbeBlocksPerCu);
  if (kind == 0)
    hipLaunchKernelGGL(k_probe_mfma, grid, dim3(kProbeThreads), 0, stream, iters,
                       sink);
  else
    hipLaunchKernelGGL(k_probe_cos, grid, dim3(kProbeThreads), 0, stream, iters,
                       sink);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? FAVOR_OK : report(FAVOR_ERR_DEVICE, hipGetErrorString(e));
}

}  // extern "C"
