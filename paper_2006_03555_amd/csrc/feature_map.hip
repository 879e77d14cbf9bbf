// feature_map.hip - the random-feature map X' = D_X X-hat (Sec. 2.3, Eqs. dqdk
// and qkprime) materialised in HBM.
//
// One workgroup handles 64 * TBW rows of one head; the projection W'' x is a
// matrix-core product in transposed orientation (result lane = row, 4
// consecutive features per lane), seeded with b'' so the epilogue is
// cos(2 pi acc) * D_X(row) * sqrt(2/M) followed by a 4-element store. The
// kernel is bound by writing X' (M elements per row against d read).
#include "favor_common.hpp"
#include "kernels.hpp"
#include "tile_common.hpp"

namespace favor {

template <typename T> struct FmapCfg { static constexpr int TBW = 4; };
template <> struct FmapCfg<float> { static constexpr int TBW = 2; };

template <typename T, typename To, int M>
__global__ __launch_bounds__(256) void k_feature_map(const T *__restrict__ X,
                                                     const float *__restrict__ W,
                                                     const float *__restrict__ bph,
                                                     To *__restrict__ Xp, int H, int L, float s,
                                                     int ntiles) {
  constexpr int TBW = FmapCfg<T>::TBW;
  using P = Mma<T>;
  using frag = typename P::frag;
  __shared__ frag WA[M / 16][2][64];
  __shared__ float bq[M];

  const int item = xcd_item(blockIdx.x, gridDim.x);
  const int bh = item / ntiles;
  const int tile = item - bh * ntiles;
  const int h = bh % H;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;

  fill_w_afrags<T, M>(WA, bq, W + (size_t)h * M * kD, bph + (size_t)h * M, s * kInv2Pi);

  const int rbase = tile * (64 * TBW) + w * (16 * TBW);
  const T *Xh = X + (size_t)bh * L * kD;
  frag xf[TBW][2];
  float dfac[TBW];
  const float cM = sqrtf(2.0f / M);
#pragma unroll
  for (int tb = 0; tb < TBW; ++tb) {
    const int t = rbase + tb * 16 + c16;
    float nrm = 0.f;
    if (t < L) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        xf[tb][ks] = load_frag<T>(Xh + (size_t)t * kD + ks * 32 + 8 * g);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float x = to_f32(xf[tb][ks][i]);
          nrm = fmaf(x, x, nrm);
        }
      }
    } else {
      xf[tb][0] = P::splat(0.f);
      xf[tb][1] = P::splat(0.f);
    }
    nrm += __shfl_xor(nrm, 16);
    nrm += __shfl_xor(nrm, 32);
    dfac[tb] = cM * expf(0.5f * s * s * nrm);
  }
  __syncthreads();

  To *Oh = Xp + (size_t)bh * L * M;
  for (int mb = 0; mb < M / 16; ++mb) {
    const frag a0 = WA[mb][0][l];
    const frag a1 = WA[mb][1][l];
    const f32x4 bcv = *reinterpret_cast<const f32x4 *>(&bq[mb * 16 + 4 * g]);
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      f32x4 p = P::mma(a0, xf[tb][0], bcv);
      p = P::mma(a1, xf[tb][1], p);
      f32x4 v;
#pragma unroll
      for (int j = 0; j < 4; ++j) v[j] = P::cos_rev(p[j]) * dfac[tb];
      const int t = rbase + tb * 16 + c16;
      if (t < L) store4(Oh + (size_t)t * M + mb * 16 + 4 * g, v);
    }
  }
}

template <typename T, typename To>
static hipError_t fmap_typed(const Shape &sh, const void *X, const float *W, const float *b,
                             void *Xp, hipStream_t st) {
  const int rows = 64 * FmapCfg<T>::TBW;
  const int ntiles = (sh.L + rows - 1) / rows;
  dim3 grid(ntiles * sh.BH);
  switch (sh.M) {
    case 64:
      hipLaunchKernelGGL((k_feature_map<T, To, 64>), grid, dim3(256), 0, st, (const T *)X, W, b,
                         (To *)Xp, sh.H, sh.L, sh.s, ntiles);
      break;
    case 128:
      hipLaunchKernelGGL((k_feature_map<T, To, 128>), grid, dim3(256), 0, st, (const T *)X, W, b,
                         (To *)Xp, sh.H, sh.L, sh.s, ntiles);
      break;
    case 256:
      hipLaunchKernelGGL((k_feature_map<T, To, 256>), grid, dim3(256), 0, st, (const T *)X, W, b,
                         (To *)Xp, sh.H, sh.L, sh.s, ntiles);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_feature_map(const Shape &sh, Dt in, Dt out, const void *X, const float *W,
                              const float *b, void *Xp, hipStream_t st) {
  if (in == Dt::BF16)
    return out == Dt::BF16 ? fmap_typed<bf16, bf16>(sh, X, W, b, Xp, st)
                           : fmap_typed<bf16, float>(sh, X, W, b, Xp, st);
  return out == Dt::BF16 ? fmap_typed<float, bf16>(sh, X, W, b, Xp, st)
                         : fmap_typed<float, float>(sh, X, W, b, Xp, st);
}

}  // namespace favor
