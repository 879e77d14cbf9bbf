// prep.hip - per-call conversion of the random features into matrix-core form.
//
// W'' = (s / 2 pi) W rounded to the element type of the inputs, laid out as
// fragments wfr[h][mb][ks][lane] = W''[16 mb + lane % 16][32 ks + 8 (lane / 16) .. + 8],
// and b'' = b / 2 pi. The 1 / 2 pi folds the cosine's argument into revolutions
// (the unit of the hardware cosine); s folds the input scale into the
// projection so that the stored inputs are used as they are.
#include "favor_common.hpp"
#include "kernels.hpp"
#include "tile_common.hpp"

namespace favor {

template <typename T>
__global__ __launch_bounds__(256) void k_prep_w(const float *__restrict__ W,
                                                const float *__restrict__ b, int M, float ws,
                                                typename Mma<T>::frag *__restrict__ wfr,
                                                float *__restrict__ bq) {
  const int h = blockIdx.y;
  const int idx = blockIdx.x * 256 + threadIdx.x;   // fragment index within the head
  const int nfrag = (M / 16) * 2 * 64;
  if (idx < nfrag) {
    const int mb = idx >> 7;
    const int ks = (idx >> 6) & 1;
    const int l = idx & 63;
    const int m = mb * 16 + (l & 15);
    float v[8];
    load8_f32(W + ((size_t)h * M + m) * kD + ks * 32 + 8 * (l >> 4), v);
    wfr[(size_t)h * nfrag + idx] = Mma<T>::from_f32(v, ws);
  }
  if (idx < M) bq[(size_t)h * M + idx] = b[(size_t)h * M + idx] * kInv2Pi;
}

hipError_t launch_prep_w(const Shape &sh, Dt in, const float *W, const float *b, void *wfr,
                         float *bq, hipStream_t st) {
  const int nfrag = (sh.M / 16) * 2 * 64;
  dim3 grid((nfrag + 255) / 256, sh.H);
  const float ws = sh.s * kInv2Pi;
  if (in == Dt::BF16)
    hipLaunchKernelGGL(k_prep_w<bf16>, grid, dim3(256), 0, st, W, b, sh.M, ws,
                       (Mma<bf16>::frag *)wfr, bq);
  else
    hipLaunchKernelGGL(k_prep_w<float>, grid, dim3(256), 0, st, W, b, sh.M, ws,
                       (Mma<float>::frag *)wfr, bq);
  return hipGetLastError();
}

}  // namespace favor
