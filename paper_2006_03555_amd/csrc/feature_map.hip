// feature_map.hip - the random-feature map X' = D_X X-hat (Sec. 2.3, Eqs. dqdk
// and qkprime), or the ReLU features of generalized attention (Sec. 2.2),
// materialised in HBM.
//
// The projection W'' x is a matrix-core product in transposed orientation
// (result lane = row), seeded with b'' so the epilogue is cos(2 pi acc) *
// D_X(row) * sqrt(2/M). The kernel is bound by writing X' (M elements per row
// against d read), so the W'' rows are ordered for whole-line stores: with bf16
// output row r of 16-feature block mb is feature perm_col(mb, r) (each lane
// then holds two runs of 8 consecutive features of its row and every 16-byte
// store instruction writes 64 contiguous bytes per row); with fp32 output the
// natural order already gives 16 contiguous bytes per lane and 64 per row.
#include "favor_common.hpp"
#include "kernels.hpp"
#include "tile_common.hpp"

namespace favor {

// One workgroup of eight waves per CU (two per SIMD: one wave's cosines and
// stores overlap the other's matrix work; the head's W'' is loaded once for
// all eight). A work item is 8 waves x TBW blocks of 16 rows.
constexpr int kFmapThreads = 512;
constexpr int kFmapWorkgroups = 256;
template <typename T> struct FmapCfg { static constexpr int TBW = 2; };

template <typename To>
__device__ __forceinline__ int fmap_row(int mb, int r) {
  if constexpr (sizeof(To) == 2) return perm_col(mb, r);
  return 16 * mb + r;
}

// W'' A-operand fragments in the store order above and b'' (natural order)
// into LDS, cooperatively (NT threads, loads in flight in batches).
template <typename T, typename To, int M, int NT, int KN>
__device__ __forceinline__ void fill_w_afrags_perm(typename Mma<T>::frag (*WA)[2][64], float *bq,
                                                   const float *__restrict__ Wh,
                                                   const float *__restrict__ bh, float ws,
                                                   float bs, int Mr, float keps) {
  constexpr int N = (M / 16) * 2 * 64;
  constexpr int NB = (N / NT) < 4 ? (N / NT) : 4;   // loads in flight per batch
  static_assert(N % (NT * NB) == 0, "thread count");
#pragma unroll
  for (int it0 = 0; it0 < N / NT; it0 += NB) {
    float v[NB][8];
#pragma unroll
    for (int it = 0; it < NB; ++it) {
      const int idx = (it0 + it) * NT + threadIdx.x;
      const int m = fmap_row<To>(idx >> 7, idx & 15);
      if (m < Mr) {   // W'' rows past the M_r drawn are zero
        load8_f32(Wh + (size_t)m * kD + ((idx >> 6) & 1) * 32 + 8 * ((idx & 63) >> 4), v[it]);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[it][i] = 0.f;
      }
    }
#pragma unroll
    for (int it = 0; it < NB; ++it) {
      const int idx = (it0 + it) * NT + threadIdx.x;
      WA[idx >> 7][(idx >> 6) & 1][idx & 63] = Mma<T>::from_f32(v[it], ws);
    }
  }
  if (threadIdx.x < M) bq[threadIdx.x] = seed_row<KN>(threadIdx.x, Mr, bh, bs, keps);
}

// The four result tiles of 64 features for one row: bf16 lanes hold features
// 8 g .. 8 g + 7 (tiles 0, 1) and 32 + 8 g .. (tiles 2, 3) of the 64; fp32 lanes
// hold 16 k + 4 g .. 16 k + 4 g + 3 in tile k. Only the first nv features of the
// 64 are stored (nv a multiple of 16: each store is all in or all out).
__device__ __forceinline__ void store_row64(bf16 *p, int g, const f32x4 (&v)[4], int nv) {
  if (nv >= 64 || 8 * g < nv) store8(p + 8 * g, v[0], v[1]);
  if (nv >= 64 || 32 + 8 * g < nv) store8(p + 32 + 8 * g, v[2], v[3]);
}
__device__ __forceinline__ void store_row64(float *p, int g, const f32x4 (&v)[4], int nv) {
#pragma unroll
  for (int k = 0; k < 4; ++k)
    if (nv >= 64 || 16 * k + 4 * g < nv) *reinterpret_cast<f32x4 *>(p + 16 * k + 4 * g) = v[k];
}

// Persistent: workgroup i takes an XCD-local range of (head, row tile) items,
// loads the head's W'' when the head changes, and prefetches the next tile's
// rows while the current one is projected and written.
template <typename T, typename To, int M, int KN>
__global__ __launch_bounds__(kFmapThreads, 1) void k_feature_map(const T *__restrict__ X,
                                                     const float *__restrict__ W,
                                                     const float *__restrict__ bph,
                                                     To *__restrict__ Xp, int H, int L, float s,
                                                     int ntiles, int nitems, float ws, float bs,
                                                     float keps, int Mr, float cM) {
  constexpr int TBW = FmapCfg<T>::TBW;
  using P = Mma<T>;
  using frag = typename P::frag;
  __shared__ frag WA[M / 16][2][64];
  __shared__ float bq[M];

  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;
  const float s2half = 0.5f * s * s;

  int begin, end;
  xcd_range(blockIdx.x, gridDim.x, nitems, begin, end);
  if (begin >= end) return;

  // rows rbase + 16 tb + c16 of an item, columns 8 g .. and 32 + 8 g ..
  auto load_rows = [&](int item, frag (&xf)[TBW][2]) {
    const int bh = item / ntiles;
    const int rbase = (item - bh * ntiles) * (kFmapThreads / 4 * TBW) + w * (16 * TBW);
    const T *Xh = X + (size_t)bh * L * kD;
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      const int t = rbase + tb * 16 + c16;
      if (t < L) {
        xf[tb][0] = load_frag<T>(Xh + (size_t)t * kD + 8 * g);
        xf[tb][1] = load_frag<T>(Xh + (size_t)t * kD + 32 + 8 * g);
      } else {
        xf[tb][0] = P::splat(0.f);
        xf[tb][1] = P::splat(0.f);
      }
    }
  };

  frag xn[TBW][2];
  load_rows(begin, xn);
  int cur = -1;
  for (int item = begin; item < end; ++item) {
    const int bh = item / ntiles;
    if (bh != cur) {   // the head's W'' fragments and b''
      const int h = bh % H;
      __syncthreads();
      fill_w_afrags_perm<T, To, M, kFmapThreads, KN>(WA, bq, W + (size_t)h * Mr * kD,
                                                     bph + (size_t)h * Mr, ws, bs, Mr, keps);
      __syncthreads();
      cur = bh;
    }
    frag xf[TBW][2];
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      xf[tb][0] = xn[tb][0];
      xf[tb][1] = xn[tb][1];
    }
    if (item + 1 < end) load_rows(item + 1, xn);

    // D_X(row) sqrt(2/M) = sqrt(2/M) exp(||s x||^2 / 2) (1 for ReLU features)
    float dfac[TBW];
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      dfac[tb] = 1.f;
      if constexpr (KN == kRelu) continue;
      float nrm = sq_sum16(xf[tb]);
      nrm += __shfl_xor(nrm, 16);
      nrm += __shfl_xor(nrm, 32);
      dfac[tb] = cM * expf(s2half * nrm);
    }

    const int rbase = (item - bh * ntiles) * (kFmapThreads / 4 * TBW) + w * (16 * TBW);
    To *Oh = Xp + (size_t)bh * L * Mr;   // rows of M_r features
    for (int q = 0; q < M / 64; ++q) {   // features 64 q .. 64 q + 63 (stored: < M_r)
      frag a[4][2];
      f32x4 bcv[4];   // b'' of result rows 4 g + j of tile k (in store order)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        a[k][0] = WA[4 * q + k][0][l];
        a[k][1] = WA[4 * q + k][1][l];
#pragma unroll
        for (int j = 0; j < 4; ++j) bcv[k][j] = bq[fmap_row<To>(4 * q + k, 4 * g + j)];
      }
#pragma unroll
      for (int tb = 0; tb < TBW; ++tb) {
        f32x4 v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          f32x4 p = P::mma(a[k][0], xf[tb][0], bcv[k]);
          p = P::mma(a[k][1], xf[tb][1], p);
#pragma unroll
          for (int j = 0; j < 4; ++j) v[k][j] = feature<KN, P>(p[j], bcv[k][j]) * dfac[tb];
        }
        const int t = rbase + tb * 16 + c16;
        if (t < L) {
          if (Mr == M)   // every tile whole: the stores need no feature mask
            store_row64(Oh + (size_t)t * M + 64 * q, g, v, 64);
          else
            store_row64(Oh + (size_t)t * Mr + 64 * q, g, v, Mr - 64 * q);
        }
      }
    }
  }
}

template <typename T, typename To, int KN>
static hipError_t fmap_typed(const Shape &sh, const void *X, const float *W, const float *b,
                             void *Xp, hipStream_t st) {
  const int rows = kFmapThreads / 4 * FmapCfg<T>::TBW;
  const int ntiles = (sh.L + rows - 1) / rows;
  const int nitems = ntiles * sh.BH;
  const int cap = kFmapWorkgroups;
  dim3 grid(nitems < cap ? nitems : cap);
  float ws, bs;
  feature_scales(sh, ws, bs);
#define FAVOR_FMAP_LAUNCH(MM)                                                               \
  hipLaunchKernelGGL((k_feature_map<T, To, MM, KN>), grid, dim3(kFmapThreads), 0, st,        \
                     (const T *)X, W, b, (To *)Xp, sh.H, sh.L, sh.s, ntiles, nitems, ws, bs, \
                     sh.keps, sh.Mr, feature_norm(sh))
  switch (sh.M) {
    case 64: FAVOR_FMAP_LAUNCH(64); break;
    case 128: FAVOR_FMAP_LAUNCH(128); break;
    case 256: FAVOR_FMAP_LAUNCH(256); break;
    default: return hipErrorInvalidValue;
  }
#undef FAVOR_FMAP_LAUNCH
  return hipGetLastError();
}

template <typename T, typename To>
static hipError_t fmap_kernel(const Shape &sh, const void *X, const float *W, const float *b,
                              void *Xp, hipStream_t st) {
  return sh.kernel == 1 ? fmap_typed<T, To, kRelu>(sh, X, W, b, Xp, st)
                        : fmap_typed<T, To, kCos>(sh, X, W, b, Xp, st);
}

hipError_t launch_feature_map(const Shape &sh, Dt in, Dt out, const void *X, const float *W,
                              const float *b, void *Xp, hipStream_t st) {
  if (in == Dt::BF16)
    return out == Dt::BF16 ? fmap_kernel<bf16, bf16>(sh, X, W, b, Xp, st)
                           : fmap_kernel<bf16, float>(sh, X, W, b, Xp, st);
  return out == Dt::BF16 ? fmap_kernel<float, bf16>(sh, X, W, b, Xp, st)
                         : fmap_kernel<float, float>(sh, X, W, b, Xp, st);
}

}  // namespace favor
