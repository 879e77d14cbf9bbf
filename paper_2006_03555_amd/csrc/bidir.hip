// bidir.hip - bidirectional FAVOR (Sec. 2.5, Algorithm 1) on CDNA4 matrix cores.
//
// Three launches, none of which stores a feature matrix:
//   k_kside     grid (splits, B*H). Each workgroup streams 64-token tiles of
//               one head's K and V, rebuilds the key features K-hat on the
//               matrix cores (projection + fused cosine), and accumulates its
//               share of Buf1 = K'^T [V 1] in fp32 accumulators. D_K and the
//               sqrt(2/M) constant are folded into the value tile C~ = D_K [V 1],
//               so the feature epilogue is a single cosine. Wave w owns features
//               [w M/4, (w+1) M/4); the ones column is one more 16-wide block.
//   k_finalize  grid (B*H). Sums the split partials in a fixed order
//               (deterministic) and writes Buf1^T as A-operand fragments in
//               chained feature order, with the denominator row replicated over
//               a 16-row block so that every lane of the Q side sees D-hat.
//   k_qside     grid (row tiles, B*H). Rebuilds query features Q-hat (transposed
//               projection, so the result chains straight into the next
//               product), multiplies by Buf1^T streaming over features in steps
//               of 32, and divides by the denominator. D_Q and sqrt(2/M) cancel
//               in the ratio and are never applied; a non-zero stabiliser is
//               rescaled by them instead.
#include "favor_common.hpp"
#include "kernels.hpp"
#include "tile_common.hpp"

namespace favor {

template <typename T, int M>
__global__ __launch_bounds__(256) void k_kside(const T *__restrict__ K, const T *__restrict__ V,
                                               const float *__restrict__ W,
                                               const float *__restrict__ bph,
                                               float *__restrict__ part, int H, int L,
                                               int rows_per_split, int nsplit, float s) {
  constexpr int MW = M / 4;
  constexpr int MB = MW / 16;
  using P = Mma<T>;
  using frag = typename P::frag;
  __shared__ KVTile<T> tl;

  const int split = blockIdx.x;
  const int bh = blockIdx.y;
  const int h = bh % H;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;
  const int r0 = split * rows_per_split;
  const int r1 = min(L, r0 + rows_per_split);

  frag Wf[MB][2];
  f32x4 bC[MB];
  load_w_bfrags<T, MB>(W + (size_t)h * M * kD, bph + (size_t)h * M, w * MW, s * kInv2Pi, Wf, bC);

  f32x4 acc[MB][5];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < 5; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  const T *Kh = K + (size_t)bh * L * kD;
  const T *Vh = V + (size_t)bh * L * kD;
  const float s2half = 0.5f * s * s;
  const float cM = sqrtf(2.0f / M);

  for (int t0 = r0; t0 < r1; t0 += 64) {
    __syncthreads();
    stage_kv_tile<T>(tl, Kh, Vh, t0, r1, s2half, cM);
    __syncthreads();
#pragma unroll
    for (int sidx = 0; sidx < 2; ++sidx) {
      f32x4 kf[MB][2];
      key_features<T, MB>(tl, Wf, bC, sidx, kf);
      frag vb[4];
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) vb[nb] = tl.VtF[nb][sidx][l];
      const frag db = tl.DF[sidx][g];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const frag a = P::pack(kf[mb][0], kf[mb][1]);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = P::mma(a, vb[nb], acc[mb][nb]);
        acc[mb][4] = P::mma(a, db, acc[mb][4]);
      }
    }
  }

  float *dst = part + ((size_t)bh * nsplit + split) * M * 65;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = w * MW + mb * 16 + 4 * g + j;
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) dst[m * 65 + nb * 16 + c16] = acc[mb][nb][j];
      if (c16 == 0) dst[m * 65 + 64] = acc[mb][4][j];
    }
}

template <typename T, int M>
__global__ __launch_bounds__(256) void k_finalize(const float *__restrict__ part, int nsplit,
                                                  typename Mma<T>::frag *__restrict__ frags) {
  constexpr int NS = M / 32;
  using frag = typename Mma<T>::frag;
  const int bh = blockIdx.x;
  const float *src = part + (size_t)bh * nsplit * M * 65;
  frag *dst = frags + (size_t)bh * 5 * NS * 64;
  for (int idx = threadIdx.x; idx < M * 65; idx += blockDim.x) {
    float sum = 0.f;
    for (int sp = 0; sp < nsplit; ++sp) sum += src[(size_t)sp * M * 65 + idx];
    const int m = idx / 65;
    const int n = idx - m * 65;
    const int sidx = m >> 5;
    const int gg = chained_group(m & 31);
    const int sl = chained_slot(m & 31);
    const T v = from_f32<T>(sum);
    if (n < 64) {
      reinterpret_cast<T *>(&dst[((n >> 4) * NS + sidx) * 64 + (n & 15) + 16 * gg])[sl] = v;
    } else {
      for (int c = 0; c < 16; ++c)
        reinterpret_cast<T *>(&dst[(4 * NS + sidx) * 64 + c + 16 * gg])[sl] = v;
    }
  }
}

// Rows per workgroup: 4 waves x TBW blocks of 16 rows.
template <typename T> struct QsideCfg { static constexpr int TBW = 4; };
template <> struct QsideCfg<float> { static constexpr int TBW = 2; };

template <typename T, typename To, int M>
__global__ __launch_bounds__(256) void k_qside(const T *__restrict__ Q,
                                               const float *__restrict__ W,
                                               const float *__restrict__ bph,
                                               const typename Mma<T>::frag *__restrict__ frags,
                                               To *__restrict__ out, int H, int L, float s,
                                               float eps) {
  constexpr int NS = M / 32;
  constexpr int TBW = QsideCfg<T>::TBW;
  using P = Mma<T>;
  using frag = typename P::frag;
  __shared__ frag WA[M / 16][2][64];
  __shared__ frag BF[5][NS][64];
  __shared__ float bq[M];

  const int bh = blockIdx.y;
  const int h = bh % H;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;

  fill_w_afrags<T, M>(WA, bq, W + (size_t)h * M * kD, bph + (size_t)h * M, s * kInv2Pi);
  {
    const frag *src = frags + (size_t)bh * 5 * NS * 64;
    frag *bf = &BF[0][0][0];
    for (int idx = tid; idx < 5 * NS * 64; idx += 256) bf[idx] = src[idx];
  }

  const int rbase = blockIdx.x * (64 * TBW) + w * (16 * TBW);
  const T *Qh = Q + (size_t)bh * L * kD;
  frag qf[TBW][2];
  float epsq[TBW];
#pragma unroll
  for (int tb = 0; tb < TBW; ++tb) {
    const int t = rbase + tb * 16 + c16;
    float nrm = 0.f;
    if (t < L) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        qf[tb][ks] = load_frag<T>(Qh + (size_t)t * kD + ks * 32 + 8 * g);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float x = to_f32(qf[tb][ks][i]);
          nrm = fmaf(x, x, nrm);
        }
      }
    } else {
      qf[tb][0] = P::splat(0.f);
      qf[tb][1] = P::splat(0.f);
    }
    nrm += __shfl_xor(nrm, 16);
    nrm += __shfl_xor(nrm, 32);
    // features here omit D_Q sqrt(2/M); the stabiliser is divided by it instead
    epsq[tb] = (eps != 0.f) ? eps / (sqrtf(2.0f / M) * expf(0.5f * s * s * nrm)) : 0.f;
  }
  __syncthreads();

  f32x4 acc[5][TBW];
#pragma unroll
  for (int nb = 0; nb < 5; ++nb)
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) acc[nb][tb] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int sidx = 0; sidx < NS; ++sidx) {
    f32x4 pf[2][TBW];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int mb = 2 * sidx + hh;
      const frag a0 = WA[mb][0][l];
      const frag a1 = WA[mb][1][l];
      const f32x4 bcv = *reinterpret_cast<const f32x4 *>(&bq[mb * 16 + 4 * g]);
#pragma unroll
      for (int tb = 0; tb < TBW; ++tb) {
        f32x4 p = P::mma(a0, qf[tb][0], bcv);
        p = P::mma(a1, qf[tb][1], p);
#pragma unroll
        for (int j = 0; j < 4; ++j) pf[hh][tb][j] = P::cos_rev(p[j]);
      }
    }
    frag qb[TBW];
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) qb[tb] = P::pack(pf[0][tb], pf[1][tb]);
#pragma unroll
    for (int nb = 0; nb < 5; ++nb) {
      const frag a = BF[nb][sidx][l];
#pragma unroll
      for (int tb = 0; tb < TBW; ++tb) acc[nb][tb] = P::mma(a, qb[tb], acc[nb][tb]);
    }
  }

  To *Oh = out + (size_t)bh * L * kD;
#pragma unroll
  for (int tb = 0; tb < TBW; ++tb) {
    const int t = rbase + tb * 16 + c16;
    if (t < L) {
      const float inv = 1.0f / (acc[4][tb][0] + epsq[tb]);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) store4(Oh + (size_t)t * kD + nb * 16 + 4 * g, acc[nb][tb] * inv);
    }
  }
}

// ---------------------------------------------------------------- launchers
#define FAVOR_DISPATCH_M(M_, ...)                                   \
  switch (M_) {                                                     \
    case 64: { constexpr int MM = 64; __VA_ARGS__; } break;          \
    case 128: { constexpr int MM = 128; __VA_ARGS__; } break;        \
    case 256: { constexpr int MM = 256; __VA_ARGS__; } break;        \
    default: return hipErrorInvalidValue;                           \
  }

hipError_t launch_kside(const Shape &sh, Dt in, const void *K, const void *V, const float *W,
                        const float *b, float *part, int rows_per_split, int nsplit,
                        hipStream_t st) {
  dim3 grid(nsplit, sh.BH);
  if (in == Dt::BF16) {
    FAVOR_DISPATCH_M(sh.M, hipLaunchKernelGGL((k_kside<bf16, MM>), grid, dim3(256), 0, st,
                                               (const bf16 *)K, (const bf16 *)V, W, b, part, sh.H,
                                               sh.L, rows_per_split, nsplit, sh.s));
  } else {
    FAVOR_DISPATCH_M(sh.M, hipLaunchKernelGGL((k_kside<float, MM>), grid, dim3(256), 0, st,
                                               (const float *)K, (const float *)V, W, b, part,
                                               sh.H, sh.L, rows_per_split, nsplit, sh.s));
  }
  return hipGetLastError();
}

hipError_t launch_finalize(const Shape &sh, Dt in, const float *part, int nsplit, void *frags,
                           hipStream_t st) {
  dim3 grid(sh.BH);
  if (in == Dt::BF16) {
    FAVOR_DISPATCH_M(sh.M, hipLaunchKernelGGL((k_finalize<bf16, MM>), grid, dim3(256), 0, st,
                                               part, nsplit, (Mma<bf16>::frag *)frags));
  } else {
    FAVOR_DISPATCH_M(sh.M, hipLaunchKernelGGL((k_finalize<float, MM>), grid, dim3(256), 0, st,
                                               part, nsplit, (Mma<float>::frag *)frags));
  }
  return hipGetLastError();
}

template <typename T, typename To>
static hipError_t qside_typed(const Shape &sh, const void *Q, const float *W, const float *b,
                              const void *frags, void *o, hipStream_t st) {
  const int rows = 64 * QsideCfg<T>::TBW;
  dim3 grid((sh.L + rows - 1) / rows, sh.BH);
  FAVOR_DISPATCH_M(sh.M, hipLaunchKernelGGL((k_qside<T, To, MM>), grid, dim3(256), 0, st,
                                             (const T *)Q, W, b,
                                             (const typename Mma<T>::frag *)frags, (To *)o, sh.H,
                                             sh.L, sh.s, sh.eps));
  return hipGetLastError();
}

hipError_t launch_qside(const Shape &sh, Dt in, Dt out, const void *Q, const float *W,
                        const float *b, const void *frags, void *o, hipStream_t st) {
  if (in == Dt::BF16)
    return out == Dt::BF16 ? qside_typed<bf16, bf16>(sh, Q, W, b, frags, o, st)
                           : qside_typed<bf16, float>(sh, Q, W, b, frags, o, st);
  return out == Dt::BF16 ? qside_typed<float, bf16>(sh, Q, W, b, frags, o, st)
                         : qside_typed<float, float>(sh, Q, W, b, frags, o, st);
}

}  // namespace favor
