// causal.hip - unidirectional FAVOR by prefix sums (Sec. 2.5.1, Eq. cumsum).
//
// The prefix tensor G^PS is never stored (the O(Md + Ld + ML) variant of
// Sec. 2.6). The sequence of each head is cut into segments; segments run in
// parallel and hand each other M x (d+1) fp32 aggregates:
//   k_kside (bidir.hip)  segment aggregates sum_{j in seg} K'_j C_j^T
//   k_seg_scan           exclusive prefix over segments, plus state_in;
//                        the total goes to state_out
//   k_causal             per segment, 64-token chunks in order. With S the
//                        state before the chunk (Q-hat, K-hat the features of
//                        the chunk's queries and keys, C~ = D_K [V 1]):
//                          Buf2 = Q-hat S + tril(Q-hat K-hat^T) C~
//                          S   <- S + K-hat^T C~
//                        which is Eq. cumsum grouped 64 tokens at a time (the
//                        diagonal block is masked to keys j <= i).
// Work split inside a workgroup of 4 waves for one chunk:
//   wave w owns features [w M/4, (w+1) M/4) of the state (fp32 accumulators)
//   and of the key projection; it publishes S (bf16/fp32 A-operand fragments)
//   and its key features (row-major fragments) through LDS; then wave w owns
//   queries 16 w .. 16 w + 15 of the chunk: it rebuilds their features over all
//   M, forms Q-hat S, the masked 16 x (16 w + 16) block of Q-hat K-hat^T and
//   its product with C~, and writes normalised rows.
#include "favor_common.hpp"
#include "kernels.hpp"
#include "tile_common.hpp"

namespace favor {

__global__ __launch_bounds__(256) void k_seg_scan(float *__restrict__ part, int nseg, int n,
                                                  const float *__restrict__ state_in,
                                                  float *__restrict__ state_out) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  const int bh = blockIdx.y;
  if (idx >= n) return;
  float run = state_in ? state_in[(size_t)bh * n + idx] : 0.f;
  float *p = part + (size_t)bh * nseg * n + idx;
  for (int sg = 0; sg < nseg; ++sg) {
    const float v = p[(size_t)sg * n];
    p[(size_t)sg * n] = run;
    run += v;
  }
  if (state_out) state_out[(size_t)bh * n + idx] = run;
}

template <typename T, int M>
struct CausalSmem {
  using frag = typename Mma<T>::frag;
  KVTile<T> tl;
  frag KA[4][M / 32][64];   // key features K-hat as A fragments: lane row t', chained m order
  frag SA[5][M / 32][64];   // S^T as A fragments: lane row n, chained m order
  frag WA[M / 16][2][64];   // W'' as A fragments for the query projection
  float bq[M];
};

template <typename T, typename To, int M>
__global__ __launch_bounds__(256) void k_causal(const T *__restrict__ Q, const T *__restrict__ K,
                                                const T *__restrict__ V,
                                                const float *__restrict__ W,
                                                const float *__restrict__ bph,
                                                const float *__restrict__ prefix,
                                                To *__restrict__ out, int H, int L, int seg_len,
                                                int nseg, float s, float eps) {
  constexpr int MW = M / 4;
  constexpr int MB = MW / 16;
  constexpr int NS = M / 32;
  using P = Mma<T>;
  using frag = typename P::frag;
  __shared__ CausalSmem<T, M> sm;

  const int seg = blockIdx.x;
  const int bh = blockIdx.y;
  const int h = bh % H;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;

  const float *Wh = W + (size_t)h * M * kD;
  const float *bhh = bph + (size_t)h * M;
  fill_w_afrags<T, M>(sm.WA, sm.bq, Wh, bhh, s * kInv2Pi);
  frag Wf[MB][2];
  f32x4 bC[MB];
  load_w_bfrags<T, MB>(Wh, bhh, w * MW, s * kInv2Pi, Wf, bC);

  // state rows m = w MW + 16 mb + 4 g + j, columns 16 nb + c16 (the fifth block
  // holds the ones column replicated over its 16 columns)
  f32x4 accS[MB][5];
  {
    const float *pre = prefix + ((size_t)bh * nseg + seg) * M * 65;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int m = w * MW + mb * 16 + 4 * g + j;
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) accS[mb][nb][j] = pre[m * 65 + nb * 16 + c16];
        accS[mb][4][j] = pre[m * 65 + 64];
      }
  }

  const T *Qh = Q + (size_t)bh * L * kD;
  const T *Kh = K + (size_t)bh * L * kD;
  const T *Vh = V + (size_t)bh * L * kD;
  To *Oh = out + (size_t)bh * L * kD;
  const float s2half = 0.5f * s * s;
  const float cM = sqrtf(2.0f / M);
  const int r0 = seg * seg_len;
  const int r1 = min(L, r0 + seg_len);

  for (int t0 = r0; t0 < r1; t0 += 64) {
    __syncthreads();
    stage_kv_tile<T>(sm.tl, Kh, Vh, t0, r1, s2half, cM);
    // publish S before this chunk's update
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int mbg = w * MB + mb;
#pragma unroll
      for (int nb = 0; nb < 5; ++nb) {
        T *p = reinterpret_cast<T *>(&sm.SA[nb][mbg >> 1][l]) + 4 * (mbg & 1);
#pragma unroll
        for (int j = 0; j < 4; ++j) p[j] = from_f32<T>(accS[mb][nb][j]);
      }
    }
    __syncthreads();

    // key features for this wave's features: publish and fold into S
#pragma unroll
    for (int sidx = 0; sidx < 2; ++sidx) {
      f32x4 kf[MB][2];
      key_features<T, MB>(sm.tl, Wf, bC, sidx, kf);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int mg = w * MW + mb * 16 + c16;
        const int sm_ = mg >> 5;
        const int lane_hi = 16 * chained_group(mg & 31);
        const int sl = chained_slot(mg & 31);
#pragma unroll
        for (int tbl = 0; tbl < 2; ++tbl)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            reinterpret_cast<T *>(&sm.KA[2 * sidx + tbl][sm_][4 * g + j + lane_hi])[sl] =
                from_f32<T>(kf[mb][tbl][j]);
      }
      frag vb[4];
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) vb[nb] = sm.tl.VtF[nb][sidx][l];
      const frag db = sm.tl.DF[sidx][g];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const frag a = P::pack(kf[mb][0], kf[mb][1]);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) accS[mb][nb] = P::mma(a, vb[nb], accS[mb][nb]);
        accS[mb][4] = P::mma(a, db, accS[mb][4]);
      }
    }
    __syncthreads();

    // queries 16 w .. 16 w + 15 of the chunk
    const int qt = t0 + 16 * w + c16;
    frag qf[2];
    float nrm = 0.f;
    if (qt < r1) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        qf[ks] = load_frag<T>(Qh + (size_t)qt * kD + ks * 32 + 8 * g);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float x = to_f32(qf[ks][i]);
          nrm = fmaf(x, x, nrm);
        }
      }
    } else {
      qf[0] = P::splat(0.f);
      qf[1] = P::splat(0.f);
    }
    nrm += __shfl_xor(nrm, 16);
    nrm += __shfl_xor(nrm, 32);
    const float epsq = (eps != 0.f) ? eps / (cM * expf(s2half * nrm)) : 0.f;

    f32x4 o[5];
    f32x4 pt[4];
#pragma unroll
    for (int nb = 0; nb < 5; ++nb) o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) pt[tb] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int sidx = 0; sidx < NS; ++sidx) {
      f32x4 pf[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int mb = 2 * sidx + hh;
        const f32x4 bcv = *reinterpret_cast<const f32x4 *>(&sm.bq[mb * 16 + 4 * g]);
        f32x4 p = P::mma(sm.WA[mb][0][l], qf[0], bcv);
        p = P::mma(sm.WA[mb][1][l], qf[1], p);
#pragma unroll
        for (int j = 0; j < 4; ++j) pf[hh][j] = P::cos_rev(p[j]);
      }
      const frag qb = P::pack(pf[0], pf[1]);
#pragma unroll
      for (int nb = 0; nb < 5; ++nb) o[nb] = P::mma(sm.SA[nb][sidx][l], qb, o[nb]);
#pragma unroll
      for (int tb = 0; tb < 4; ++tb)
        if (tb <= w) pt[tb] = P::mma(sm.KA[tb][sidx][l], qb, pt[tb]);
    }
    // keys after the query inside the diagonal block: t' = 16 w + 4 g + j > t = 16 w + c16
#pragma unroll
    for (int tb = 0; tb < 4; ++tb)
      if (tb == w) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (4 * g + j > c16) pt[tb][j] = 0.f;
      }
#pragma unroll
    for (int sp = 0; sp < 2; ++sp) {
      if (2 * sp <= w) {
        const frag pb = P::pack(pt[2 * sp], pt[2 * sp + 1]);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) o[nb] = P::mma(sm.tl.VtF[nb][sp][l], pb, o[nb]);
        o[4] = P::mma(sm.tl.DF[sp][g], pb, o[4]);
      }
    }
    if (qt < r1) {
      const float inv = 1.0f / (o[4][0] + epsq);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) store4(Oh + (size_t)qt * kD + nb * 16 + 4 * g, o[nb] * inv);
    }
  }
}

hipError_t launch_seg_scan(const Shape &sh, float *part, int nseg, const float *state_in,
                           float *state_out, hipStream_t st) {
  const int n = sh.M * 65;
  dim3 grid((n + 255) / 256, sh.BH);
  hipLaunchKernelGGL(k_seg_scan, grid, dim3(256), 0, st, part, nseg, n, state_in, state_out);
  return hipGetLastError();
}

template <typename T, typename To>
static hipError_t causal_typed(const Shape &sh, const void *Q, const void *K, const void *V,
                               const float *W, const float *b, const float *prefix, void *o,
                               int seg_len, int nseg, hipStream_t st) {
  dim3 grid(nseg, sh.BH);
#define FAVOR_CAUSAL_LAUNCH(MM)                                                             \
  hipLaunchKernelGGL((k_causal<T, To, MM>), grid, dim3(256), 0, st, (const T *)Q,             \
                     (const T *)K, (const T *)V, W, b, prefix, (To *)o, sh.H, sh.L, seg_len,  \
                     nseg, sh.s, sh.eps)
  switch (sh.M) {
    case 64: FAVOR_CAUSAL_LAUNCH(64); break;
    case 128: FAVOR_CAUSAL_LAUNCH(128); break;
    case 256:
      if constexpr (sizeof(T) == 2) {
        FAVOR_CAUSAL_LAUNCH(256);
        break;
      }
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
#undef FAVOR_CAUSAL_LAUNCH
  return hipGetLastError();
}

hipError_t launch_causal(const Shape &sh, Dt in, Dt out, const void *Q, const void *K,
                         const void *V, const float *W, const float *b, const float *prefix,
                         void *o, int seg_len, int nseg, hipStream_t st) {
  if (in == Dt::BF16)
    return out == Dt::BF16
               ? causal_typed<bf16, bf16>(sh, Q, K, V, W, b, prefix, o, seg_len, nseg, st)
               : causal_typed<bf16, float>(sh, Q, K, V, W, b, prefix, o, seg_len, nseg, st);
  return out == Dt::BF16
             ? causal_typed<float, bf16>(sh, Q, K, V, W, b, prefix, o, seg_len, nseg, st)
             : causal_typed<float, float>(sh, Q, K, V, W, b, prefix, o, seg_len, nseg, st);
}

}  // namespace favor
