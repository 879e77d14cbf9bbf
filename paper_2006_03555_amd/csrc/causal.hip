// causal.hip - unidirectional FAVOR by prefix sums (Sec. 2.5.1, Eq. cumsum).
//
// The prefix tensor G^PS is never stored (the O(Md + Ld + ML) variant of
// Sec. 2.6). The sequence of each head is cut into segments; segments run in
// parallel and hand each other M x (d+1) fp32 aggregates:
//   k_kside (bidir.hip)  segment aggregates sum_{j in seg} K'_j C_j^T
//   k_seg_scan           exclusive prefix over segments, plus state_in;
//                        state_in + total goes to state_out and, when both
//                        directions are requested, the total alone (the
//                        bidirectional Buf1 = K'^T [V 1]) to its own buffer
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
//   and its key features, transposed on the matrix cores to token-major
//   fragments, through LDS; then wave w owns queries 16 w .. 16 w + 15 of the
//   chunk: it rebuilds their features over all M, forms Q-hat S and the masked
//   16 x 64 block of Q-hat K-hat^T with its product with C~ (all waves do the
//   same work, keys after the query are zeroed), and writes normalised rows.
// Keys, values and queries of the next chunk are loaded while this one is
// computed.
#include "favor_common.hpp"
#include "kernels.hpp"
#include "tile_common.hpp"

namespace favor {

__global__ __launch_bounds__(256) void k_seg_scan(float *__restrict__ part, int nseg, int n,
                                                  const float *__restrict__ state_in,
                                                  float *__restrict__ state_out,
                                                  float *__restrict__ total) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  const int bh = blockIdx.y;
  if (idx >= n) return;
  const float s0 = state_in ? state_in[(size_t)bh * n + idx] : 0.f;
  float run = 0.f;   // aggregate of the segments before sg (tokens of this call only)
  float *p = part + (size_t)bh * nseg * n + idx;
  int sg = 0;
  for (; sg + 8 <= nseg; sg += 8) {   // eight loads in flight
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = p[(size_t)(sg + k) * n];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      p[(size_t)(sg + k) * n] = s0 + run;
      run += v[k];
    }
  }
  for (; sg < nseg; ++sg) {
    const float v = p[(size_t)sg * n];
    p[(size_t)sg * n] = s0 + run;
    run += v;
  }
  if (state_out) state_out[(size_t)bh * n + idx] = s0 + run;
  if (total) total[(size_t)bh * n + idx] = run;
}

template <typename T, int M>
struct CausalSmem {
  using frag = typename Mma<T>::frag;
  KVTile<T> tl;
  frag KA[4][M / 32][64];   // key features K-hat as A fragments: lane row t', chained m order
  frag SA[4][M / 32][64];   // S^T (value columns) as A fragments: lane row n, chained m order
  frag SZ[M / 32][4];       // the ones column of S^T: one fragment per lane group
  frag WA[M / 16][2][64];   // W'' fragments (A operand of the query projection, B of the key one)
  frag SEL[4][64];          // selection matrices for the matrix-core transposes
  float bq[M];
};

template <typename T, typename To, int M>
__global__ __launch_bounds__(256) void k_causal(const T *__restrict__ Q, const T *__restrict__ K,
                                                const T *__restrict__ V,
                                                const typename Mma<T>::frag *__restrict__ wfr,
                                                const float *__restrict__ bqg,
                                                const float *__restrict__ prefix,
                                                To *__restrict__ out, int H, int L, int seg_len,
                                                int nseg, float s, float eps) {
  constexpr int MW = M / 4;
  constexpr int MB = MW / 16;
  constexpr int NS = M / 32;
  using P = Mma<T>;
  using frag = typename P::frag;
  __shared__ CausalSmem<T, M> sm;

  const int item = xcd_item(blockIdx.x, gridDim.x);
  const int bh = item / nseg;
  const int seg = item - bh * nseg;
  const int h = bh % H;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;

  const frag *wh = wfr + (size_t)h * (M / 16) * 2 * 64;
  copy_frags<frag, (M / 16) * 2 * 64>(&sm.WA[0][0][0], wh);
  if (tid < M) sm.bq[tid] = bqg[(size_t)h * M + tid];
  if (w == 0) {
    sm.SEL[0][l] = select_frag<T>(0);
    sm.SEL[1][l] = select_frag<T>(1);
    sm.SEL[2][l] = chained_select_frag<T>(0);
    sm.SEL[3][l] = chained_select_frag<T>(1);
  }

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

  __syncthreads();
  TileRegs<T> rg;
  load_tile_regs<T>(rg, Kh, Vh, r0, r1);
  frag qn[2];
  load_query_frags<T>(qn, Qh, r0 + 16 * w + c16, r1);
  KVTile<T> &tl = sm.tl;
  for (int t0 = r0; t0 < r1; t0 += 64) {
    const bool next = t0 + 64 < r1;
    // the previous chunk's readers are done: stage this chunk's prefetched keys
    // and values and publish S (the state before this chunk)
    {
      const frag sel[2] = {sm.SEL[0][l], sm.SEL[1][l]};
      stage_tile<T>(tl, rg, sel, t0, r1, s2half, cM);
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int mbg = w * MB + mb;
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        T *p = reinterpret_cast<T *>(&sm.SA[nb][mbg >> 1][l]) + 4 * (mbg & 1);
#pragma unroll
        for (int j = 0; j < 4; ++j) p[j] = from_f32<T>(accS[mb][nb][j]);
      }
      if (c16 == 0) {   // ones column: identical in every lane of the group
        T *p = reinterpret_cast<T *>(&sm.SZ[mbg >> 1][g]) + 4 * (mbg & 1);
#pragma unroll
        for (int j = 0; j < 4; ++j) p[j] = from_f32<T>(accS[mb][4][j]);
      }
    }
    const frag qf[2] = {qn[0], qn[1]};
    __syncthreads();
    if (next) {
      load_tile_regs<T>(rg, Kh, Vh, t0 + 64, r1);
      load_query_frags<T>(qn, Qh, t0 + 64 + 16 * w + c16, r1);
    }

    // key features of this wave's feature range: fold into S, and publish them
    // transposed (row = token) for the intra-chunk products
#pragma unroll
    for (int sidx = 0; sidx < 2; ++sidx) {
      f32x4 kf[MB][2];
      key_features_lds<T, MB>(tl, sm.WA, sm.bq, w * MB, sidx, kf);
      frag vb[4];
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) vb[nb] = tl.VtF[nb][sidx][l];
      const frag db = tl.DF[sidx][g];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const frag a = P::pack(kf[mb][0], kf[mb][1]);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) accS[mb][nb] = P::mma(a, vb[nb], accS[mb][nb]);
        accS[mb][4] = P::mma(a, db, accS[mb][4]);
        const int mbg = w * MB + mb;
#pragma unroll
        for (int tbl = 0; tbl < 2; ++tbl) {
          // exact transpose on the matrix cores: lane = token, rows = 4 features
          const f32x4 c = P::mma(a, sm.SEL[2 + tbl][l], f32x4{0.f, 0.f, 0.f, 0.f});
          T *p = reinterpret_cast<T *>(&sm.KA[2 * sidx + tbl][mbg >> 1][l]) + 4 * (mbg & 1);
#pragma unroll
          for (int j = 0; j < 4; ++j) p[j] = from_f32<T>(c[j]);
        }
      }
    }
    __syncthreads();

    // queries 16 w .. 16 w + 15 of the chunk (every wave does the same work)
    const int qt = t0 + 16 * w + c16;
    float epsq = 0.f;
    if (eps != 0.f) {
      float nrm = 0.f;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float x = to_f32(qf[ks][i]);
          nrm = fmaf(x, x, nrm);
        }
      nrm += __shfl_xor(nrm, 16);
      nrm += __shfl_xor(nrm, 32);
      epsq = eps / (cM * expf(s2half * nrm));
    }

    f32x4 o[5];
    f32x4 pt[4];
#pragma unroll
    for (int nb = 0; nb < 5; ++nb) o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) pt[tb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // operands of one feature step (32 features): W'' for the query projection,
    // S^T (value columns and ones column) and the key features; loaded one step
    // ahead so their LDS latency overlaps the current step's matrix work
    struct StepOps {
      frag wa[2][2];
      frag sa[4];
      frag sz;
      frag ka[4];
      f32x4 bc[2];
    };
    auto load_ops = [&](StepOps &op, int sidx) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        op.wa[hh][0] = sm.WA[2 * sidx + hh][0][l];
        op.wa[hh][1] = sm.WA[2 * sidx + hh][1][l];
        op.bc[hh] = *reinterpret_cast<const f32x4 *>(&sm.bq[(2 * sidx + hh) * 16 + 4 * g]);
      }
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) op.sa[nb] = sm.SA[nb][sidx][l];
      op.sz = sm.SZ[sidx][g];
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) op.ka[tb] = sm.KA[tb][sidx][l];
    };
    // software pipeline: the projection of step sidx + 1 is issued to the matrix
    // cores before the cosines of step sidx run on the vector unit
    auto project = [&](const StepOps &op, f32x4 (&pr)[2]) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        pr[hh] = P::mma(op.wa[hh][0], qf[0], op.bc[hh]);
        pr[hh] = P::mma(op.wa[hh][1], qf[1], pr[hh]);
      }
    };
    StepOps cur, nxt;
    load_ops(cur, 0);
    f32x4 pc[2];
    project(cur, pc);
    if (NS > 1) load_ops(nxt, 1);
#pragma unroll
    for (int sidx = 0; sidx < NS; ++sidx) {
      f32x4 pn[2];
      if (sidx + 1 < NS) project(nxt, pn);
      __builtin_amdgcn_sched_barrier(0);
      f32x4 pf[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int j = 0; j < 4; ++j) pf[hh][j] = P::cos_rev(pc[hh][j]);
      const frag qb = P::pack(pf[0], pf[1]);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) o[nb] = P::mma(cur.sa[nb], qb, o[nb]);
      o[4] = P::mma(cur.sz, qb, o[4]);
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) pt[tb] = P::mma(cur.ka[tb], qb, pt[tb]);
      if (sidx + 1 < NS) {
        cur = nxt;
        pc[0] = pn[0];
        pc[1] = pn[1];
        if (sidx + 2 < NS) load_ops(nxt, sidx + 2);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // keep keys t' = 16 tb + 4 g + j up to the query t = 16 w + c16
#pragma unroll
    for (int tb = 0; tb < 4; ++tb)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        pt[tb][j] = (16 * tb + 4 * g + j <= 16 * w + c16) ? pt[tb][j] : 0.f;
#pragma unroll
    for (int sp = 0; sp < 2; ++sp) {
      const frag pb = P::pack(pt[2 * sp], pt[2 * sp + 1]);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) o[nb] = P::mma(tl.VtF[nb][sp][l], pb, o[nb]);
      o[4] = P::mma(tl.DF[sp][g], pb, o[4]);
    }
    if (qt < r1) {
      const float inv = 1.0f / (o[4][0] + epsq);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) store4(Oh + (size_t)qt * kD + nb * 16 + 4 * g, o[nb] * inv);
    }
    __syncthreads();
  }
}

hipError_t launch_seg_scan(const Shape &sh, float *part, int nseg, const float *state_in,
                           float *state_out, float *total, hipStream_t st) {
  const int n = sh.M * 65;
  dim3 grid((n + 255) / 256, sh.BH);
  hipLaunchKernelGGL(k_seg_scan, grid, dim3(256), 0, st, part, nseg, n, state_in, state_out,
                     total);
  return hipGetLastError();
}

template <typename T, typename To>
static hipError_t causal_typed(const Shape &sh, const void *Q, const void *K, const void *V,
                               const void *wfr, const float *bq, const float *prefix, void *o,
                               int seg_len, int nseg, hipStream_t st) {
  dim3 grid(nseg * sh.BH);
#define FAVOR_CAUSAL_LAUNCH(MM)                                                             \
  hipLaunchKernelGGL((k_causal<T, To, MM>), grid, dim3(256), 0, st, (const T *)Q,             \
                     (const T *)K, (const T *)V, (const typename Mma<T>::frag *)wfr, bq, prefix,  \
                     (To *)o, sh.H, sh.L, seg_len,                                           \
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
                         const void *V, const void *wfr, const float *bq, const float *prefix,
                         void *o, int seg_len, int nseg, hipStream_t st) {
  if (in == Dt::BF16)
    return out == Dt::BF16
               ? causal_typed<bf16, bf16>(sh, Q, K, V, wfr, bq, prefix, o, seg_len, nseg, st)
               : causal_typed<bf16, float>(sh, Q, K, V, wfr, bq, prefix, o, seg_len, nseg, st);
  return out == Dt::BF16
             ? causal_typed<float, bf16>(sh, Q, K, V, wfr, bq, prefix, o, seg_len, nseg, st)
             : causal_typed<float, float>(sh, Q, K, V, wfr, bq, prefix, o, seg_len, nseg, st);
}

}  // namespace favor
