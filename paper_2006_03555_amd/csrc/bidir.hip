// bidir.hip - bidirectional FAVOR (Sec. 2.5, Algorithm 1) on CDNA4 matrix cores.
//
// Three launches, none of which stores a feature matrix:
//   k_kside     grid (splits * B*H). The workgroup converts the head's W to
//               W'' = (s / 2 pi) W fragments in LDS ((s / sqrt M) W for ReLU
//               features; one workgroup per head also stores them for the
//               Q side). Each workgroup streams 64-token tiles of
//               one head's K and V, rebuilds the key features K-hat on the
//               matrix cores (projection + fused cosine), and accumulates its
//               share of Buf1 = K'^T [V 1] in fp32 accumulators. D_K and the
//               sqrt(2/M) constant are folded into the value tile C~ = D_K [V 1],
//               so the feature epilogue is a single cosine. Wave w owns features
//               [w M/4, (w+1) M/4); the ones column is one more 16-wide block.
//   k_finalize  grid (fragment blocks, B*H). Sums the split partials in a fixed order
//               (deterministic) and writes Buf1^T as A-operand fragments in
//               chained feature order, with the denominator row replicated over
//               a 16-row block so that every lane of the Q side sees D-hat.
//   k_qside     grid (row tiles * B*H). Rebuilds query features Q-hat (transposed
//               projection, so the result chains straight into the next
//               product), multiplies by Buf1^T streaming over features in steps
//               of 32, and divides by the denominator. D_Q and sqrt(2/M) cancel
//               in the ratio and are never applied; a non-zero stabiliser is
//               rescaled by them instead, and without renormalisation they
//               multiply the numerator. ReLU features (generalized attention,
//               Sec. 2.2) replace the cosine by max(., 0) + keps with D = 1.
#include "favor_common.hpp"
#include "kernels.hpp"
#include "tile_common.hpp"

namespace favor {

// The head's W'' = ws W as B-operand fragments [M/16][2][64] (lane col m) and
// b'' = bs b, built into LDS by all NT threads of the
// workgroup: thread i converts the eight consecutive floats W[m][8 c .. 8 c + 7]
// (m = i / 8, c = i % 8; row-contiguous, so the loads are fully coalesced) into
// lane 16 (c % 4) + m % 16 of fragment (m / 16, c / 4). All loads are issued
// before the first LDS store.
template <typename T, int M, int NT, int KN>
__device__ __forceinline__ void fill_w_bfrags_lds(typename Mma<T>::frag (*WB)[2][64], float *bq,
                                                  const float *__restrict__ Wh,
                                                  const float *__restrict__ bh, float ws,
                                                  float bs, int Mr, float keps) {
  constexpr int N = M * 8;   // fragment lanes of the head
  constexpr int IT = N / NT;
  static_assert(N % NT == 0 && M <= NT, "thread count");
  const int tid = threadIdx.x;
  float v[IT][8];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int idx = it * NT + tid;
    if ((idx >> 3) < Mr) {   // W'' rows past the M_r drawn are zero
      load8_f32(Wh + (size_t)idx * 8, v[it]);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[it][i] = 0.f;
    }
  }
  const float bb = tid < M ? seed_row<KN>(tid, Mr, bh, bs, keps) : 0.f;
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int idx = it * NT + tid;
    const int m = idx >> 3;
    const int c = idx & 7;
    WB[m >> 4][c >> 2][16 * (c & 3) + (m & 15)] = Mma<T>::from_f32(v[it], ws);
  }
  if (tid < M) bq[tid] = bb;
}

// Workgroup = NG groups of four waves. Group G takes the 64-token tiles
// r0 + 64 (NG i + G) of the split; wave q of every group owns features
// [q M/4, (q+1) M/4). With NG = 2 two waves share each SIMD (one builds features
// while the other contracts) and one W'' build and one partial store serve the
// whole split: at the end the groups hand each other half of their
// accumulators through LDS and each stores the summed half.
template <typename T, int M, int NG>
struct KsideSmem {
  typename Mma<T>::frag WB[M / 16][2][64];   // the head's W'' fragments
  float bq[M];                               // b''
  union {
    KVTile<T> tl[NG][2];
    f32x4 red[NG][4][M / 128][5][64];   // [group][wave][half of the blocks][column block][lane]
  };
};
template <typename T, int M>
struct KsideSmem<T, M, 1> {
  typename Mma<T>::frag WB[M / 16][2][64];
  float bq[M];
  KVTile<T> tl[1][2];
};

// AGG (backward pass): K holds the queries and V the output gradient; the value
// rows are weighted by aux[t].x and aux[t].y takes the place of the ones column,
// so the partials are sum_t Q-hat_t^T [a_t dout_t, e_t]. W'' is not stored.
template <typename T, int M, int NG, int KN, bool AGG = false>
__global__ __launch_bounds__(256 * NG, sizeof(T) == 2 && NG == 1 ? 2 : 1) void k_kside(
    const T *__restrict__ K, const T *__restrict__ V, const float *__restrict__ W,
    const float *__restrict__ b, typename Mma<T>::frag *__restrict__ wfr,
    float *__restrict__ bqg, float *__restrict__ part, int H, int L, int rows_per_split,
    int nsplit, float s, float ws, float bs, float keps, int Mr, float cM,
    const float2 *__restrict__ aux) {
  const int item = xcd_item(blockIdx.x, gridDim.x);
  const int bh = item / nsplit;
  const int split = item - bh * nsplit;
  constexpr int MW = M / 4;
  constexpr int MB = MW / 16;
  static_assert(NG == 1 || MB % 2 == 0, "the groups split the feature blocks in halves");
  using P = Mma<T>;
  using frag = typename P::frag;
  __shared__ KsideSmem<T, M, NG> sm;

  const int h = bh % H;
  const int G = threadIdx.x >> 8;
  const int tid = threadIdx.x & 255;   // thread within the group
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;
  const int r0 = split * rows_per_split;
  const int r1 = min(L, r0 + rows_per_split);
  const int ntiles = (r1 - r0 + 63) / 64;
  const int nit = (ntiles + NG - 1) / NG;   // every group runs nit iterations

  const T *Kh = K + (size_t)bh * L * kD;
  const T *Vh = V + (size_t)bh * L * kD;
  const float s2half = 0.5f * s * s;

  // first tile's loads in flight while W'' is built
  TileRegs<T> rg;
  load_tile_regs<T>(rg, Kh, Vh, r0 + 64 * G, r1, tid);

  fill_w_bfrags_lds<T, M, 256 * NG, KN>(sm.WB, sm.bq, W + (size_t)h * Mr * kD,
                                        b + (size_t)h * Mr, ws, bs, Mr, keps);
  __syncthreads();
  // one workgroup per head stores W'' and b'' for later launches
  if (!AGG && bh < H && split == 0) {
    constexpr int NF = (M / 16) * 2 * 64;
    frag *dst = wfr + (size_t)h * NF;
    for (int i = threadIdx.x; i < NF; i += 256 * NG) dst[i] = (&sm.WB[0][0][0])[i];
    if (threadIdx.x < M) bqg[(size_t)h * M + threadIdx.x] = sm.bq[threadIdx.x];
  }
  frag Wf[MB][2];
  f32x4 bC[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    Wf[mb][0] = sm.WB[w * MB + mb][0][l];
    Wf[mb][1] = sm.WB[w * MB + mb][1][l];
    const float bb = sm.bq[16 * (w * MB + mb) + c16];
    bC[mb] = f32x4{bb, bb, bb, bb};
  }
  frag sel[2] = {select_frag<T>(0), select_frag<T>(1)};

  f32x4 acc[MB][5];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < 5; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // the row weights of the backward pass's aggregation (0 past r1)
  auto stage_agg = [&](KVTile<T> &tl, int t0) __attribute__((always_inline)) {
    const int t = t0 + (tid >> 2);
    const float2 a = t < r1 ? aux[(size_t)bh * L + t] : float2{0.f, 0.f};
    stage_tile_rows<T>(tl, rg, sel, a.x, a.y, tid);
  };
  if constexpr (AGG)
    stage_agg(sm.tl[G][0], r0 + 64 * G);
  else
    stage_tile<T, KN>(sm.tl[G][0], rg, sel, r0 + 64 * G, r1, s2half, cM, tid);
  __syncthreads();
  int buf = 0;
  for (int it = 0; it < nit; ++it, buf ^= 1) {
    // tiles past r1 (a group's last one when ntiles is not a multiple of NG)
    // load nothing and stage zero value weights
    const int tn = r0 + 64 * (NG * (it + 1) + G);
    const bool next = it + 1 < nit;
    if (next) load_tile_regs<T>(rg, Kh, Vh, tn, r1, tid);
    const KVTile<T> &tc = sm.tl[G][buf];
#pragma unroll
    for (int sidx = 0; sidx < 2; ++sidx) {
      f32x4 kf[MB][2];
      key_features<T, MB, KN>(tc, Wf, bC, sidx, kf);
      frag vb[4];
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) vb[nb] = tc.VtF[nb][sidx][l];
      const frag db = tc.DF[sidx][g];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const frag a = P::pack(kf[mb][0], kf[mb][1]);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = P::mma(a, vb[nb], acc[mb][nb]);
        acc[mb][4] = P::mma(a, db, acc[mb][4]);
      }
    }
    if (next) {
      if constexpr (AGG)
        stage_agg(sm.tl[G][buf ^ 1], tn);
      else
        stage_tile<T, KN>(sm.tl[G][buf ^ 1], rg, sel, tn, r1, s2half, cM, tid);
    }
    __syncthreads();
  }

  float *dst = part + ((size_t)bh * nsplit + split) * M * 65;
  auto store_block = [&](int mb, const f32x4 (&a)[5]) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = w * MW + mb * 16 + 4 * g + j;
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) dst[m * 65 + nb * 16 + c16] = a[nb][j];
      if (c16 == 0) dst[m * 65 + 64] = a[4][j];
    }
  };
  if constexpr (NG == 1) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) store_block(mb, acc[mb]);
  } else {
    // group G stores feature blocks [G MB/2, (G+1) MB/2) of every wave and hands
    // the other half to the group that stores it (the tile buffers are free)
    constexpr int HB = MB / 2;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
      if ((mb / HB) != G)
#pragma unroll
        for (int nb = 0; nb < 5; ++nb) sm.red[G][w][mb % HB][nb][l] = acc[mb][nb];
    __syncthreads();
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
      if ((mb / HB) == G) {
        f32x4 a[5];
#pragma unroll
        for (int nb = 0; nb < 5; ++nb) {
          const f32x4 o = sm.red[G ^ 1][w][mb % HB][nb][l];
#pragma unroll
          for (int j = 0; j < 4; ++j) a[nb][j] = acc[mb][nb][j] + o[j];
        }
        store_block(mb, a);
      }
  }
}

// Four threads per (fragment block, lane): each sums every fourth split of the
// fragment's 8 chained-order entries, the four partial sums are combined in a
// fixed order (deterministic), and the first thread stores 16/32 B.
template <typename T, int M>
__global__ __launch_bounds__(256) void k_finalize(const float *__restrict__ part, int nsplit,
                                                  typename Mma<T>::frag *__restrict__ frags) {
  constexpr int NS = M / 32;
  const int bh = blockIdx.y;
  const int unit = blockIdx.x * 64 + (threadIdx.x >> 2);  // (fragment block, lane)
  const int q = threadIdx.x & 3;
  if (unit >= 5 * NS * 64) return;
  const int fi = unit >> 6;                               // fragment block = nb * NS + sidx
  const int l = unit & 63;
  const int nb = fi / NS;
  const int sidx = fi - nb * NS;
  const int g = l >> 4;
  const int n = nb < 4 ? perm_col(nb, l & 15) : 64;   // lane row = value column (permuted)
  const float *src = part + (size_t)bh * nsplit * M * 65;
  float v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = 0.f;
  for (int sp = q; sp < nsplit; sp += 4) {
    const float *ps = src + (size_t)sp * M * 65 + n;
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += ps[(sidx * 32 + 16 * (i >> 2) + 4 * g + (i & 3)) * 65];
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    v[i] += __shfl_xor(v[i], 1);
    v[i] += __shfl_xor(v[i], 2);
  }
  if (q == 0) frags[((size_t)bh * 5 * NS + fi) * 64 + l] = Mma<T>::from_f32(v, 1.f);
}

// Rows per workgroup: 4 waves x TBW blocks of 16 rows.
template <typename T> struct QsideCfg { static constexpr int TBW = 4; };
template <> struct QsideCfg<float> { static constexpr int TBW = 2; };

// Query fragments of one tile for this wave: rows rbase + 16 tb + lane % 16.
template <typename T, int TBW>
__device__ __forceinline__ void load_q_frags(typename Mma<T>::frag (&qf)[TBW][2],
                                             const T *__restrict__ Qh, int rbase, int L) {
  const int l = lane_id();
#pragma unroll
  for (int tb = 0; tb < TBW; ++tb) {
    const int t = rbase + tb * 16 + (l & 15);
    if (t < L) {
      qf[tb][0] = load_frag<T>(Qh + (size_t)t * kD + 8 * (l >> 4));
      qf[tb][1] = load_frag<T>(Qh + (size_t)t * kD + 32 + 8 * (l >> 4));
    } else {
      qf[tb][0] = Mma<T>::splat(0.f);
      qf[tb][1] = Mma<T>::splat(0.f);
    }
  }
}

// Finalisation of a query row: divide by D-hat, divide by D-hat + eps, or
// (renormalisation off) scale the numerator by the query factor.
constexpr int kFinDiv = 0;
constexpr int kFinDivEps = 1;
constexpr int kFinScale = 2;

// SAVE: also write the row's 1 / (D-hat + eps) in the units of the unscaled
// features (rsave [B*H][L]), which the backward pass reads.
template <typename T, typename To, int M, int KN, int FIN, bool SAVE>
__global__ __launch_bounds__(256, sizeof(T) == 2 ? 2 : 1) void k_qside(const T *__restrict__ Q,
                                                  const typename Mma<T>::frag *__restrict__ wfr,
                                                  const float *__restrict__ bqg,
                                                  const typename Mma<T>::frag *__restrict__ frags,
                                                  To *__restrict__ out, float *__restrict__ rsave,
                                                  int H, int L, float s, float eps, float cM,
                                                  int ntiles, int nitems) {
  constexpr int NS = M / 32;
  constexpr int TBW = QsideCfg<T>::TBW;
  using P = Mma<T>;
  using frag = typename P::frag;
  __shared__ frag WA[M / 16][2][64];
  __shared__ frag BF[5][NS][64];
  __shared__ float bq[M];

  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;

  int begin, end;
  xcd_range(blockIdx.x, gridDim.x, nitems, begin, end);
  if (begin >= end) return;

  frag qn[TBW][2];
  {
    const int bh = begin / ntiles;
    load_q_frags<T, TBW>(qn, Q + (size_t)bh * L * kD,
                         (begin - bh * ntiles) * (64 * TBW) + w * (16 * TBW), L);
  }
  int cur = -1;
  for (int item = begin; item < end; ++item) {
    const int bh = item / ntiles;
    const int tile = item - bh * ntiles;
    if (bh != cur) {   // the head's W'' and Buf1^T fragments into LDS
      const int h = bh % H;
      __syncthreads();
      copy_frags<frag, (M / 16) * 2 * 64>(&WA[0][0][0], wfr + (size_t)h * (M / 16) * 2 * 64);
      copy_frags<frag, 5 * NS * 64>(&BF[0][0][0], frags + (size_t)bh * 5 * NS * 64);
      if (tid < M) bq[tid] = bqg[(size_t)h * M + tid];
      __syncthreads();
      cur = bh;
    }
    const int rbase = tile * (64 * TBW) + w * (16 * TBW);
    frag qf[TBW][2];
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      qf[tb][0] = qn[tb][0];
      qf[tb][1] = qn[tb][1];
    }
    if (item + 1 < end) {   // prefetch the next tile's queries
      const int bn = (item + 1) / ntiles;
      load_q_frags<T, TBW>(qn, Q + (size_t)bn * L * kD,
                           (item + 1 - bn * ntiles) * (64 * TBW) + w * (16 * TBW), L);
    }
    // per row: the stabiliser in units of the unscaled features (kFinDivEps) or
    // the factor D_Q sqrt(2/M) the features omit (kFinScale); ReLU features
    // have D_Q = 1 and carry their own scale
    float epsq[TBW];
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      epsq[tb] = FIN == kFinDiv ? 0.f : FIN == kFinDivEps ? eps : 1.f;
      if constexpr (KN == kCos && FIN != kFinDiv) {
        float nrm = sq_sum16(qf[tb]);
        nrm += __shfl_xor(nrm, 16);
        nrm += __shfl_xor(nrm, 32);
        // features here omit D_Q sqrt(2/M); the stabiliser is divided by it instead
        const float dq = cM * expf(0.5f * s * s * nrm);
        epsq[tb] = FIN == kFinDivEps ? eps / dq : dq;
      }
    }

    // 32 features per step: project and take the cosines, then contract with
    // Buf1^T (the first step starts the accumulators from zero)
    f32x4 acc[5][TBW];
    auto feature_step = [&](int sidx, bool first) __attribute__((always_inline)) {
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
          for (int j = 0; j < 4; ++j) pf[hh][tb][j] = feature<KN, P>(p[j], bcv[j]);
        }
      }
      frag qb[TBW];
#pragma unroll
      for (int tb = 0; tb < TBW; ++tb) qb[tb] = P::pack(pf[0][tb], pf[1][tb]);
#pragma unroll
      for (int nb = 0; nb < 5; ++nb) {
        const frag a = BF[nb][sidx][l];
#pragma unroll
        for (int tb = 0; tb < TBW; ++tb)
          acc[nb][tb] = P::mma(a, qb[tb], first ? f32x4{0.f, 0.f, 0.f, 0.f} : acc[nb][tb]);
      }
    };
    feature_step(0, true);
#pragma unroll 2
    for (int sidx = 1; sidx < NS; ++sidx) feature_step(sidx, false);

    To *Oh = out + (size_t)bh * L * kD;
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      const int t = rbase + tb * 16 + c16;
      if (t < L) {
        const float inv =
            FIN == kFinScale ? epsq[tb] : __builtin_amdgcn_rcpf(acc[4][tb][0] + epsq[tb]);
        if constexpr (SAVE) {
          if (g == 0) rsave[(size_t)bh * L + t] = inv;
        }
        // blocks 2 p, 2 p + 1 hold value columns 32 p + 8 g .. + 7 in this lane
#pragma unroll
        for (int pp = 0; pp < 2; ++pp)
          store8(Oh + (size_t)t * kD + 32 * pp + 8 * g, acc[2 * pp][tb] * inv,
                 acc[2 * pp + 1][tb] * inv);
      }
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

template <int KN, bool AGG>
static hipError_t kside_kernel(const Shape &sh, Dt in, const void *K, const void *V,
                               const float *W, const float *b, void *wfr, float *bq, float *part,
                               int rows_per_split, int nsplit, hipStream_t st,
                               const float2 *aux) {
  dim3 grid(nsplit * sh.BH);
  float ws, bs;
  feature_scales(sh, ws, bs);
  if (in == Dt::BF16) {
    FAVOR_DISPATCH_M(sh.M,
                     hipLaunchKernelGGL((k_kside<bf16, MM, kside_groups(Dt::BF16, MM), KN, AGG>),
                                        grid, dim3(256 * kside_groups(Dt::BF16, MM)), 0, st,
                                        (const bf16 *)K, (const bf16 *)V, W, b,
                                        (Mma<bf16>::frag *)wfr, bq, part, sh.H, sh.L,
                                        rows_per_split, nsplit, sh.s, ws, bs, sh.keps, sh.Mr,
                                        feature_norm(sh), aux));
  } else {
    FAVOR_DISPATCH_M(sh.M, hipLaunchKernelGGL((k_kside<float, MM, 1, KN, AGG>), grid, dim3(256),
                                               0, st, (const float *)K, (const float *)V, W, b,
                                               (Mma<float>::frag *)wfr, bq, part, sh.H, sh.L,
                                               rows_per_split, nsplit, sh.s, ws, bs, sh.keps,
                                               sh.Mr, feature_norm(sh),
                                               aux));
  }
  return hipGetLastError();
}

hipError_t launch_kside(const Shape &sh, Dt in, const void *K, const void *V, const float *W,
                        const float *b, void *wfr, float *bq, float *part, int rows_per_split,
                        int nsplit, hipStream_t st) {
  return sh.kernel == 1 ? kside_kernel<kRelu, false>(sh, in, K, V, W, b, wfr, bq, part,
                                                     rows_per_split, nsplit, st, nullptr)
                        : kside_kernel<kCos, false>(sh, in, K, V, W, b, wfr, bq, part,
                                                    rows_per_split, nsplit, st, nullptr);
}

hipError_t launch_kside_agg(const Shape &sh, Dt in, const void *Q, const void *dout,
                            const float *W, const float *b, const float2 *aux, float *part,
                            int rows_per_split, int nsplit, hipStream_t st) {
  return sh.kernel == 1 ? kside_kernel<kRelu, true>(sh, in, Q, dout, W, b, nullptr, nullptr,
                                                    part, rows_per_split, nsplit, st, aux)
                        : kside_kernel<kCos, true>(sh, in, Q, dout, W, b, nullptr, nullptr, part,
                                                   rows_per_split, nsplit, st, aux);
}

hipError_t launch_finalize(const Shape &sh, Dt in, const float *part, int nsplit, void *frags,
                           hipStream_t st) {
  dim3 grid((5 * (sh.M / 32) * 64 + 63) / 64, sh.BH);
  if (in == Dt::BF16) {
    FAVOR_DISPATCH_M(sh.M, hipLaunchKernelGGL((k_finalize<bf16, MM>), grid, dim3(256), 0, st,
                                               part, nsplit, (Mma<bf16>::frag *)frags));
  } else {
    FAVOR_DISPATCH_M(sh.M, hipLaunchKernelGGL((k_finalize<float, MM>), grid, dim3(256), 0, st,
                                               part, nsplit, (Mma<float>::frag *)frags));
  }
  return hipGetLastError();
}

// Persistent Q side: at most two workgroups per CU, each walking a contiguous
// XCD-local range of row tiles.
constexpr int kQsideMaxWorkgroups = 512;

template <typename T, typename To, int KN, int FIN, bool SAVE = false>
static hipError_t qside_launch(const Shape &sh, const void *Q, const void *wfr, const float *bq,
                               const void *frags, void *o, hipStream_t st,
                               float *rsave = nullptr) {
  const int rows = 64 * QsideCfg<T>::TBW;
  const int ntiles = (sh.L + rows - 1) / rows;
  const int nitems = ntiles * sh.BH;
  dim3 grid(min(nitems, kQsideMaxWorkgroups));
  FAVOR_DISPATCH_M(sh.M, hipLaunchKernelGGL((k_qside<T, To, MM, KN, FIN, SAVE>), grid, dim3(256),
                                             0, st, (const T *)Q,
                                             (const typename Mma<T>::frag *)wfr, bq,
                                             (const typename Mma<T>::frag *)frags, (To *)o, rsave,
                                             sh.H, sh.L, sh.s, sh.eps, feature_norm(sh), ntiles,
                                             nitems));
  return hipGetLastError();
}

template <typename T, typename To, int KN>
static hipError_t qside_kernel(const Shape &sh, const void *Q, const void *wfr, const float *bq,
                               const void *frags, void *o, hipStream_t st) {
  if (!sh.renorm) return qside_launch<T, To, KN, kFinScale>(sh, Q, wfr, bq, frags, o, st);
  if (sh.eps != 0.f) return qside_launch<T, To, KN, kFinDivEps>(sh, Q, wfr, bq, frags, o, st);
  return qside_launch<T, To, KN, kFinDiv>(sh, Q, wfr, bq, frags, o, st);
}

template <typename T, typename To>
static hipError_t qside_typed(const Shape &sh, const void *Q, const void *wfr, const float *bq,
                              const void *frags, void *o, hipStream_t st) {
  return sh.kernel == 1 ? qside_kernel<T, To, kRelu>(sh, Q, wfr, bq, frags, o, st)
                        : qside_kernel<T, To, kCos>(sh, Q, wfr, bq, frags, o, st);
}

template <typename T, int KN>
static hipError_t qside_save(const Shape &sh, const void *Q, const void *wfr, const float *bq,
                             const void *frags, void *o, float *rsave, hipStream_t st) {
  if (sh.eps != 0.f)
    return qside_launch<T, T, KN, kFinDivEps, true>(sh, Q, wfr, bq, frags, o, st, rsave);
  return qside_launch<T, T, KN, kFinDiv, true>(sh, Q, wfr, bq, frags, o, st, rsave);
}

hipError_t launch_qside_save(const Shape &sh, Dt in, const void *Q, const void *wfr,
                             const float *bq, const void *frags, void *o, float *rsave,
                             hipStream_t st) {
  if (!sh.renorm) return hipErrorInvalidValue;
  if (in == Dt::BF16)
    return sh.kernel == 1 ? qside_save<bf16, kRelu>(sh, Q, wfr, bq, frags, o, rsave, st)
                          : qside_save<bf16, kCos>(sh, Q, wfr, bq, frags, o, rsave, st);
  return sh.kernel == 1 ? qside_save<float, kRelu>(sh, Q, wfr, bq, frags, o, rsave, st)
                        : qside_save<float, kCos>(sh, Q, wfr, bq, frags, o, rsave, st);
}

hipError_t launch_qside(const Shape &sh, Dt in, Dt out, const void *Q, const void *wfr,
                        const float *bq, const void *frags, void *o, hipStream_t st) {
  if (in == Dt::BF16)
    return out == Dt::BF16 ? qside_typed<bf16, bf16>(sh, Q, wfr, bq, frags, o, st)
                           : qside_typed<bf16, float>(sh, Q, wfr, bq, frags, o, st);
  return out == Dt::BF16 ? qside_typed<float, bf16>(sh, Q, wfr, bq, frags, o, st)
                         : qside_typed<float, float>(sh, Q, wfr, bq, frags, o, st);
}

}  // namespace favor
