// backward.hip - gradients of FAVOR attention with respect to Q, K, V (and the
// carried causal state): Algorithm 1 (Sec. 2.5) and Eq. cumsum (Sec. 2.5.1)
// taken in reverse, on the CDNA4 matrix cores.
//
// Notation: q-hat, k-hat are the features without their D factors (cos features:
// cos(2 pi (W'' x + b'')); ReLU features: max(W'' x, 0) + keps), D~ = D_X sqrt(2/M)
// (1 for ReLU), C~ = D~_K [V 1]. With S the M x (d+1) aggregate a row sees
// (Buf1 for the bidirectional form, the prefix G^PS_i for the causal one) and
// r = 1 / (D-hat + eps) in units of q-hat, the gradient of a row's output
// passes back as
//   u = [dout, -dout . out] (renormalised) or [dout, 0],  alpha = r or D~_Q,
//   g~ = S u                  (M; the true dQ' is alpha g~ / D~_Q)
//   dQ = alpha [s^2 (g~ . q-hat) q - (g~ o sin) (s W)]   (cos features)
//      = alpha (g~ o [W'' q > 0]) W''                      (ReLU features)
// and the key side receives, per row, q-hat (x) u~ with u~ = alpha u:
//   R = sum of q-hat_i (x) u~_i over the rows that see key j (all rows, or i >= j),
//   dK'_j = R C_j,  dV_j = D~_K R^T k-hat_j (first d columns),
//   dK = D~_K [s^2 (h . k-hat) k - (h o sin) (s W)] with h = dK', or (h o step) W''.
// Kernels:
//   k_bwd_dq     per row tile (bidirectional, persistent) or per 64-token chunk
//                (causal): projection, features and slopes of its queries on the
//                matrix cores, g~ = S u plus, causal, the keys of the chunk up to
//                the query (tril(C~ u^T) against the chunk's key features), the
//                input-gradient product with W''^T; writes dQ and (alpha, alpha u_d)
//   k_bwd_dkv    per key tile / chunk: key features and slopes, h = R C_j plus,
//                causal, the queries of the chunk from the key on; dV = R^T k-hat plus,
//                causal, tril-transposed (q-hat . k-hat) u~; dK as above
//   k_sum_splits fixed-order sum of split partials (Buf1, dBuf1)
//   k_suffix_scan exclusive suffix scan of chunk aggregates plus dstate_out (the
//                causal R per chunk) and dstate_in
// The aggregation of q-hat (x) u~ over row ranges is k_kside's weighted mode.
#include <type_traits>

#include "favor_common.hpp"
#include "kernels.hpp"
#include "tile_common.hpp"

namespace favor {

constexpr int kBwdBidirThreads = 512;   // the bidirectional kernels: two waves per SIMD

// Copy N fragments global -> LDS with the whole workgroup.
template <typename F, int N>
__device__ __forceinline__ void copy_frags_wg(F *__restrict__ dst, const F *__restrict__ src) {
  for (int idx = threadIdx.x; idx < N; idx += blockDim.x) dst[idx] = src[idx];
}

// ------------------------------------------------------------ small kernels
__global__ __launch_bounds__(256) void k_sum_splits(const f32x4 *__restrict__ part, int ns, int n4,
                                                    f32x4 *__restrict__ dst) {
  const int bh = blockIdx.y;
  const int u = blockIdx.x * 256 + threadIdx.x;
  if (u >= n4) return;
  const f32x4 *p = part + (size_t)bh * ns * n4 + u;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  int sp = 0;
  for (; sp + 4 <= ns; sp += 4) {   // four loads in flight, added in order
    const f32x4 a = p[(size_t)sp * n4], b = p[(size_t)(sp + 1) * n4];
    const f32x4 c = p[(size_t)(sp + 2) * n4], d = p[(size_t)(sp + 3) * n4];
    acc += a;
    acc += b;
    acc += c;
    acc += d;
  }
  for (; sp < ns; ++sp) acc += p[(size_t)sp * n4];
  dst[(size_t)bh * n4 + u] = acc;
}

// part [BH][nch][n4]: chunk c becomes dsout + sum_{c' > c} part[c']; the total
// (dsout + every chunk) goes to dsin. Either pointer may be null. dsout and dsin
// hold the M_r rows drawn (n4u = M_r 65 / 4 units per head; the rows past them
// are padding, zero in part). bias (nullable, [BH][n4] like part): added to
// every chunk's suffix but not to dsin: the bidirectional aggregate dBuf1 that
// every key of the sequence sees, when both directions are differentiated in
// one pass.
__global__ __launch_bounds__(256) void k_suffix_scan(f32x4 *__restrict__ part, int nch, int n4,
                                                     int n4u, const f32x4 *__restrict__ dsout,
                                                     f32x4 *__restrict__ dsin,
                                                     const f32x4 *__restrict__ bias) {
  const int bh = blockIdx.y;
  const int u = blockIdx.x * 256 + threadIdx.x;
  if (u >= n4) return;
  const bool drawn = u < n4u;
  f32x4 *p = part + (size_t)bh * nch * n4 + u;
  f32x4 run = dsout && drawn ? dsout[(size_t)bh * n4u + u] : f32x4{0.f, 0.f, 0.f, 0.f};
  const f32x4 bv = bias ? bias[(size_t)bh * n4 + u] : f32x4{0.f, 0.f, 0.f, 0.f};
  int c = nch - 1;
  for (; c >= 7; c -= 8) {   // eight loads in flight
    f32x4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = p[(size_t)(c - k) * n4];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      p[(size_t)(c - k) * n4] = run + bv;
      run += v[k];
    }
  }
  for (; c >= 0; --c) {
    const f32x4 v = p[(size_t)c * n4];
    p[(size_t)c * n4] = run + bv;
    run += v;
  }
  if (dsin && drawn) dsin[(size_t)bh * n4u + u] = run;
}

// ------------------------------------------------------------ LDS builders
// W''^T for the input-gradient products as A operand: row = input column
// perm_col(kb, lane % 16) (store order), k = feature m = 32 s + chained(g, i).
template <typename T, int M>
__device__ __forceinline__ void build_wt(typename Mma<T>::frag (*WT)[M / 32][64],
                                         const float *__restrict__ Wh, float scale, int Mr) {
  constexpr int NS = M / 32;
  for (int idx = threadIdx.x; idx < 4 * NS * 64; idx += blockDim.x) {
    const int l = idx & 63;
    const int s = (idx >> 6) % NS;
    const int kb = idx / (64 * NS);
    const int g = l >> 4;
    const int k = perm_col(kb, l & 15);
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int m = 32 * s + 16 * (i >> 2) + 4 * g + (i & 3);
      v[i] = m < Mr ? Wh[m * kD + k] : 0.f;   // rows past the M_r drawn are zero
    }
    WT[kb][s][l] = Mma<T>::from_f32(v, scale);
  }
}

// An aggregate S [M][65] (fp32, row-major) as A operand over its value
// columns: row = m = 16 mb + lane % 16, k = column 32 ks + 8 g + i (loaded
// order); its last column separately (sz).
template <typename T, int M>
__device__ __forceinline__ void build_state_rows(typename Mma<T>::frag (*SA)[2][64], float *sz,
                                                 const float *__restrict__ S) {
  for (int idx = threadIdx.x; idx < (M / 16) * 2 * 64; idx += blockDim.x) {
    const int l = idx & 63;
    const int ks = (idx >> 6) & 1;
    const int mb = idx >> 7;
    const float *row = S + (size_t)(16 * mb + (l & 15)) * 65 + 32 * ks + 8 * (l >> 4);
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = row[i];
    SA[mb][ks][l] = Mma<T>::from_f32(v, 1.f);
  }
  for (int m = threadIdx.x; m < M; m += blockDim.x) sz[m] = S[(size_t)m * 65 + 64];
}

// The value columns of S as A operand over features: row = column
// perm_col(nb, lane % 16), k = m = 32 s + chained(g, i).
template <typename T, int M>
__device__ __forceinline__ void build_state_cols(typename Mma<T>::frag (*SB)[M / 32][64],
                                                 const float *__restrict__ S) {
  constexpr int NS = M / 32;
  for (int idx = threadIdx.x; idx < 4 * NS * 64; idx += blockDim.x) {
    const int l = idx & 63;
    const int s = (idx >> 6) % NS;
    const int nb = idx / (64 * NS);
    const int g = l >> 4;
    const int n = perm_col(nb, l & 15);
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = S[(size_t)(32 * s + 16 * (i >> 2) + 4 * g + (i & 3)) * 65 + n];
    SB[nb][s][l] = Mma<T>::from_f32(v, 1.f);
  }
}

// Selection matrix in loaded k order: B[k][c] = (k == 8 (c / 4) + 4 half + c % 4),
// which moves value column perm_col(2 kh + half, c) of a row fragment of k-step
// kh into lane c.
template <typename T>
__device__ __forceinline__ typename Mma<T>::frag select_perm(int half) {
  const int l = lane_id();
  const int c = l & 15;
  float v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (8 * (l >> 4) + i == 8 * (c >> 2) + 4 * half + (c & 3)) ? 1.f : 0.f;
  return Mma<T>::from_f32(v, 1.f);
}

// Row fragments of a [L][64] tensor (lane row t = row0 + lane % 16, columns
// 8 g .. and 32 + 8 g ..), zero past L.
template <typename T>
__device__ __forceinline__ void load_rows64(typename Mma<T>::frag (&f)[2], const T *__restrict__ X,
                                            int t, int L) {
  const int g = lane_id() >> 4;
  if (t < L) {
    f[0] = load_frag<T>(X + (size_t)t * kD + 8 * g);
    f[1] = load_frag<T>(X + (size_t)t * kD + 32 + 8 * g);
  } else {
    f[0] = Mma<T>::splat(0.f);
    f[1] = Mma<T>::splat(0.f);
  }
}

// Dot product of the 16 values of two fragment pairs (a lane's share of two
// rows): dot2 on bf16 pairs (two exact products and an fp32 sum per
// instruction, no conversions), fused multiply-adds on fp32 values.
__device__ __forceinline__ float dot16(const bf16x8 (&a)[2], const bf16x8 (&b)[2]) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  struct Pairs { bf16x2 p[4]; };
  float n = 0.f;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const Pairs x = __builtin_bit_cast(Pairs, a[k]);
    const Pairs y = __builtin_bit_cast(Pairs, b[k]);
#pragma unroll
    for (int i = 0; i < 4; ++i) n = __builtin_amdgcn_fdot2_f32_bf16(x.p[i], y.p[i], n, false);
  }
  return n;
}
__device__ __forceinline__ float dot16(const f32x8 (&a)[2], const f32x8 (&b)[2]) {
  float n = 0.f;
#pragma unroll
  for (int k = 0; k < 2; ++k)
#pragma unroll
    for (int i = 0; i < 8; ++i) n = fmaf(a[k][i], b[k][i], n);
  return n;
}
template <typename T>
__device__ __forceinline__ float sq_norm16(const typename Mma<T>::frag (&f)[2]) {
  float n = sq_sum16(f);
  n += __shfl_xor(n, 16);
  n += __shfl_xor(n, 32);
  return n;
}

// Features of blocks mb0 .. mb0 + MB - 1 of the 64 rows of a chunk (lane row =
// row 16 tb + lane % 16 of rf[tb]) in the key orientation, packed as A operand
// (row = feature m, k = the chunk's rows in chained order, halves sidx = 0, 1).
template <typename T, int MB, int KN>
__device__ __forceinline__ void chunk_features_t(typename Mma<T>::frag (*dst)[2][64],
                                                 const typename Mma<T>::frag (*WA)[2][64],
                                                 const float *bq,
                                                 const typename Mma<T>::frag (&rf)[4][2],
                                                 int mb0) {
  using P = Mma<T>;
  const int l = lane_id();
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int mbg = mb0 + mb;
    const auto b0 = WA[mbg][0][l];
    const auto b1 = WA[mbg][1][l];
    const float bb = bq[16 * mbg + (l & 15)];
    f32x4 f[4];
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      f32x4 p = P::mma(rf[tb][0], b0, f32x4{bb, bb, bb, bb});
      p = P::mma(rf[tb][1], b1, p);
#pragma unroll
      for (int j = 0; j < 4; ++j) f[tb][j] = feature<KN, P>(p[j], bb);
    }
    dst[mbg][0][l] = P::pack(f[0], f[1]);
    dst[mbg][1][l] = P::pack(f[2], f[3]);
  }
}

// ------------------------------------------------------------ shared row work
// Gradient of one 16-row block of queries (lane column = query i = row0 + lane % 16;
// qf, df the query and dout fragments, alpha and u_d of the row), with the
// aggregate S in LDS (SA rows over value columns, sz its column d), W'' (WA, bq)
// and the input-gradient matrix WT. INTRA adds g~ += K-hat^T P2 with the chunk's
// key features KT (row m, k = keys) and P2 packed as B operand (k = keys).
template <typename T, int M, int KN, bool INTRA>
__device__ __forceinline__ void query_grad(
    const typename Mma<T>::frag (*WA)[2][64], const float *bq,
    const typename Mma<T>::frag (*WT)[M / 32][64], const typename Mma<T>::frag (*SA)[2][64],
    const float *sz, const typename Mma<T>::frag (*KT)[2][64],
    const typename Mma<T>::frag (&pb2)[2], const typename Mma<T>::frag (&qf)[2],
    const typename Mma<T>::frag (&df)[2], float alpha, float ud, float s,
    f32x4 (&dacc)[4], float &dot2, int s0 = 0, int s1 = M / 32) {
  using P = Mma<T>;
  using frag = typename P::frag;
  constexpr float sgn = KN == kCos ? -1.f : 1.f;
  // two feature steps per unrolled iteration; at M = 64 (two steps in all) a
  // full unroll would spill, so the loop stays rolled
  constexpr int kFeatureUnroll = M > 64 ? 2 : 1;
  const int l = lane_id();
  const int g = l >> 4;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) dacc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
  dot2 = 0.f;
#pragma unroll kFeatureUnroll
  for (int sidx = s0; sidx < s1; ++sidx) {
    f32x4 G[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int mb = 2 * sidx + hh;
      const f32x4 bcv = *reinterpret_cast<const f32x4 *>(&bq[16 * mb + 4 * g]);
      const f32x4 szv = *reinterpret_cast<const f32x4 *>(&sz[16 * mb + 4 * g]);
      f32x4 p = P::mma(WA[mb][0][l], qf[0], bcv);
      p = P::mma(WA[mb][1][l], qf[1], p);
      f32x4 gt = P::mma(SA[mb][0][l], df[0], f32x4{0.f, 0.f, 0.f, 0.f});
      gt = P::mma(SA[mb][1][l], df[1], gt);
      if constexpr (INTRA) {
        gt = P::mma(KT[mb][0][l], pb2[0], gt);
        gt = P::mma(KT[mb][1][l], pb2[1], gt);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float gj = fmaf(szv[j], ud, gt[j]);
        dot2 = fmaf(gj, feature<KN, P>(p[j], bcv[j]), dot2);
        G[hh][j] = sgn * alpha * gj * feature_slope<KN, P>(p[j], bcv[j]);
      }
    }
    const frag gb = P::pack(G[0], G[1]);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) dacc[kb] = P::mma(WT[kb][sidx][l], gb, dacc[kb]);
  }
  dot2 += __shfl_xor(dot2, 16);
  dot2 += __shfl_xor(dot2, 32);
}

// dQ row store: dQ = WT G + alpha s^2 (g~ . q-hat) q (cos features).
// Store 8 consecutive values, or (ACC) add them to what dst holds: the fp32
// gradients of a feature slice after the first (a gradient is a sum over
// features, see the launchers), or the gradient of one direction onto the
// other's when both are differentiated in one call (bf16 too: one more
// rounding of the sum).
template <bool ACC, typename T>
__device__ __forceinline__ void put8(T *p, f32x4 a, f32x4 b) {
  if constexpr (ACC) {
    float v[8];
    load8_f32(p, v);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      a[i] += v[i];
      b[i] += v[4 + i];
    }
  }
  store8(p, a, b);
}

template <typename T, int KN, bool ACC = false>
__device__ __forceinline__ void store_qgrad(T *dst, const f32x4 (&dacc)[4],
                                            const typename Mma<T>::frag (&qf)[2], float alpha,
                                            float dot2, float s) {
  const int g = lane_id() >> 4;
  const float cx = KN == kCos ? alpha * s * s * dot2 : 0.f;
#pragma unroll
  for (int pp = 0; pp < 2; ++pp) {
    f32x4 lo, hi;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo[e] = fmaf(cx, to_f32(qf[pp][e]), dacc[2 * pp][e]);
      hi[e] = fmaf(cx, to_f32(qf[pp][4 + e]), dacc[2 * pp + 1][e]);
    }
    put8<ACC>(dst + 32 * pp + 8 * g, lo, hi);
  }
}

// alpha and u_d of query row i (lane column) from its query, dout and output
// fragments and its saved row scale rs (renormalised; 0 past the end).
template <typename T, int KN, bool RN>
__device__ __forceinline__ void row_weights_loaded(const typename Mma<T>::frag (&qf)[2],
                                                   const typename Mma<T>::frag (&df)[2],
                                                   const typename Mma<T>::frag (&of)[2], float rs,
                                                   int i, int L, float cM, float s2half,
                                                   float &alpha, float &ud) {
  if constexpr (RN) {
    float dot = dot16(df, of);
    dot += __shfl_xor(dot, 16);
    dot += __shfl_xor(dot, 32);
    alpha = rs;
    ud = -dot;
  } else {
    float a = 1.f;
    if constexpr (KN == kCos) a = cM * expf(s2half * sq_norm16<T>(qf));
    alpha = i < L ? a : 0.f;
    ud = 0.f;
  }
}

// The output row and saved row scale of query row i (renormalised calls).
template <typename T, bool RN>
__device__ __forceinline__ void load_row_stats(typename Mma<T>::frag (&of)[2], float &rs,
                                               const T *__restrict__ Oh,
                                               const float *__restrict__ rsave_h, int i, int L) {
  if constexpr (RN) {
    load_rows64<T>(of, Oh, i, L);
    rs = i < L ? rsave_h[i] : 0.f;
  } else {
    rs = 0.f;
  }
}

template <typename T, int KN, bool RN>
__device__ __forceinline__ void row_weights(const typename Mma<T>::frag (&qf)[2],
                                            const typename Mma<T>::frag (&df)[2],
                                            const T *__restrict__ Oh,
                                            const float *__restrict__ rsave_h, int i, int L,
                                            float cM, float s2half, float &alpha, float &ud) {
  typename Mma<T>::frag of[2];
  float rs;
  load_row_stats<T, RN>(of, rs, Oh, rsave_h, i, L);
  row_weights_loaded<T, KN, RN>(qf, df, of, rs, i, L, cM, s2half, alpha, ud);
}

// ------------------------------------------------------------ bidirectional dQ
template <typename T, int M>
struct DqSmem {
  using frag = typename Mma<T>::frag;
  frag WA[M / 16][2][64];    // W'' (projection, lane row m)
  frag WT[4][M / 32][64];    // the input-gradient matrix (see build_wt)
  frag SA[M / 16][2][64];    // Buf1 rows over value columns
  float sz[M];               // Buf1 column d
  float bq[M];               // b''
};

// Items are (head, tile of 8 waves x TBW x 16 rows), walked persistently over
// XCD-local ranges; Buf1 [BH][M][65] fp32.
template <typename T, int M, int KN, bool RN, int TBW, bool ACC>
__global__ __launch_bounds__(kBwdBidirThreads) void k_bwd_dq(
    const T *__restrict__ Q, const T *__restrict__ dout, const T *__restrict__ out,
    const float *__restrict__ rsave, const typename Mma<T>::frag *__restrict__ wfr,
    const float *__restrict__ bqg, const float *__restrict__ W, const float *__restrict__ buf1,
    T *__restrict__ dQ, float2 *__restrict__ aux, int H, int L, float s, int Mr, float cM,
    int Mall, int m0, float wts, int ntiles, int nitems) {
  using frag = typename Mma<T>::frag;
  __shared__ DqSmem<T, M> sm;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int g = (tid & 63) >> 4;
  const int c16 = tid & 15;
  const float s2half = 0.5f * s * s;
  int begin, end;
  xcd_range(blockIdx.x, gridDim.x, nitems, begin, end);
  int cur = -1;
  for (int item = begin; item < end; ++item) {
    const int bh = item / ntiles;
    const int tile = item - bh * ntiles;
    const int h = bh % H;
    if (bh != cur) {
      __syncthreads();
      copy_frags_wg<frag, (M / 16) * 2 * 64>(&sm.WA[0][0][0], wfr + ((size_t)h * (Mall / 16) + m0 / 16) * 2 * 64);
      if (tid < M) sm.bq[tid] = bqg[(size_t)h * Mall + m0 + tid];
      build_wt<T, M>(sm.WT, W + ((size_t)h * Mr + m0) * kD, wts, Mr - m0);
      build_state_rows<T, M>(sm.SA, sm.sz, buf1 + ((size_t)bh * Mall + m0) * 65);
      cur = bh;
      __syncthreads();
    }
    const T *Qh = Q + (size_t)bh * L * kD;
    const T *dOh = dout + (size_t)bh * L * kD;
    const T *Oh = out + (size_t)bh * L * kD;
    const frag none[2] = {};
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      const int i = tile * (kBwdBidirThreads / 4) * TBW + 16 * (w * TBW + tb) + c16;
      frag qf[2], df[2];
      load_rows64<T>(qf, Qh, i, L);
      load_rows64<T>(df, dOh, i, L);
      float alpha, ud;
      row_weights<T, KN, RN>(qf, df, Oh, rsave + (size_t)bh * L, i, L, cM, s2half, alpha, ud);
      f32x4 dacc[4];
      float dot2;
      query_grad<T, M, KN, false>(sm.WA, sm.bq, sm.WT, sm.SA, sm.sz, nullptr, none, qf, df, alpha,
                                  ud, s, dacc, dot2);
      if (i < L) {
        store_qgrad<T, KN, ACC>(dQ + ((size_t)bh * L + i) * kD, dacc, qf, alpha, dot2, s);
        if (g == 0) aux[(size_t)bh * L + i] = make_float2(alpha, alpha * ud);
      }
    }
  }
}

// ------------------------------------------------------------ causal dQ
// The segment-scan kernels run eight waves: wave w works on row block w % 4 of
// the chunk over half hf = w / 4 of the feature steps (the two halves' partial
// sums meet in LDS), and on FB feature blocks of the carried state.
constexpr int kScanThreads = 512;
template <int M>
struct ScanSplit {
  static constexpr int NB = M / 16;                 // feature blocks
  static constexpr int FB = NB >= 8 ? NB / 8 : 1;   // blocks per state wave
  static constexpr int FW = NB / FB;                // waves holding state (4 or 8)
  static constexpr int NS = M / 32;                 // feature steps
};

template <typename T, int M>
struct DqScanSmem {
  using frag = typename Mma<T>::frag;
  frag WA[M / 16][2][64];
  frag WT[4][M / 32][64];
  frag SA[M / 16][2][64];    // S before the chunk, rows over value columns
  float sz[M];
  float bq[M];
  frag KT[M / 16][2][64];    // the chunk's key features (row m, k = keys)
  frag VtF[4][2][64];        // C~ of the chunk: row = value column (permuted), k = keys
  frag DF[2][4];             // its column d (D~ per key), one fragment per lane group
  f32x4 dk[16];              // D~ of the chunk's 64 keys
  f32x4 red[4][4][64];       // the second half's partial dQ per row block
  float redd[4][64];         // and its g~ . q-hat
};

// One workgroup per (head, segment of the forward plan). The state waves keep
// rows of S^T (value columns in permuted order, fp32; lanes = their features)
// in registers, publish S before each 64-token chunk and fold the chunk's
// C~^T K-hat in after; the chunk's queries take S u plus the masked intra-chunk
// terms.
template <typename T, int M, int KN, bool RN, bool ACC>
__global__ __launch_bounds__(kScanThreads) void k_bwd_dq_scan(
    const T *__restrict__ Q, const T *__restrict__ K, const T *__restrict__ V,
    const T *__restrict__ dout, const T *__restrict__ out, const float *__restrict__ rsave,
    const typename Mma<T>::frag *__restrict__ wfr, const float *__restrict__ bqg,
    const float *__restrict__ W, const float *__restrict__ prefix, T *__restrict__ dQ,
    float2 *__restrict__ aux, int H, int L, int seg_len, int nseg, float s, int Mr, float cM,
    int Mall, int m0, float wts) {
  using SP = ScanSplit<M>;
  constexpr int FB = SP::FB;
  using P = Mma<T>;
  using frag = typename P::frag;
  __shared__ DqScanSmem<T, M> sm;
  const int item = xcd_item(blockIdx.x, gridDim.x);
  const int bh = item / nseg;
  const int seg = item - bh * nseg;
  const int h = bh % H;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;
  const int qb = w & 3;          // row block of the chunk
  const int hf = w >> 2;         // half of the feature steps
  const bool sw = w < SP::FW;    // holds a slice of the state
  const float s2half = 0.5f * s * s;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  const int r0 = seg * seg_len;
  const int r1 = min(L, r0 + seg_len);

  copy_frags_wg<frag, (M / 16) * 2 * 64>(&sm.WA[0][0][0], wfr + ((size_t)h * (Mall / 16) + m0 / 16) * 2 * 64);
  if (tid < M) sm.bq[tid] = bqg[(size_t)h * Mall + m0 + tid];
  build_wt<T, M>(sm.WT, W + ((size_t)h * Mr + m0) * kD, wts, Mr - m0);
  // S^T slice: acc[nb][mb] rows = value column perm_col(nb, 4 g + j) (block 4: column
  // d replicated), lane = feature m = 16 (w FB + mb) + lane % 16
  f32x4 acc[5][FB];
  if (sw) {
    const float *S = prefix + (((size_t)bh * nseg + seg) * Mall + m0) * 65;
#pragma unroll
    for (int mb = 0; mb < FB; ++mb) {
      const float *row = S + (size_t)(16 * (w * FB + mb) + c16) * 65;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) acc[nb][mb][j] = row[perm_col(nb, 4 * g + j)];
        acc[4][mb][j] = row[64];
      }
    }
  }
  const frag sel[2] = {select_perm<T>(0), select_perm<T>(1)};
  const T *Qh = Q + (size_t)bh * L * kD;
  const T *Kh = K + (size_t)bh * L * kD;
  const T *Vh = V + (size_t)bh * L * kD;
  const T *dOh = dout + (size_t)bh * L * kD;
  const T *Oh = out + (size_t)bh * L * kD;
  const int s0 = hf * (SP::NS / 2);
  const int s1 = s0 + SP::NS / 2;
  __syncthreads();

  // the keys and values of a chunk (all four blocks in every wave). bf16: loaded
  // one chunk ahead, once the previous chunk's are no longer read, and the row
  // statistics are loaded at the top of the chunk but used after its barrier;
  // fp32 fragments are twice as wide and take the chunk's loads at its top (the
  // registers would not hold both)
  constexpr bool kAhead = sizeof(T) == 2;
  frag ka[4][2], va[4][2];
  auto load_kv = [&](int tc) __attribute__((always_inline)) {
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      const int t = tc + 16 * tb + c16;
      load_rows64<T>(ka[tb], Kh, t, r1);
      load_rows64<T>(va[tb], Vh, t, r1);
    }
  };
  if (kAhead && r0 < r1) load_kv(r0);
  for (int t0 = r0; t0 < r1; t0 += 64) {
    if constexpr (!kAhead) load_kv(t0);
    // this row block's queries, output gradient, output and row scale
    const int i = t0 + 16 * qb + c16;
    frag qf[2], df[2], of[2];
    float rs, alpha, ud;
    load_rows64<T>(qf, Qh, i, r1);
    load_rows64<T>(df, dOh, i, r1);
    load_row_stats<T, RN>(of, rs, Oh, rsave + (size_t)bh * L, i, r1);
    if constexpr (!kAhead)
      row_weights_loaded<T, KN, RN>(qf, df, of, rs, i, r1, cM, s2half, alpha, ud);
    if (sw) chunk_features_t<T, FB, KN>(sm.KT, sm.WA, sm.bq, ka, w * FB);
    if (hf == 0) {   // C~ of key block qb
      const int t = t0 + 16 * qb + c16;
      frag ko[2], vo[2];
      if constexpr (kAhead) {
        // the chunk's rows are held (loaded a chunk ahead); qb is uniform over
        // the wave, so taking block qb is a scalar choice, not a runtime
        // register index
        const int qbu = __builtin_amdgcn_readfirstlane(qb);
        ko[0] = ka[0][0];
        ko[1] = ka[0][1];
        vo[0] = va[0][0];
        vo[1] = va[0][1];
#pragma unroll
        for (int tb = 1; tb < 4; ++tb)
          if (tb == qbu) {
            ko[0] = ka[tb][0];
            ko[1] = ka[tb][1];
            vo[0] = va[tb][0];
            vo[1] = va[tb][1];
          }
      } else {   // fp32: loaded again (a runtime register index would go to scratch)
        load_rows64<T>(ko, Kh, t, r1);
        load_rows64<T>(vo, Vh, t, r1);
      }
      float Do = 1.f;
      if constexpr (KN == kCos) Do = cM * expf(s2half * sq_norm16<T>(ko));
      Do = t < r1 ? Do : 0.f;
      if (g == 0) reinterpret_cast<float *>(sm.dk)[16 * qb + c16] = Do;   // for every wave's P2
      float Dj[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) Dj[j] = __shfl(Do, 4 * g + j);
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const f32x4 c = P::mma(vo[kh], sel[half], zero4);
          T *p = reinterpret_cast<T *>(&sm.VtF[2 * kh + half][qb >> 1][l]) + 4 * (qb & 1);
#pragma unroll
          for (int j = 0; j < 4; ++j) p[j] = from_f32<T>(c[j] * Dj[j]);
        }
      if (c16 == 0) {
        T *p = reinterpret_cast<T *>(&sm.DF[qb >> 1][g]) + 4 * (qb & 1);
#pragma unroll
        for (int j = 0; j < 4; ++j) p[j] = from_f32<T>(Dj[j]);
      }
    }
    if (sw) {   // publish S (before the chunk)
#pragma unroll
      for (int mb = 0; mb < FB; ++mb) {
        const int mbg = w * FB + mb;
        sm.SA[mbg][0][l] = P::pack(acc[0][mb], acc[1][mb]);
        sm.SA[mbg][1][l] = P::pack(acc[2][mb], acc[3][mb]);
        if (g == 0) sm.sz[16 * mbg + c16] = acc[4][mb][0];
      }
    }
    __syncthreads();

    if (sw) {   // fold the chunk into S^T: rows value columns, k = keys, columns m
#pragma unroll
      for (int mb = 0; mb < FB; ++mb)
#pragma unroll
        for (int sidx = 0; sidx < 2; ++sidx) {
          const frag kb = sm.KT[w * FB + mb][sidx][l];
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) acc[nb][mb] = P::mma(sm.VtF[nb][sidx][l], kb, acc[nb][mb]);
          acc[4][mb] = P::mma(sm.DF[sidx][g], kb, acc[4][mb]);
        }
    }

    if constexpr (kAhead)
      row_weights_loaded<T, KN, RN>(qf, df, of, rs, i, r1, cM, s2half, alpha, ud);
    // queries of row block qb, feature steps [s0, s1)
    // P2[j][i] = D~_j (v_j . dout_i + u_d,i) for keys j <= i (B operand, k = keys)
    frag pb2[2];
    {
      f32x4 pt[4];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        f32x4 c = P::mma(va[kb][0], df[0], zero4);
        c = P::mma(va[kb][1], df[1], c);
        const f32x4 D = sm.dk[4 * kb + g];   // keys 16 kb + 4 g + j
#pragma unroll
        for (int j = 0; j < 4; ++j)
          pt[kb][j] = 16 * kb + 4 * g + j <= 16 * qb + c16 ? D[j] * (c[j] + ud) : 0.f;
      }
      pb2[0] = P::pack(pt[0], pt[1]);
      pb2[1] = P::pack(pt[2], pt[3]);
    }
    // the chunk's keys and values are read for the last time above
    if (kAhead && t0 + 64 < r1) load_kv(t0 + 64);
    f32x4 dacc[4];
    float dot2;
    query_grad<T, M, KN, true>(sm.WA, sm.bq, sm.WT, sm.SA, sm.sz, sm.KT, pb2, qf, df, alpha, ud,
                               s, dacc, dot2, s0, s1);
    if (hf == 1) {
#pragma unroll
      for (int k = 0; k < 4; ++k) sm.red[qb][k][l] = dacc[k];
      sm.redd[qb][l] = dot2;
    }
    __syncthreads();
    if (hf == 0) {
#pragma unroll
      for (int k = 0; k < 4; ++k) dacc[k] += sm.red[qb][k][l];
      dot2 += sm.redd[qb][l];
      if (i < r1) {
        store_qgrad<T, KN, ACC>(dQ + ((size_t)bh * L + i) * kD, dacc, qf, alpha, dot2, s);
        if (g == 0) aux[(size_t)bh * L + i] = make_float2(alpha, alpha * ud);
      }
    }
  }
}

// ------------------------------------------------------------ key-side rows
// Gradient of one 16-row block of keys (lane column = key j): h = R C_j (+ INTRA_K:
// Q-hat^T P3 with the chunk's query features QT and P3 packed, k = queries), dK
// from h; dV = R^T k-hat (+ INTRA_V: u~^T (P4 masked) with the chunk's query
// features QA and u~^T in UF). KPART / VPART select what is computed.
template <typename T, int M, int KN, bool KPART, bool VPART, bool INTRA>
__device__ __forceinline__ void key_grad(
    const typename Mma<T>::frag (*WA)[2][64], const float *bq,
    const typename Mma<T>::frag (*WT)[M / 32][64], const typename Mma<T>::frag (*RA)[2][64],
    const float *rz, const typename Mma<T>::frag (*RB)[M / 32][64],
    const typename Mma<T>::frag (*QT)[2][64], const typename Mma<T>::frag (&pb3)[2],
    const typename Mma<T>::frag (*QA)[M / 32][64], const typename Mma<T>::frag (*UF)[2][64],
    const typename Mma<T>::frag (&kf)[2], const typename Mma<T>::frag (&vf)[2], int jpos,
    f32x4 (&kacc)[4], float &doth, f32x4 (&vacc)[4], int s0 = 0, int s1 = M / 32) {
  using P = Mma<T>;
  using frag = typename P::frag;
  constexpr float sgn = KN == kCos ? -1.f : 1.f;
  // two feature steps per unrolled iteration; at M = 64 (two steps in all) a
  // full unroll would spill, so the loop stays rolled
  constexpr int kFeatureUnroll = M > 64 ? 2 : 1;
  const int l = lane_id();
  const int g = l >> 4;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  f32x4 p4[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    kacc[k] = zero4;
    vacc[k] = zero4;
    p4[k] = zero4;
  }
  doth = 0.f;
#pragma unroll kFeatureUnroll
  for (int sidx = s0; sidx < s1; ++sidx) {
    f32x4 kh[2], G[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int mb = 2 * sidx + hh;
      const f32x4 bcv = *reinterpret_cast<const f32x4 *>(&bq[16 * mb + 4 * g]);
      f32x4 p = P::mma(WA[mb][0][l], kf[0], bcv);
      p = P::mma(WA[mb][1][l], kf[1], p);
#pragma unroll
      for (int j = 0; j < 4; ++j) kh[hh][j] = feature<KN, P>(p[j], bcv[j]);
      if constexpr (KPART) {
        f32x4 hv = P::mma(RA[mb][0][l], vf[0], zero4);
        hv = P::mma(RA[mb][1][l], vf[1], hv);
        if constexpr (INTRA) {
          hv = P::mma(QT[mb][0][l], pb3[0], hv);
          hv = P::mma(QT[mb][1][l], pb3[1], hv);
        }
        const f32x4 rzv = *reinterpret_cast<const f32x4 *>(&rz[16 * mb + 4 * g]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float hj = hv[j] + rzv[j];
          doth = fmaf(hj, kh[hh][j], doth);
          G[hh][j] = sgn * hj * feature_slope<KN, P>(p[j], bcv[j]);
        }
      }
    }
    if constexpr (KPART) {
      const frag gb = P::pack(G[0], G[1]);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) kacc[kb] = P::mma(WT[kb][sidx][l], gb, kacc[kb]);
    }
    if constexpr (VPART) {
      const frag kb_ = P::pack(kh[0], kh[1]);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) vacc[nb] = P::mma(RB[nb][sidx][l], kb_, vacc[nb]);
      if constexpr (INTRA) {
#pragma unroll
        for (int qb = 0; qb < 4; ++qb) p4[qb] = P::mma(QA[qb][sidx][l], kb_, p4[qb]);
      }
    }
  }
  if constexpr (KPART) {
    doth += __shfl_xor(doth, 16);
    doth += __shfl_xor(doth, 32);
  }
  if constexpr (VPART && INTRA) {
    // keep queries i >= j, then u~^T (q-hat . k-hat)
#pragma unroll
    for (int qb = 0; qb < 4; ++qb)
#pragma unroll
      for (int j = 0; j < 4; ++j) p4[qb][j] = 16 * qb + 4 * g + j >= jpos ? p4[qb][j] : 0.f;
#pragma unroll
    for (int sidx = 0; sidx < 2; ++sidx) {
      const frag pb = P::pack(p4[2 * sidx], p4[2 * sidx + 1]);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) vacc[nb] = P::mma(UF[nb][sidx][l], pb, vacc[nb]);
    }
  }
}

// dK = D~ (WT G + s^2 (h . k-hat) k) (cos features), D~ (WT G) (ReLU); dV = D~ vacc.
template <typename T, int KN, bool ACC = false>
__device__ __forceinline__ void store_kgrad(T *dst, const f32x4 (&kacc)[4],
                                            const typename Mma<T>::frag (&kf)[2], float D,
                                            float doth, float s) {
  const int g = lane_id() >> 4;
  const float cx = KN == kCos ? s * s * doth : 0.f;
#pragma unroll
  for (int pp = 0; pp < 2; ++pp) {
    f32x4 lo, hi;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo[e] = D * fmaf(cx, to_f32(kf[pp][e]), kacc[2 * pp][e]);
      hi[e] = D * fmaf(cx, to_f32(kf[pp][4 + e]), kacc[2 * pp + 1][e]);
    }
    put8<ACC>(dst + 32 * pp + 8 * g, lo, hi);
  }
}
template <typename T, bool ACC = false>
__device__ __forceinline__ void store_vgrad(T *dst, const f32x4 (&vacc)[4], float D) {
  const int g = lane_id() >> 4;
#pragma unroll
  for (int pp = 0; pp < 2; ++pp)
    put8<ACC>(dst + 32 * pp + 8 * g, vacc[2 * pp] * D, vacc[2 * pp + 1] * D);
}

// ------------------------------------------------------------ bidirectional dK, dV
template <typename T, int M>
struct DkvSmem {
  using frag = typename Mma<T>::frag;
  frag WA[M / 16][2][64];
  float bq[M];
  frag WT[4][M / 32][64];
  frag RA[M / 16][2][64];   // dBuf1 rows over value columns
  float rz[M];              // dBuf1 column d
  frag RB[4][M / 32][64];   // dBuf1 value columns over features
};

template <typename T, int M, int KN, int TBW, bool ACC>
__global__ __launch_bounds__(kBwdBidirThreads) void k_bwd_dkv(
    const T *__restrict__ K, const T *__restrict__ V,
    const typename Mma<T>::frag *__restrict__ wfr, const float *__restrict__ bqg,
    const float *__restrict__ W, const float *__restrict__ dbuf1, T *__restrict__ dK,
    T *__restrict__ dV, int H, int L, float s, int Mr, float cM, int Mall, int m0, float wts,
    int ntiles, int nitems) {
  using frag = typename Mma<T>::frag;
  __shared__ DkvSmem<T, M> sm;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int c16 = tid & 15;
  const float s2half = 0.5f * s * s;
  int begin, end;
  xcd_range(blockIdx.x, gridDim.x, nitems, begin, end);
  int cur = -1;
  for (int item = begin; item < end; ++item) {
    const int bh = item / ntiles;
    const int tile = item - bh * ntiles;
    const int h = bh % H;
    if (bh != cur) {
      __syncthreads();
      copy_frags_wg<frag, (M / 16) * 2 * 64>(&sm.WA[0][0][0], wfr + ((size_t)h * (Mall / 16) + m0 / 16) * 2 * 64);
      if (tid < M) sm.bq[tid] = bqg[(size_t)h * Mall + m0 + tid];
      build_wt<T, M>(sm.WT, W + ((size_t)h * Mr + m0) * kD, wts, Mr - m0);
      const float *Rs = dbuf1 + ((size_t)bh * Mall + m0) * 65;
      build_state_rows<T, M>(sm.RA, sm.rz, Rs);
      build_state_cols<T, M>(sm.RB, Rs);
      cur = bh;
      __syncthreads();
    }
    const T *Kh = K + (size_t)bh * L * kD;
    const T *Vh = V + (size_t)bh * L * kD;
    const frag none[2] = {};
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      const int j = tile * (kBwdBidirThreads / 4) * TBW + 16 * (w * TBW + tb) + c16;
      frag kf[2], vf[2];
      load_rows64<T>(kf, Kh, j, L);
      load_rows64<T>(vf, Vh, j, L);
      float D = 1.f;
      if constexpr (KN == kCos) D = cM * expf(s2half * sq_norm16<T>(kf));
      f32x4 kacc[4], vacc[4];
      float doth;
      key_grad<T, M, KN, true, true, false>(sm.WA, sm.bq, sm.WT, sm.RA, sm.rz, sm.RB, nullptr,
                                            none, nullptr, nullptr, kf, vf, 0, kacc, doth,
                                            vacc);
      if (j < L) {
        store_kgrad<T, KN, ACC>(dK + ((size_t)bh * L + j) * kD, kacc, kf, D, doth, s);
        store_vgrad<T, ACC>(dV + ((size_t)bh * L + j) * kD, vacc, D);
      }
    }
  }
}

// ------------------------------------------------------------ causal dK / dV
template <typename T, int M, bool KPART>
struct DkvScanSmem {
  using frag = typename Mma<T>::frag;
  frag WA[M / 16][2][64];
  float bq[M];
  frag QT[M / 16][2][64];      // the chunk's query features (row m, k = queries)
  frag UF[4][2][64];           // u~^T: row = value column (permuted), k = queries
  frag UD[KPART ? 2 : 1][4];   // u~ column d, one fragment per lane group
  // dK: R rows over value columns, its column d, the input-gradient matrix
  frag WT[KPART ? 4 : 1][KPART ? M / 32 : 1][64];
  frag RA[KPART ? M / 16 : 1][2][64];
  float rz[KPART ? M : 1];
  // dV: R value columns over features, query features with lane row = query
  frag RB[KPART ? 1 : 4][KPART ? 1 : M / 32][64];
  frag QA[KPART ? 1 : 4][KPART ? 1 : M / 32][64];
  f32x4 red[4][4][64];         // the second half's partial sums per row block
  float redd[4][64];           // and its h . k-hat
};

// One workgroup per (head, segment), chunks from the last to the first. The
// state waves keep their slice of R, the aggregate of q-hat (x) u~ over the rows
// after the chunk plus dstate_out: as R^T (rows = value columns permuted, lanes =
// m) for dK, as R (rows m, lanes = value columns) for dV. Each chunk publishes
// R, then folds its own rows in; its keys take R plus the masked intra-chunk
// terms.
template <typename T, int M, int KN, bool KPART, bool ACC>
__global__ __launch_bounds__(kScanThreads) void k_bwd_dkv_scan(
    const T *__restrict__ Q, const T *__restrict__ K, const T *__restrict__ V,
    const T *__restrict__ dout, const float2 *__restrict__ aux,
    const typename Mma<T>::frag *__restrict__ wfr, const float *__restrict__ bqg,
    const float *__restrict__ W, const float *__restrict__ suffix, T *__restrict__ dK,
    T *__restrict__ dV, int H, int L, int seg_len, int nseg, float s, int Mr, float cM, int Mall, int m0,
    float wts) {
  using SP = ScanSplit<M>;
  constexpr int FB = SP::FB;
  using P = Mma<T>;
  using frag = typename P::frag;
  __shared__ DkvScanSmem<T, M, KPART> sm;
  const int item = xcd_item(blockIdx.x, gridDim.x);
  const int bh = item / nseg;
  const int seg = item - bh * nseg;
  const int h = bh % H;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;
  const int qb = w & 3;
  const int hf = w >> 2;
  const bool sw = w < SP::FW;
  const float s2half = 0.5f * s * s;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  const int r0 = seg * seg_len;
  const int r1 = min(L, r0 + seg_len);
  const int s0 = hf * (SP::NS / 2);
  const int s1 = s0 + SP::NS / 2;

  copy_frags_wg<frag, (M / 16) * 2 * 64>(&sm.WA[0][0][0], wfr + ((size_t)h * (Mall / 16) + m0 / 16) * 2 * 64);
  if (tid < M) sm.bq[tid] = bqg[(size_t)h * Mall + m0 + tid];
  if constexpr (KPART) build_wt<T, M>(sm.WT, W + ((size_t)h * Mr + m0) * kD, wts, Mr - m0);
  // dK: acc[nb][mb] rows value column perm_col(nb, 4 g + j) (block 4: column d),
  // lane m = 16 (w FB + mb) + lane % 16. dV: acc[mb][nb] rows m = 16 (w FB + mb)
  // + 4 g + j, lane value column perm_col(nb, lane % 16).
  f32x4 acc[KPART ? 5 : FB][KPART ? FB : 4];
  if (sw) {
    const float *R = suffix + (((size_t)bh * nseg + seg) * Mall + m0) * 65;
#pragma unroll
    for (int mb = 0; mb < FB; ++mb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if constexpr (KPART) {
          const float *row = R + (size_t)(16 * (w * FB + mb) + c16) * 65;
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) acc[nb][mb][j] = row[perm_col(nb, 4 * g + j)];
          acc[4][mb][j] = row[64];
        } else {
          const float *row = R + (size_t)(16 * (w * FB + mb) + 4 * g + j) * 65;
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) acc[mb][nb][j] = row[perm_col(nb, c16)];
        }
      }
  }
  const frag sel[2] = {select_perm<T>(0), select_perm<T>(1)};
  const T *Qh = Q + (size_t)bh * L * kD;
  const T *Kh = K + (size_t)bh * L * kD;
  const T *Vh = V + (size_t)bh * L * kD;
  const T *dOh = dout + (size_t)bh * L * kD;
  const float2 *auh = aux + (size_t)bh * L;
  __syncthreads();

  // The dV pass with bf16 operands has registers to spare: the rows the next
  // chunk in scan order reads (its keys, queries, output gradients and row
  // weights) are loaded once this chunk has consumed its own, right after its
  // first barrier, so that their latency hides behind this chunk's products;
  // the key rows, read until the end of the chunk, go to a second buffer.
  constexpr bool kAhead = !KPART && sizeof(T) == 2;
  frag kf[2], vf[2], kfn[2], qa[4][2], dob[2], qo[2];
  float2 ao = make_float2(0.f, 0.f);
  auto load_ahead = [&](int tc, frag (&kdst)[2]) __attribute__((always_inline)) {
    const int t = tc + 16 * qb + c16;
    load_rows64<T>(kdst, Kh, t, r1);
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) load_rows64<T>(qa[tb], Qh, tc + 16 * tb + c16, r1);
    if (hf == 0) {
      load_rows64<T>(dob, dOh, t, r1);
      ao = t < r1 ? auh[t] : make_float2(0.f, 0.f);
    }
    load_rows64<T>(qo, Qh, t, r1);
  };
  const int nch = (r1 - r0 + 63) / 64;
  if (kAhead && nch > 0) load_ahead(r0 + 64 * (nch - 1), kf);
  for (int c = nch - 1; c >= 0; --c) {
    const int t0 = r0 + 64 * c;
    // this row block's keys and values, loaded with the chunk's other rows
    const int j = t0 + 16 * qb + c16;
    if constexpr (!kAhead) {
      load_rows64<T>(kf, Kh, j, r1);
      load_rows64<T>(vf, Vh, j, r1);
      // the chunk's queries: features (row m) of the state waves' blocks, u~^T
      // of row block qb; (alpha, alpha u_d) of every row
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) load_rows64<T>(qa[tb], Qh, t0 + 16 * tb + c16, r1);
    }
    if (sw) chunk_features_t<T, FB, KN>(sm.QT, sm.WA, sm.bq, qa, w * FB);
    frag da[4][2];
    float2 au[4];
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
      const int t = t0 + 16 * tb + c16;
      load_rows64<T>(da[tb], dOh, t, r1);
      au[tb] = t < r1 ? auh[t] : make_float2(0.f, 0.f);
    }
    if (hf == 0) {   // row block qb of the output gradients and row weights
      if constexpr (KPART) {
        // held in da, au; qb is uniform over the wave, so taking block qb is a
        // scalar choice, not a runtime register index
        const int qbu = __builtin_amdgcn_readfirstlane(qb);
        dob[0] = da[0][0];
        dob[1] = da[0][1];
        ao = au[0];
#pragma unroll
        for (int tb = 1; tb < 4; ++tb)
          if (tb == qbu) {
            dob[0] = da[tb][0];
            dob[1] = da[tb][1];
            ao = au[tb];
          }
      } else if constexpr (!kAhead) {   // fp32 dV pass: loaded again
        const int t = t0 + 16 * qb + c16;
        load_rows64<T>(dob, dOh, t, r1);
        ao = t < r1 ? auh[t] : make_float2(0.f, 0.f);
      }
      float aj[4], ej[4];   // of queries 16 qb + 4 g + j
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        aj[j] = __shfl(ao.x, 4 * g + j);
        ej[j] = __shfl(ao.y, 4 * g + j);
      }
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const f32x4 cc = P::mma(dob[kh], sel[half], zero4);
          T *p = reinterpret_cast<T *>(&sm.UF[2 * kh + half][qb >> 1][l]) + 4 * (qb & 1);
#pragma unroll
          for (int j = 0; j < 4; ++j) p[j] = from_f32<T>(cc[j] * aj[j]);
        }
      if constexpr (KPART) {
        if (c16 == 0) {
          T *p = reinterpret_cast<T *>(&sm.UD[qb >> 1][g]) + 4 * (qb & 1);
#pragma unroll
          for (int j = 0; j < 4; ++j) p[j] = from_f32<T>(ej[j]);
        }
      }
    }
    if constexpr (!KPART) {
      // row block qb's features with lane row = query (k = m), steps [s0, s1)
      if constexpr (!kAhead) load_rows64<T>(qo, Qh, t0 + 16 * qb + c16, r1);
#pragma unroll 2
      for (int sidx = s0; sidx < s1; ++sidx) {
        f32x4 f[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int mb = 2 * sidx + hh;
          const f32x4 bcv = *reinterpret_cast<const f32x4 *>(&sm.bq[16 * mb + 4 * g]);
          f32x4 p = P::mma(sm.WA[mb][0][l], qo[0], bcv);
          p = P::mma(sm.WA[mb][1][l], qo[1], p);
#pragma unroll
          for (int j = 0; j < 4; ++j) f[hh][j] = feature<KN, P>(p[j], bcv[j]);
        }
        sm.QA[qb][sidx][l] = P::pack(f[0], f[1]);
      }
    }
    if (sw) {   // publish R (after the chunk)
#pragma unroll
      for (int mb = 0; mb < FB; ++mb) {
        const int mbg = w * FB + mb;
        if constexpr (KPART) {
          sm.RA[mbg][0][l] = P::pack(acc[0][mb], acc[1][mb]);
          sm.RA[mbg][1][l] = P::pack(acc[2][mb], acc[3][mb]);
          if (g == 0) sm.rz[16 * mbg + c16] = acc[4][mb][0];
        } else {
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) {
            T *p = reinterpret_cast<T *>(&sm.RB[nb][mbg >> 1][l]) + 4 * (mbg & 1);
#pragma unroll
            for (int j = 0; j < 4; ++j) p[j] = from_f32<T>(acc[mb][nb][j]);
          }
        }
      }
    }
    __syncthreads();
    if constexpr (kAhead) {
      if (c > 0) load_ahead(t0 - 64, kfn);
    }

    if (sw) {   // fold the chunk's rows into R
#pragma unroll
      for (int mb = 0; mb < FB; ++mb)
#pragma unroll
        for (int sidx = 0; sidx < 2; ++sidx) {
          const frag qt = sm.QT[w * FB + mb][sidx][l];
          if constexpr (KPART) {
#pragma unroll
            for (int nb = 0; nb < 4; ++nb)
              acc[nb][mb] = P::mma(sm.UF[nb][sidx][l], qt, acc[nb][mb]);
            acc[4][mb] = P::mma(sm.UD[sidx][g], qt, acc[4][mb]);
          } else {
#pragma unroll
            for (int nb = 0; nb < 4; ++nb)
              acc[mb][nb] = P::mma(qt, sm.UF[nb][sidx][l], acc[mb][nb]);
          }
        }
    }

    // keys of row block qb, feature steps [s0, s1)
    // P3[i][j] = alpha_i (dout_i . v_j + u_d,i) for queries i >= j (B operand, k = queries)
    frag pb3[2];
    if constexpr (KPART) {
      f32x4 pt[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        f32x4 cc = P::mma(da[q][0], vf[0], zero4);
        cc = P::mma(da[q][1], vf[1], cc);
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const float a = __shfl(au[q].x, 4 * g + jj);
          const float e = __shfl(au[q].y, 4 * g + jj);
          pt[q][jj] = 16 * q + 4 * g + jj >= 16 * qb + c16 ? fmaf(a, cc[jj], e) : 0.f;
        }
      }
      pb3[0] = P::pack(pt[0], pt[1]);
      pb3[1] = P::pack(pt[2], pt[3]);
    }
    f32x4 kacc[4], vacc[4];
    float doth;
    // the tables of the other part are one-element placeholders, never read
    using T2 = const frag(*)[2][64];
    using TS = const frag(*)[M / 32][64];
    key_grad<T, M, KN, KPART, !KPART, true>(
        sm.WA, sm.bq, reinterpret_cast<TS>(&sm.WT[0][0][0]), reinterpret_cast<T2>(&sm.RA[0][0][0]),
        sm.rz, reinterpret_cast<TS>(&sm.RB[0][0][0]), sm.QT, pb3,
        reinterpret_cast<TS>(&sm.QA[0][0][0]), sm.UF, kf, vf, 16 * qb + c16, kacc, doth,
        vacc, s0, s1);
    f32x4 (&part)[4] = KPART ? kacc : vacc;
    if (hf == 1) {
#pragma unroll
      for (int k = 0; k < 4; ++k) sm.red[qb][k][l] = part[k];
      sm.redd[qb][l] = doth;
    }
    __syncthreads();
    if (hf == 0) {
#pragma unroll
      for (int k = 0; k < 4; ++k) part[k] += sm.red[qb][k][l];
      doth += sm.redd[qb][l];
      float D = 1.f;
      if constexpr (KN == kCos) D = cM * expf(s2half * sq_norm16<T>(kf));
      if (j < r1) {
        if constexpr (KPART)
          store_kgrad<T, KN, ACC>(dK + ((size_t)bh * L + j) * kD, kacc, kf, D, doth, s);
        else
          store_vgrad<T, ACC>(dV + ((size_t)bh * L + j) * kD, vacc, D);
      }
    }
    if constexpr (kAhead) {
      kf[0] = kfn[0];
      kf[1] = kfn[1];
    }
  }
}

// ------------------------------------------------------------ launchers
// M dispatch up to MAX_ (fp32 operands double the LDS tables: the fp32
// kernels stop at M = 128 bidirectional and M = 64 causal).
#define FAVOR_BWD_DISPATCH_M(MAX_, M_, ...)                                \
  switch (M_) {                                                            \
    case 64: { constexpr int MM = 64; __VA_ARGS__; } break;                 \
    case 128:                                                              \
      if constexpr (MAX_ >= 128) {                                          \
        constexpr int MM = 128;                                            \
        __VA_ARGS__;                                                       \
        break;                                                             \
      } else {                                                             \
        return hipErrorInvalidValue;                                       \
      }                                                                    \
    case 256:                                                              \
      if constexpr (MAX_ >= 256) {                                          \
        constexpr int MM = 256;                                            \
        __VA_ARGS__;                                                       \
        break;                                                             \
      } else {                                                             \
        return hipErrorInvalidValue;                                       \
      }                                                                    \
    default: return hipErrorInvalidValue;                                  \
  }

template <typename T> constexpr int bwd_max_m(bool causal) {
  return sizeof(T) == 2 ? 256 : (causal ? 64 : 128);
}

// Scale of W in the input-gradient products: s for cos features (2 pi W'' = s W),
// s / sqrt(M) for ReLU features (W'' itself).
static float wt_scale(const Shape &sh) {
  return sh.kernel == 1 ? sh.s / sqrtf((float)sh.Mr) : sh.s;
}

// Rows per persistent bidirectional tile: 8 waves x kBwdTbw blocks of 16 (one
// block per call of the row functions).
constexpr int kBwdTbw = 2;
constexpr int kBwdMaxWorkgroups = 256;

hipError_t launch_sum_splits(const Shape &sh, const float *part, int ns, float *dst,
                             hipStream_t st) {
  const int n4 = sh.M * 65 / 4;
  dim3 grid((n4 + 255) / 256, sh.BH);
  hipLaunchKernelGGL(k_sum_splits, grid, dim3(256), 0, st, (const f32x4 *)part, ns, n4,
                     (f32x4 *)dst);
  return hipGetLastError();
}

hipError_t launch_suffix_scan(const Shape &sh, float *part, int nch, const float *dsout,
                              float *dsin, hipStream_t st, const float *bias) {
  const int n4 = sh.M * 65 / 4;
  dim3 grid((n4 + 255) / 256, sh.BH);
  hipLaunchKernelGGL(k_suffix_scan, grid, dim3(256), 0, st, (f32x4 *)part, nch, n4,
                     sh.Mr * 65 / 4, (const f32x4 *)dsout, (f32x4 *)dsin, (const f32x4 *)bias);
  return hipGetLastError();
}

// Calls f(integral_constant KN, bool_constant RN) for the shape's feature kernel
// and renormalisation.
template <typename F>
static hipError_t bwd_variant(const Shape &sh, F &&f) {
  using relu = std::integral_constant<int, kRelu>;
  using cosk = std::integral_constant<int, kCos>;
  if (sh.kernel == 1) return sh.renorm ? f(relu{}, std::true_type{}) : f(relu{}, std::false_type{});
  return sh.renorm ? f(cosk{}, std::true_type{}) : f(cosk{}, std::false_type{});
}

// Feature slices of the gradient launches. A gradient is a sum over features
// once the per-row weights (out, r, alpha) are fixed, so a shape wider than the
// kernels' LDS tables (fp32 operands: bwd_max_m features) runs as slices
// [m0, m0 + ms) of the M rows, the slices after the first adding into the fp32
// gradients; slices wholly past the M_r features drawn add nothing and are
// skipped. f(ms, m0, first) launches one slice.
template <typename T, typename F>
static hipError_t over_slices(const Shape &sh, bool causal, F &&f) {
  const int ms = sh.M < bwd_max_m<T>(causal) ? sh.M : bwd_max_m<T>(causal);
  for (int m0 = 0; m0 < sh.M && m0 < sh.Mr; m0 += ms) {
    const hipError_t e = f(ms, m0, m0 == 0);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Calls f(bool_constant ACC): false for the first slice, true after it (fp32 only).
template <typename T, typename F>
static hipError_t with_acc(bool first, F &&f) {
  if constexpr (sizeof(T) == 4) {
    if (!first) return f(std::true_type{});
  }
  return f(std::false_type{});
}

// accumulate (causal only): every slice adds onto what dQ holds (the other
// direction's gradient, when both are differentiated in one call).
template <typename T>
static hipError_t bwd_dq_typed(const Shape &sh, bool causal, const BwdArgs &a, hipStream_t st,
                               bool accumulate) {
  const float wts = wt_scale(sh);
  return bwd_variant(sh, [&](auto kn, auto rn) -> hipError_t {
    constexpr int KN = decltype(kn)::value;
    constexpr bool RN = decltype(rn)::value;
    return over_slices<T>(sh, causal, [&](int ms, int m0, bool first) -> hipError_t {
      if (causal && accumulate) {
        dim3 grid(a.nseg * sh.BH);
        FAVOR_BWD_DISPATCH_M(bwd_max_m<T>(true), ms,
            hipLaunchKernelGGL((k_bwd_dq_scan<T, MM, KN, RN, true>), grid, dim3(kScanThreads),
                               0, st, (const T *)a.Q, (const T *)a.K, (const T *)a.V,
                               (const T *)a.dout, (const T *)a.out, a.rsave,
                               (const typename Mma<T>::frag *)a.wfr, a.bq, a.W, a.state,
                               (T *)a.dQ, a.aux, sh.H, sh.L, a.seg_len, a.nseg, sh.s, sh.Mr,
                               feature_norm(sh), sh.M, m0, wts));
        return hipGetLastError();
      }
      return with_acc<T>(first, [&](auto acc) -> hipError_t {
        constexpr bool ACC = decltype(acc)::value;
        if (causal) {
          dim3 grid(a.nseg * sh.BH);
          FAVOR_BWD_DISPATCH_M(bwd_max_m<T>(true), ms,
              hipLaunchKernelGGL((k_bwd_dq_scan<T, MM, KN, RN, ACC>), grid, dim3(kScanThreads),
                                 0, st, (const T *)a.Q, (const T *)a.K, (const T *)a.V,
                                 (const T *)a.dout, (const T *)a.out, a.rsave,
                                 (const typename Mma<T>::frag *)a.wfr, a.bq, a.W, a.state,
                                 (T *)a.dQ, a.aux, sh.H, sh.L, a.seg_len, a.nseg, sh.s, sh.Mr,
                                 feature_norm(sh), sh.M, m0, wts));
        } else {
          const int rows = kBwdBidirThreads / 4 * kBwdTbw;
          const int ntiles = (sh.L + rows - 1) / rows;
          const int nitems = ntiles * sh.BH;
          dim3 grid(min(nitems, kBwdMaxWorkgroups));
          FAVOR_BWD_DISPATCH_M(bwd_max_m<T>(false), ms,
              hipLaunchKernelGGL((k_bwd_dq<T, MM, KN, RN, kBwdTbw, ACC>), grid,
                                 dim3(kBwdBidirThreads), 0, st, (const T *)a.Q,
                                 (const T *)a.dout, (const T *)a.out, a.rsave,
                                 (const typename Mma<T>::frag *)a.wfr, a.bq, a.W, a.state,
                                 (T *)a.dQ, a.aux, sh.H, sh.L, sh.s, sh.Mr, feature_norm(sh),
                                 sh.M, m0, wts, ntiles, nitems));
        }
        return hipGetLastError();
      });
    });
  });
}

hipError_t launch_bwd_dq(const Shape &sh, Dt in, bool causal, const BwdArgs &a, hipStream_t st,
                         bool accumulate) {
  if (in == Dt::BF16) return bwd_dq_typed<bf16>(sh, causal, a, st, accumulate);
  return bwd_dq_typed<float>(sh, causal, a, st, accumulate);
}

template <typename T>
static hipError_t bwd_dkv_typed(const Shape &sh, bool causal, const BwdArgs &a, hipStream_t st) {
  const float wts = wt_scale(sh);
  return bwd_variant(sh, [&](auto kn, auto) -> hipError_t {
    constexpr int KN = decltype(kn)::value;
    return over_slices<T>(sh, causal, [&](int ms, int m0, bool first) -> hipError_t {
      return with_acc<T>(first, [&](auto acc) -> hipError_t {
        constexpr bool ACC = decltype(acc)::value;
        if (causal) {
          dim3 grid(a.nseg * sh.BH);
          FAVOR_BWD_DISPATCH_M(bwd_max_m<T>(true), ms, {
            hipLaunchKernelGGL((k_bwd_dkv_scan<T, MM, KN, false, ACC>), grid,
                               dim3(kScanThreads), 0, st, (const T *)a.Q, (const T *)a.K,
                               (const T *)a.V, (const T *)a.dout, a.aux,
                               (const typename Mma<T>::frag *)a.wfr, a.bq, a.W, a.state,
                               (T *)a.dK, (T *)a.dV, sh.H, sh.L, a.seg_len, a.nseg, sh.s, sh.Mr,
                               feature_norm(sh), sh.M, m0, wts);
            hipLaunchKernelGGL((k_bwd_dkv_scan<T, MM, KN, true, ACC>), grid,
                               dim3(kScanThreads), 0, st, (const T *)a.Q, (const T *)a.K,
                               (const T *)a.V, (const T *)a.dout, a.aux,
                               (const typename Mma<T>::frag *)a.wfr, a.bq, a.W, a.state,
                               (T *)a.dK, (T *)a.dV, sh.H, sh.L, a.seg_len, a.nseg, sh.s, sh.Mr,
                               feature_norm(sh), sh.M, m0, wts);
          });
        } else {
          const int rows = kBwdBidirThreads / 4 * kBwdTbw;
          const int ntiles = (sh.L + rows - 1) / rows;
          const int nitems = ntiles * sh.BH;
          dim3 grid(min(nitems, kBwdMaxWorkgroups));
          FAVOR_BWD_DISPATCH_M(bwd_max_m<T>(false), ms,
              hipLaunchKernelGGL((k_bwd_dkv<T, MM, KN, kBwdTbw, ACC>), grid,
                                 dim3(kBwdBidirThreads), 0, st, (const T *)a.K, (const T *)a.V,
                                 (const typename Mma<T>::frag *)a.wfr, a.bq, a.W, a.state,
                                 (T *)a.dK, (T *)a.dV, sh.H, sh.L, sh.s, sh.Mr,
                                 feature_norm(sh), sh.M, m0, wts, ntiles, nitems));
        }
        return hipGetLastError();
      });
    });
  });
}

hipError_t launch_bwd_dkv(const Shape &sh, Dt in, bool causal, const BwdArgs &a, hipStream_t st) {
  if (in == Dt::BF16) return bwd_dkv_typed<bf16>(sh, causal, a, st);
  return bwd_dkv_typed<float>(sh, causal, a, st);
}

}  // namespace favor
