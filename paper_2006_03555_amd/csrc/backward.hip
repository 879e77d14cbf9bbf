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

constexpr int kBwdThreads = 256;

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
// (dsout + every chunk) goes to dsin. Either pointer may be null.
__global__ __launch_bounds__(256) void k_suffix_scan(f32x4 *__restrict__ part, int nch, int n4,
                                                     const f32x4 *__restrict__ dsout,
                                                     f32x4 *__restrict__ dsin) {
  const int bh = blockIdx.y;
  const int u = blockIdx.x * 256 + threadIdx.x;
  if (u >= n4) return;
  f32x4 *p = part + (size_t)bh * nch * n4 + u;
  f32x4 run = dsout ? dsout[(size_t)bh * n4 + u] : f32x4{0.f, 0.f, 0.f, 0.f};
  int c = nch - 1;
  for (; c >= 7; c -= 8) {   // eight loads in flight
    f32x4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = p[(size_t)(c - k) * n4];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      p[(size_t)(c - k) * n4] = run;
      run += v[k];
    }
  }
  for (; c >= 0; --c) {
    const f32x4 v = p[(size_t)c * n4];
    p[(size_t)c * n4] = run;
    run += v;
  }
  if (dsin) dsin[(size_t)bh * n4 + u] = run;
}

// ------------------------------------------------------------ LDS builders
// W''^T for the input-gradient products as A operand: row = input column
// perm_col(kb, lane % 16) (store order), k = feature m = 32 s + chained(g, i).
template <typename T, int M>
__device__ __forceinline__ void build_wt(typename Mma<T>::frag (*WT)[M / 32][64],
                                         const float *__restrict__ Wh, float scale) {
  constexpr int NS = M / 32;
  for (int idx = threadIdx.x; idx < 4 * NS * 64; idx += kBwdThreads) {
    const int l = idx & 63;
    const int s = (idx >> 6) % NS;
    const int kb = idx / (64 * NS);
    const int g = l >> 4;
    const int k = perm_col(kb, l & 15);
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = Wh[(32 * s + 16 * (i >> 2) + 4 * g + (i & 3)) * kD + k];
    WT[kb][s][l] = Mma<T>::from_f32(v, scale);
  }
}

// An aggregate S [M][65] (fp32, row-major) as A operand over its value
// columns: row = m = 16 mb + lane % 16, k = column 32 ks + 8 g + i (loaded
// order); its last column separately (sz).
template <typename T, int M>
__device__ __forceinline__ void build_state_rows(typename Mma<T>::frag (*SA)[2][64], float *sz,
                                                 const float *__restrict__ S) {
  for (int idx = threadIdx.x; idx < (M / 16) * 2 * 64; idx += kBwdThreads) {
    const int l = idx & 63;
    const int ks = (idx >> 6) & 1;
    const int mb = idx >> 7;
    const float *row = S + (size_t)(16 * mb + (l & 15)) * 65 + 32 * ks + 8 * (l >> 4);
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = row[i];
    SA[mb][ks][l] = Mma<T>::from_f32(v, 1.f);
  }
  for (int m = threadIdx.x; m < M; m += kBwdThreads) sz[m] = S[(size_t)m * 65 + 64];
}

// The value columns of S as A operand over features: row = column
// perm_col(nb, lane % 16), k = m = 32 s + chained(g, i).
template <typename T, int M>
__device__ __forceinline__ void build_state_cols(typename Mma<T>::frag (*SB)[M / 32][64],
                                                 const float *__restrict__ S) {
  constexpr int NS = M / 32;
  for (int idx = threadIdx.x; idx < 4 * NS * 64; idx += kBwdThreads) {
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

template <typename T>
__device__ __forceinline__ float sq_norm16(const typename Mma<T>::frag (&f)[2]) {
  float n = 0.f;
#pragma unroll
  for (int k = 0; k < 2; ++k)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float x = to_f32(f[k][i]);
      n = fmaf(x, x, n);
    }
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
                                                 const typename Mma<T>::frag (&rf)[4][2], int mb0,
                                                 float keps) {
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
      for (int j = 0; j < 4; ++j) f[tb][j] = feature<KN, P>(p[j], keps);
    }
    dst[mbg][0][l] = P::pack(f[0], f[1]);
    dst[mbg][1][l] = P::pack(f[2], f[3]);
  }
}

// ------------------------------------------------------------ dQ
template <typename T, int M, bool CAUSAL>
struct DqSmem {
  using frag = typename Mma<T>::frag;
  frag WA[M / 16][2][64];    // W'' (projection, lane row m)
  frag WT[4][M / 32][64];    // the input-gradient matrix (see build_wt)
  frag SA[M / 16][2][64];    // S rows over value columns
  float sz[M];               // S column d
  float bq[M];               // b''
  frag KT[CAUSAL ? M / 16 : 1][2][64];   // the chunk's key features (row m, k = keys)
  frag VA[CAUSAL ? 4 : 1][2][64];        // the chunk's value rows (lane row = key)
  float dk[CAUSAL ? 64 : 1];             // D~ of the chunk's keys (0 past L)
};

// Bidirectional: items are (head, tile of 64 TBW rows), walked persistently over
// XCD-local ranges; the state is Buf1 [BH][M][65]. Causal: one item per
// workgroup, a 64-token chunk (TBW = 1) with its prefix state [BH][nch][M][65].
template <typename T, int M, int KN, bool RN, bool CAUSAL, int TBW>
__global__ __launch_bounds__(kBwdThreads) void k_bwd_dq(
    const T *__restrict__ Q, const T *__restrict__ K, const T *__restrict__ V,
    const T *__restrict__ dout, const T *__restrict__ out, const float *__restrict__ rsave,
    const typename Mma<T>::frag *__restrict__ wfr, const float *__restrict__ bqg,
    const float *__restrict__ W, const float *__restrict__ state, T *__restrict__ dQ,
    float2 *__restrict__ aux, int H, int L, float s, float keps, float wts, int ntiles,
    int nitems) {
  static_assert(!CAUSAL || TBW == 1, "a causal chunk is one 16-row block per wave");
  constexpr int NS = M / 32;
  constexpr int MB = M / 64;   // feature blocks per wave for the chunk's keys
  using P = Mma<T>;
  using frag = typename P::frag;
  __shared__ DqSmem<T, M, CAUSAL> sm;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;
  const float cM = sqrtf(2.0f / M);
  const float s2half = 0.5f * s * s;
  constexpr float sgn = KN == kCos ? -1.f : 1.f;

  int begin, end;
  if constexpr (CAUSAL) {
    begin = xcd_item(blockIdx.x, gridDim.x);
    end = begin + 1;
  } else {
    xcd_range(blockIdx.x, gridDim.x, nitems, begin, end);
  }
  int cur = -1;
  for (int item = begin; item < end; ++item) {
    const int bh = item / ntiles;
    const int tile = item - bh * ntiles;
    const int h = bh % H;
    const int t0 = tile * 64 * TBW;
    if (bh != cur) {
      __syncthreads();
      copy_frags<frag, (M / 16) * 2 * 64>(&sm.WA[0][0][0], wfr + (size_t)h * (M / 16) * 2 * 64);
      if (tid < M) sm.bq[tid] = bqg[(size_t)h * M + tid];
      build_wt<T, M>(sm.WT, W + (size_t)h * M * kD, wts);
      if constexpr (!CAUSAL) build_state_rows<T, M>(sm.SA, sm.sz, state + (size_t)bh * M * 65);
      cur = bh;
      __syncthreads();
    }
    if constexpr (CAUSAL) {
      build_state_rows<T, M>(sm.SA, sm.sz, state + ((size_t)bh * ntiles + tile) * M * 65);
      const T *Kh = K + (size_t)bh * L * kD;
      frag ka[4][2];
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) load_rows64<T>(ka[tb], Kh, t0 + 16 * tb + c16, L);
      chunk_features_t<T, MB, KN>(sm.KT, sm.WA, sm.bq, ka, w * MB, keps);
      frag va[2];
      load_rows64<T>(va, V + (size_t)bh * L * kD, t0 + 16 * w + c16, L);
      sm.VA[w][0][l] = va[0];
      sm.VA[w][1][l] = va[1];
      const float nrm = sq_norm16<T>(ka[w]);
      const bool in = t0 + 16 * w + c16 < L;
      const float D = !in ? 0.f : (KN == kCos ? cM * expf(s2half * nrm) : 1.f);
      if (g == 0) sm.dk[16 * w + c16] = D;
      __syncthreads();
    }

    const T *Qh = Q + (size_t)bh * L * kD;
    const T *dOh = dout + (size_t)bh * L * kD;
    const T *Oh = out + (size_t)bh * L * kD;
    frag qf[TBW][2], df[TBW][2];
    float alpha[TBW], ud[TBW];
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      const int i = t0 + 16 * (w * TBW + tb) + c16;
      load_rows64<T>(qf[tb], Qh, i, L);
      load_rows64<T>(df[tb], dOh, i, L);
      if constexpr (RN) {
        frag of[2];
        load_rows64<T>(of, Oh, i, L);
        float dot = 0.f;
#pragma unroll
        for (int k = 0; k < 2; ++k)
#pragma unroll
          for (int e = 0; e < 8; ++e) dot = fmaf(to_f32(df[tb][k][e]), to_f32(of[k][e]), dot);
        dot += __shfl_xor(dot, 16);
        dot += __shfl_xor(dot, 32);
        alpha[tb] = i < L ? rsave[(size_t)bh * L + i] : 0.f;
        ud[tb] = -dot;
      } else {
        float a = 1.f;
        if constexpr (KN == kCos) a = cM * expf(s2half * sq_norm16<T>(qf[tb]));
        alpha[tb] = i < L ? a : 0.f;
        ud[tb] = 0.f;
      }
    }

    // causal: P2[j][i] = D~_j (v_j . dout_i + u_d,i) for keys j <= i of the chunk,
    // packed as B operand (k = keys in chained order, column = query)
    frag pb2[2];
    if constexpr (CAUSAL) {
      f32x4 pt[4];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        f32x4 c = P::mma(sm.VA[kb][0][l], df[0][0], f32x4{0.f, 0.f, 0.f, 0.f});
        c = P::mma(sm.VA[kb][1][l], df[0][1], c);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int jp = 16 * kb + 4 * g + j;
          pt[kb][j] = jp <= 16 * w + c16 ? sm.dk[jp] * (c[j] + ud[0]) : 0.f;
        }
      }
      pb2[0] = P::pack(pt[0], pt[1]);
      pb2[1] = P::pack(pt[2], pt[3]);
    }

    f32x4 dacc[TBW][4];
    float dot2[TBW];
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      dot2[tb] = 0.f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) dacc[tb][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll 2
    for (int sidx = 0; sidx < NS; ++sidx) {
      f32x4 G[TBW][2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int mb = 2 * sidx + hh;
        const frag a0 = sm.WA[mb][0][l];
        const frag a1 = sm.WA[mb][1][l];
        const f32x4 bcv = *reinterpret_cast<const f32x4 *>(&sm.bq[16 * mb + 4 * g]);
        const frag s0 = sm.SA[mb][0][l];
        const frag s1 = sm.SA[mb][1][l];
        const f32x4 szv = *reinterpret_cast<const f32x4 *>(&sm.sz[16 * mb + 4 * g]);
#pragma unroll
        for (int tb = 0; tb < TBW; ++tb) {
          f32x4 p = P::mma(a0, qf[tb][0], bcv);
          p = P::mma(a1, qf[tb][1], p);
          f32x4 gt = P::mma(s0, df[tb][0], f32x4{0.f, 0.f, 0.f, 0.f});
          gt = P::mma(s1, df[tb][1], gt);
          if constexpr (CAUSAL) {
            gt = P::mma(sm.KT[mb][0][l], pb2[0], gt);
            gt = P::mma(sm.KT[mb][1][l], pb2[1], gt);
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float gj = fmaf(szv[j], ud[tb], gt[j]);
            dot2[tb] = fmaf(gj, feature<KN, P>(p[j], keps), dot2[tb]);
            G[tb][hh][j] = sgn * alpha[tb] * gj * feature_slope<KN, P>(p[j]);
          }
        }
      }
#pragma unroll
      for (int tb = 0; tb < TBW; ++tb) {
        const frag gb = P::pack(G[tb][0], G[tb][1]);
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) dacc[tb][kb] = P::mma(sm.WT[kb][sidx][l], gb, dacc[tb][kb]);
      }
    }

#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      const int i = t0 + 16 * (w * TBW + tb) + c16;
      float d2 = dot2[tb];
      d2 += __shfl_xor(d2, 16);
      d2 += __shfl_xor(d2, 32);
      const float cx = KN == kCos ? alpha[tb] * s * s * d2 : 0.f;
      if (i < L) {
        T *dst = dQ + ((size_t)bh * L + i) * kD;
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
          f32x4 lo, hi;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            lo[e] = fmaf(cx, to_f32(qf[tb][pp][e]), dacc[tb][2 * pp][e]);
            hi[e] = fmaf(cx, to_f32(qf[tb][pp][4 + e]), dacc[tb][2 * pp + 1][e]);
          }
          store8(dst + 32 * pp + 8 * g, lo, hi);
        }
        if (g == 0) aux[(size_t)bh * L + i] = make_float2(alpha[tb], alpha[tb] * ud[tb]);
      }
    }
  }
}

// ------------------------------------------------------------ dK, dV
constexpr int kPartBoth = 0;   // dK and dV (bidirectional)
constexpr int kPartDv = 1;     // dV only (causal)
constexpr int kPartDk = 2;     // dK only (causal)

template <typename T, int M, bool CAUSAL, int PART>
struct DkvSmem {
  using frag = typename Mma<T>::frag;
  static constexpr bool kK = PART != kPartDv;
  static constexpr bool kV = PART != kPartDk;
  frag WA[M / 16][2][64];
  float bq[M];
  frag WT[kK ? 4 : 1][kK ? M / 32 : 1][64];
  frag RA[kK ? M / 16 : 1][2][64];        // R rows over value columns
  float rz[kK ? M : 1];                   // R column d
  frag RB[kV ? 4 : 1][kV ? M / 32 : 1][64];   // R value columns over features
  // causal dV: the chunk's query features (lane row = query, k = m) and u~^T
  frag QA[CAUSAL && kV ? 4 : 1][CAUSAL && kV ? M / 32 : 1][64];
  frag UF[CAUSAL && kV ? 4 : 1][2][64];
  // causal dK: the chunk's query features (row m, k = queries), dout rows, weights
  frag QT[CAUSAL && kK ? M / 16 : 1][2][64];
  frag DA[CAUSAL && kK ? 4 : 1][2][64];
  float2 au[CAUSAL && kK ? 64 : 1];
};

template <typename T, int M, int KN, bool CAUSAL, int PART, int TBW>
__global__ __launch_bounds__(kBwdThreads) void k_bwd_dkv(
    const T *__restrict__ Q, const T *__restrict__ K, const T *__restrict__ V,
    const T *__restrict__ dout, const float2 *__restrict__ aux,
    const typename Mma<T>::frag *__restrict__ wfr, const float *__restrict__ bqg,
    const float *__restrict__ W, const float *__restrict__ rstate, T *__restrict__ dK,
    T *__restrict__ dV, int H, int L, float s, float keps, float wts, int ntiles, int nitems) {
  static_assert(!CAUSAL || TBW == 1, "a causal chunk is one 16-row block per wave");
  constexpr bool kK = PART != kPartDv;
  constexpr bool kV = PART != kPartDk;
  constexpr int NS = M / 32;
  constexpr int MB = M / 64;
  using P = Mma<T>;
  using frag = typename P::frag;
  __shared__ DkvSmem<T, M, CAUSAL, PART> sm;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;
  const float cM = sqrtf(2.0f / M);
  const float s2half = 0.5f * s * s;
  constexpr float sgn = KN == kCos ? -1.f : 1.f;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};

  int begin, end;
  if constexpr (CAUSAL) {
    begin = xcd_item(blockIdx.x, gridDim.x);
    end = begin + 1;
  } else {
    xcd_range(blockIdx.x, gridDim.x, nitems, begin, end);
  }
  int cur = -1;
  for (int item = begin; item < end; ++item) {
    const int bh = item / ntiles;
    const int tile = item - bh * ntiles;
    const int h = bh % H;
    const int t0 = tile * 64 * TBW;
    const float *Rs = CAUSAL ? rstate + ((size_t)bh * ntiles + tile) * M * 65
                             : rstate + (size_t)bh * M * 65;
    if (bh != cur) {
      __syncthreads();
      copy_frags<frag, (M / 16) * 2 * 64>(&sm.WA[0][0][0], wfr + (size_t)h * (M / 16) * 2 * 64);
      if (tid < M) sm.bq[tid] = bqg[(size_t)h * M + tid];
      if constexpr (kK) build_wt<T, M>(sm.WT, W + (size_t)h * M * kD, wts);
      if constexpr (!CAUSAL) {
        if constexpr (kK) build_state_rows<T, M>(sm.RA, sm.rz, Rs);
        if constexpr (kV) build_state_cols<T, M>(sm.RB, Rs);
      }
      cur = bh;
      __syncthreads();
    }
    if constexpr (CAUSAL) {
      if constexpr (kK) build_state_rows<T, M>(sm.RA, sm.rz, Rs);
      if constexpr (kV) build_state_cols<T, M>(sm.RB, Rs);
      const T *Qh = Q + (size_t)bh * L * kD;
      const T *dOh = dout + (size_t)bh * L * kD;
      const int iq = t0 + 16 * w + c16;   // this wave's queries
      if constexpr (kV) {
        // features of queries 16 w .. (lane row = query), and u~^T = alpha dout^T
        frag qf[2];
        load_rows64<T>(qf, Qh, iq, L);
#pragma unroll
        for (int sidx = 0; sidx < NS; ++sidx) {
          f32x4 f[2];
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int mb = 2 * sidx + hh;
            const f32x4 bcv = *reinterpret_cast<const f32x4 *>(&sm.bq[16 * mb + 4 * g]);
            f32x4 p = P::mma(sm.WA[mb][0][l], qf[0], bcv);
            p = P::mma(sm.WA[mb][1][l], qf[1], p);
#pragma unroll
            for (int j = 0; j < 4; ++j) f[hh][j] = feature<KN, P>(p[j], keps);
          }
          sm.QA[w][sidx][l] = P::pack(f[0], f[1]);
        }
        frag dfq[2];
        load_rows64<T>(dfq, dOh, iq, L);
        float aj[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int t = t0 + 16 * w + 4 * g + j;
          aj[j] = t < L ? aux[(size_t)bh * L + t].x : 0.f;
        }
        const frag sel[2] = {select_perm<T>(0), select_perm<T>(1)};
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            const f32x4 c = P::mma(dfq[kh], sel[half], zero4);
            T *p = reinterpret_cast<T *>(&sm.UF[2 * kh + half][w >> 1][l]) + 4 * (w & 1);
#pragma unroll
            for (int j = 0; j < 4; ++j) p[j] = from_f32<T>(c[j] * aj[j]);
          }
      }
      if constexpr (kK) {
        frag qa[4][2];
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) load_rows64<T>(qa[tb], Qh, t0 + 16 * tb + c16, L);
        chunk_features_t<T, MB, KN>(sm.QT, sm.WA, sm.bq, qa, w * MB, keps);
        frag dfq[2];
        load_rows64<T>(dfq, dOh, iq, L);
        sm.DA[w][0][l] = dfq[0];
        sm.DA[w][1][l] = dfq[1];
        if (g == 0) sm.au[16 * w + c16] = iq < L ? aux[(size_t)bh * L + iq] : make_float2(0.f, 0.f);
      }
      __syncthreads();
    }

    const T *Kh = K + (size_t)bh * L * kD;
    const T *Vh = V + (size_t)bh * L * kD;
    frag kf[TBW][2], vf[TBW][2];
    float Dk[TBW];
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      const int j = t0 + 16 * (w * TBW + tb) + c16;
      load_rows64<T>(kf[tb], Kh, j, L);
      load_rows64<T>(vf[tb], Vh, j, L);
      float D = 1.f;
      if constexpr (KN == kCos) D = cM * expf(s2half * sq_norm16<T>(kf[tb]));
      Dk[tb] = j < L ? D : 0.f;
    }
    // causal dK: P3[i][j] = alpha_i (dout_i . v_j + u_d,i) for queries i >= j
    frag pb3[2];
    if constexpr (CAUSAL && kK) {
      f32x4 pt[4];
#pragma unroll
      for (int qb = 0; qb < 4; ++qb) {
        f32x4 c = P::mma(sm.DA[qb][0][l], vf[0][0], zero4);
        c = P::mma(sm.DA[qb][1][l], vf[0][1], c);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int ip = 16 * qb + 4 * g + j;
          const float2 a = sm.au[ip];
          pt[qb][j] = ip >= 16 * w + c16 ? fmaf(a.x, c[j], a.y) : 0.f;
        }
      }
      pb3[0] = P::pack(pt[0], pt[1]);
      pb3[1] = P::pack(pt[2], pt[3]);
    }

    f32x4 kacc[TBW][4], vacc[TBW][4], p4[4];
    float doth[TBW];
#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      doth[tb] = 0.f;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        kacc[tb][k] = zero4;
        vacc[tb][k] = zero4;
      }
    }
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) p4[qb] = zero4;

#pragma unroll 2
    for (int sidx = 0; sidx < NS; ++sidx) {
      f32x4 kh[TBW][2], G[TBW][2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int mb = 2 * sidx + hh;
        const frag a0 = sm.WA[mb][0][l];
        const frag a1 = sm.WA[mb][1][l];
        const f32x4 bcv = *reinterpret_cast<const f32x4 *>(&sm.bq[16 * mb + 4 * g]);
#pragma unroll
        for (int tb = 0; tb < TBW; ++tb) {
          f32x4 p = P::mma(a0, kf[tb][0], bcv);
          p = P::mma(a1, kf[tb][1], p);
#pragma unroll
          for (int j = 0; j < 4; ++j) kh[tb][hh][j] = feature<KN, P>(p[j], keps);
          if constexpr (kK) {
            f32x4 hv = P::mma(sm.RA[mb][0][l], vf[tb][0], zero4);
            hv = P::mma(sm.RA[mb][1][l], vf[tb][1], hv);
            if constexpr (CAUSAL) {
              hv = P::mma(sm.QT[mb][0][l], pb3[0], hv);
              hv = P::mma(sm.QT[mb][1][l], pb3[1], hv);
            }
            const f32x4 rzv = *reinterpret_cast<const f32x4 *>(&sm.rz[16 * mb + 4 * g]);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const float hj = hv[j] + rzv[j];
              doth[tb] = fmaf(hj, kh[tb][hh][j], doth[tb]);
              G[tb][hh][j] = sgn * hj * feature_slope<KN, P>(p[j]);
            }
          }
        }
      }
#pragma unroll
      for (int tb = 0; tb < TBW; ++tb) {
        if constexpr (kK) {
          const frag gb = P::pack(G[tb][0], G[tb][1]);
#pragma unroll
          for (int kb = 0; kb < 4; ++kb) kacc[tb][kb] = P::mma(sm.WT[kb][sidx][l], gb, kacc[tb][kb]);
        }
        if constexpr (kV) {
          const frag kb_ = P::pack(kh[tb][0], kh[tb][1]);
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) vacc[tb][nb] = P::mma(sm.RB[nb][sidx][l], kb_, vacc[tb][nb]);
          if constexpr (CAUSAL) {
#pragma unroll
            for (int qb = 0; qb < 4; ++qb) p4[qb] = P::mma(sm.QA[qb][sidx][l], kb_, p4[qb]);
          }
        }
      }
    }
    if constexpr (CAUSAL && kV) {
      // keep queries i >= j, then u~^T (q-hat . k-hat) into the value gradient
#pragma unroll
      for (int qb = 0; qb < 4; ++qb)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          p4[qb][j] = 16 * qb + 4 * g + j >= 16 * w + c16 ? p4[qb][j] : 0.f;
#pragma unroll
      for (int sidx = 0; sidx < 2; ++sidx) {
        const frag pb = P::pack(p4[2 * sidx], p4[2 * sidx + 1]);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) vacc[0][nb] = P::mma(sm.UF[nb][sidx][l], pb, vacc[0][nb]);
      }
    }

#pragma unroll
    for (int tb = 0; tb < TBW; ++tb) {
      const int j = t0 + 16 * (w * TBW + tb) + c16;
      float dh = doth[tb];
      if constexpr (kK) {
        dh += __shfl_xor(dh, 16);
        dh += __shfl_xor(dh, 32);
      }
      if (j < L) {
        const float D = Dk[tb];
        if constexpr (kK) {
          const float cx = KN == kCos ? s * s * dh : 0.f;
          T *dst = dK + ((size_t)bh * L + j) * kD;
#pragma unroll
          for (int pp = 0; pp < 2; ++pp) {
            f32x4 lo, hi;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              lo[e] = D * fmaf(cx, to_f32(kf[tb][pp][e]), kacc[tb][2 * pp][e]);
              hi[e] = D * fmaf(cx, to_f32(kf[tb][pp][4 + e]), kacc[tb][2 * pp + 1][e]);
            }
            store8(dst + 32 * pp + 8 * g, lo, hi);
          }
        }
        if constexpr (kV) {
          T *dst = dV + ((size_t)bh * L + j) * kD;
#pragma unroll
          for (int pp = 0; pp < 2; ++pp)
            store8(dst + 32 * pp + 8 * g, vacc[tb][2 * pp] * D, vacc[tb][2 * pp + 1] * D);
        }
      }
    }
  }
}

// ------------------------------------------------------------ launchers
// M dispatch; fp32 operands double the LDS tables, so fp32 stops at M = 128.
#define FAVOR_BWD_DISPATCH_M(T_, M_, ...)                                  \
  switch (M_) {                                                            \
    case 64: { constexpr int MM = 64; __VA_ARGS__; } break;                 \
    case 128: { constexpr int MM = 128; __VA_ARGS__; } break;               \
    case 256:                                                              \
      if constexpr (sizeof(T_) == 2) {                                      \
        constexpr int MM = 256;                                            \
        __VA_ARGS__;                                                       \
        break;                                                             \
      } else {                                                             \
        return hipErrorInvalidValue;                                       \
      }                                                                    \
    default: return hipErrorInvalidValue;                                  \
  }

// Scale of W in the input-gradient products: s for cos features (2 pi W'' = s W),
// s / sqrt(M) for ReLU features (W'' itself).
static float wt_scale(const Shape &sh) {
  return sh.kernel == 1 ? sh.s / sqrtf((float)sh.M) : sh.s;
}

// Rows per persistent bidirectional tile: 4 waves x TBW blocks of 16.
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
                              float *dsin, hipStream_t st) {
  const int n4 = sh.M * 65 / 4;
  dim3 grid((n4 + 255) / 256, sh.BH);
  hipLaunchKernelGGL(k_suffix_scan, grid, dim3(256), 0, st, (f32x4 *)part, nch, n4,
                     (const f32x4 *)dsout, (f32x4 *)dsin);
  return hipGetLastError();
}

template <typename T, bool CAUSAL>
static hipError_t bwd_dq_typed(const Shape &sh, const BwdArgs &a, hipStream_t st) {
  constexpr int TBW = CAUSAL ? 1 : kBwdTbw;
  const int rows = 64 * TBW;
  const int ntiles = (sh.L + rows - 1) / rows;
  const int nitems = ntiles * sh.BH;
  dim3 grid(CAUSAL ? nitems : min(nitems, kBwdMaxWorkgroups));
  const float wts = wt_scale(sh);
  auto go = [&](auto kn, auto rn) -> hipError_t {
    constexpr int KN = decltype(kn)::value;
    constexpr bool RN = decltype(rn)::value;
    FAVOR_BWD_DISPATCH_M(T, sh.M,
        hipLaunchKernelGGL((k_bwd_dq<T, MM, KN, RN, CAUSAL, TBW>), grid, dim3(kBwdThreads), 0, st,
                           (const T *)a.Q, (const T *)a.K, (const T *)a.V, (const T *)a.dout,
                           (const T *)a.out, a.rsave, (const typename Mma<T>::frag *)a.wfr, a.bq,
                           a.W, a.state, (T *)a.dQ, (float2 *)a.aux, sh.H, sh.L, sh.s, sh.keps,
                           wts, ntiles, nitems));
    return hipGetLastError();
  };
  using relu = std::integral_constant<int, kRelu>;
  using cosk = std::integral_constant<int, kCos>;
  if (sh.kernel == 1) return sh.renorm ? go(relu{}, std::true_type{}) : go(relu{}, std::false_type{});
  return sh.renorm ? go(cosk{}, std::true_type{}) : go(cosk{}, std::false_type{});
}

hipError_t launch_bwd_dq(const Shape &sh, Dt in, bool causal, const BwdArgs &a, hipStream_t st) {
  if (in == Dt::BF16)
    return causal ? bwd_dq_typed<bf16, true>(sh, a, st) : bwd_dq_typed<bf16, false>(sh, a, st);
  if (sh.M > 128) return hipErrorInvalidValue;
  return causal ? bwd_dq_typed<float, true>(sh, a, st) : bwd_dq_typed<float, false>(sh, a, st);
}

template <typename T, bool CAUSAL, int PART>
static hipError_t bwd_dkv_typed(const Shape &sh, const BwdArgs &a, hipStream_t st) {
  constexpr int TBW = CAUSAL ? 1 : kBwdTbw;
  const int rows = 64 * TBW;
  const int ntiles = (sh.L + rows - 1) / rows;
  const int nitems = ntiles * sh.BH;
  dim3 grid(CAUSAL ? nitems : min(nitems, kBwdMaxWorkgroups));
  const float wts = wt_scale(sh);
  auto go = [&](auto kn) -> hipError_t {
    constexpr int KN = decltype(kn)::value;
    FAVOR_BWD_DISPATCH_M(T, sh.M,
        hipLaunchKernelGGL((k_bwd_dkv<T, MM, KN, CAUSAL, PART, TBW>), grid, dim3(kBwdThreads), 0,
                           st, (const T *)a.Q, (const T *)a.K, (const T *)a.V, (const T *)a.dout,
                           (const float2 *)a.aux, (const typename Mma<T>::frag *)a.wfr, a.bq, a.W,
                           a.state, (T *)a.dK, (T *)a.dV, sh.H, sh.L, sh.s, sh.keps, wts, ntiles,
                           nitems));
    return hipGetLastError();
  };
  if (sh.kernel == 1) return go(std::integral_constant<int, kRelu>{});
  return go(std::integral_constant<int, kCos>{});
}

hipError_t launch_bwd_dkv(const Shape &sh, Dt in, bool causal, const BwdArgs &a, hipStream_t st) {
  if (in == Dt::BF16) {
    if (!causal) return bwd_dkv_typed<bf16, false, kPartBoth>(sh, a, st);
    hipError_t e = bwd_dkv_typed<bf16, true, kPartDv>(sh, a, st);
    if (e != hipSuccess) return e;
    return bwd_dkv_typed<bf16, true, kPartDk>(sh, a, st);
  }
  if (sh.M > 128) return hipErrorInvalidValue;
  if (!causal) return bwd_dkv_typed<float, false, kPartBoth>(sh, a, st);
  hipError_t e = bwd_dkv_typed<float, true, kPartDv>(sh, a, st);
  if (e != hipSuccess) return e;
  return bwd_dkv_typed<float, true, kPartDk>(sh, a, st);
}

}  // namespace favor
