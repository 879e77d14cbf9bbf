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
// computed. ReLU features (generalized attention, Sec. 2.2) replace the cosine
// by max(., 0) + keps with D = 1; without renormalisation the numerator is
// scaled by the query factor D_Q sqrt(2/M) (1 for ReLU) instead of divided.
#include <type_traits>

#include "favor_common.hpp"
#include "kernels.hpp"
#include "tile_common.hpp"

namespace favor {

// Workgroup (feature block of 32 rows, head): the 32 x 65 aggregates of its
// rows are 520 consecutive float4; thread u takes unit u (one thread per unit,
// so every unit's loads are in flight together) and walks the segments eight
// loads at a time, replacing every segment aggregate by the
// exclusive prefix (plus state_in). The total of this call's tokens goes
// through LDS into the Buf1^T fragments when frags is non-null: fragment lane
// (nb, l) of this k-step holds, in slot i, feature 16 (i / 4) + 4 (l / 16) + i % 4
// of value column pi(nb, l % 16) (block 4: the denominator column 64 in all
// 16 lane rows), written as one vector store. total (nullable) receives the
// same total in the layout of an aggregate ([M][65] fp32 per head), for the
// backward pass.
constexpr int kSegScanThreads = 576;   // 520 float4 units of a 32-row block, nine waves

template <typename E>
__global__ __launch_bounds__(kSegScanThreads) void k_seg_scan(float *__restrict__ part, int nseg, int M,
                                                  int Mr, const float *__restrict__ state_in,
                                                  float *__restrict__ state_out,
                                                  E *__restrict__ frags,
                                                  float *__restrict__ total) {
  constexpr int kUnits = 32 * 65 / 4;   // float4 per 32-row block
  __shared__ f32x4 tot[kUnits];
  const int sidx = blockIdx.x;
  const int bh = blockIdx.y;
  const int n65 = M * 65;
  // state_in / state_out hold the M_r rows drawn: the same row-major index, a
  // head stride of M_r rows, and no padding rows (M_r 65 is a multiple of 4)
  const int nuser = Mr * 65 / 4;
  const size_t head = (size_t)bh * nuser + (size_t)sidx * kUnits;   // in float4
  f32x4 *p = reinterpret_cast<f32x4 *>(part) + (size_t)bh * nseg * (n65 / 4) + sidx * kUnits;
  const size_t stride = n65 / 4;   // one segment, in float4
  static_assert(kUnits <= kSegScanThreads, "one thread per unit");
  const int u = threadIdx.x;
  if (u < kUnits) {
    const bool drawn = sidx * kUnits + u < nuser;
    const f32x4 s0 = state_in && drawn ? reinterpret_cast<const f32x4 *>(state_in)[head + u]
                                       : f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 run = {0.f, 0.f, 0.f, 0.f};   // aggregate of the segments before sg
    int sg = 0;
    for (; sg + 8 <= nseg; sg += 8) {   // eight loads in flight
      f32x4 v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = p[(sg + k) * stride + u];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        p[(sg + k) * stride + u] = s0 + run;
        run += v[k];
      }
    }
    for (; sg < nseg; ++sg) {
      const f32x4 v = p[sg * stride + u];
      p[sg * stride + u] = s0 + run;
      run += v;
    }
    if (state_out && drawn) reinterpret_cast<f32x4 *>(state_out)[head + u] = s0 + run;
    if (total)
      reinterpret_cast<f32x4 *>(total)[(size_t)bh * (n65 / 4) + (size_t)sidx * kUnits + u] = run;
    tot[u] = run;
  }
  if (!frags) return;
  __syncthreads();
  const float *t = reinterpret_cast<const float *>(tot);
  const int ns = M / 32;
  for (int f = threadIdx.x; f < 5 * 64; f += kSegScanThreads) {
    const int nb = f >> 6;
    const int l = f & 63;
    const int gq = l >> 4;
    const int n = nb < 4 ? perm_col(nb, l & 15) : 64;
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = t[(16 * (i >> 2) + 4 * gq + (i & 3)) * 65 + n];
    reinterpret_cast<typename Mma<E>::frag *>(frags)[((size_t)bh * 5 * ns + nb * ns + sidx) * 64 + l] =
        Mma<E>::from_f32(v, 1.f);
  }
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

// SAVE: also write each row's 1 / (D-hat + eps) in units of the unscaled
// features (rsave [B*H][L]) for the backward pass.
// PART: 0 all M features; 1 and 2 the features [m0, m0 + M) of Mall (the
// head strides of W'', b'' and the prefix states): pass 1 stores each row's raw
// numerators and denominator (halves [B*H][L][kHalfRow]), pass 2 adds its own
// and finalises. Buf2 is a sum over features, so the two passes together give
// the one-pass result; they let fp32 inputs take M = 256 on tables sized for 128.
constexpr int kHalfRow = 68;   // 64 numerators, the denominator, padding to 16 bytes
template <typename T, typename To, int M, int KN, bool RN, bool SAVE, int PART>
__global__ __launch_bounds__(256) void k_causal(const T *__restrict__ Q, const T *__restrict__ K,
                                                const T *__restrict__ V,
                                                const typename Mma<T>::frag *__restrict__ wfr,
                                                const float *__restrict__ bqg,
                                                const float *__restrict__ prefix,
                                                To *__restrict__ out, float *__restrict__ rsave,
                                                float *__restrict__ halves, int H, int L,
                                                int seg_len, int nseg, float s, float eps,
                                                float cM, int Mall, int m0) {
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

  const frag *wh = wfr + ((size_t)h * (Mall / 16) + m0 / 16) * 2 * 64;
  copy_frags<frag, (M / 16) * 2 * 64>(&sm.WA[0][0][0], wh);
  if (tid < M) sm.bq[tid] = bqg[(size_t)h * Mall + m0 + tid];
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
    const float *pre = prefix + (((size_t)bh * nseg + seg) * Mall + m0) * 65;
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
  const int r0 = seg * seg_len;
  const int r1 = min(L, r0 + seg_len);

  __syncthreads();
  TileRegs<T> rg;
  load_tile_regs<T>(rg, Kh, Vh, r0, r1, tid);
  frag qn[2];
  load_query_frags<T>(qn, Qh, r0 + 16 * w + c16, r1);
  KVTile<T> &tl = sm.tl;
  for (int t0 = r0; t0 < r1; t0 += 64) {
    const bool next = t0 + 64 < r1;
    // the previous chunk's readers are done: stage this chunk's prefetched keys
    // and values and publish S (the state before this chunk)
    {
      const frag sel[2] = {sm.SEL[0][l], sm.SEL[1][l]};
      stage_tile<T, KN>(tl, rg, sel, t0, r1, s2half, cM, tid);
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
      load_tile_regs<T>(rg, Kh, Vh, t0 + 64, r1, tid);
      load_query_frags<T>(qn, Qh, t0 + 64 + 16 * w + c16, r1);
    }

    // key features of this wave's feature range: fold into S, and publish them
    // transposed (row = token) for the intra-chunk products
#pragma unroll
    for (int sidx = 0; sidx < 2; ++sidx) {
      f32x4 kf[MB][2];
      key_features_lds<T, MB, KN>(tl, sm.WA, sm.bq, w * MB, sidx, kf);
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
    // the stabiliser in units of the unscaled features, or (renormalisation
    // off) the factor D_Q sqrt(2/M) they omit; ReLU features carry their scale
    float epsq = RN ? (KN == kCos ? 0.f : eps) : 1.f;
    if (KN == kCos && (!RN || eps != 0.f)) {
      float nrm = sq_sum16(qf);
      nrm += __shfl_xor(nrm, 16);
      nrm += __shfl_xor(nrm, 32);
      const float dq = cM * expf(s2half * nrm);
      epsq = RN ? eps / dq : dq;
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
        for (int j = 0; j < 4; ++j) pf[hh][j] = feature<KN, P>(pc[hh][j], cur.bc[hh][j]);
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
      float *hp = halves + ((size_t)bh * L + qt) * kHalfRow;
      if constexpr (PART == 1) {   // raw partials of the first feature half
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
          *reinterpret_cast<f32x4 *>(hp + nb * 16 + 4 * g) = o[nb];
        if (g == 0) hp[64] = o[4][0];
      } else {
        if constexpr (PART == 2) {
#pragma unroll
          for (int nb = 0; nb < 4; ++nb)
            o[nb] += *reinterpret_cast<const f32x4 *>(hp + nb * 16 + 4 * g);
          o[4][0] += hp[64];
        }
        const float inv = RN ? 1.0f / (o[4][0] + epsq) : epsq;
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
          store4(Oh + (size_t)qt * kD + nb * 16 + 4 * g, o[nb] * inv);
        if constexpr (SAVE) {
          if (g == 0) rsave[(size_t)bh * L + qt] = inv;
        }
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Feature-split form for bf16 inputs, chunks of T = 64 or 32 tokens. Wave w
// owns features [w MW, (w + 1) MW), MW = M / 4, for the keys and for the
// queries of every chunk: its slice of the state S (fp32 accumulators, rows m
// of its slice, 65 columns padded to 80 with the ones column replicated over
// the last 16) never leaves its registers, its W'' fragments are loaded once,
// and its key features are transposed on the matrix cores without LDS. Since
//   Buf2 = Q-hat S + tril(Q-hat K-hat^T) C~ = sum over feature slices,
// each wave forms partial numerators and denominators for all T tokens of
// the chunk. The chunk's output is cut into four units, each finalised by one
// wave from its own partial and the three others, handed over through LDS:
// T = 64, unit w = tokens 16 w .. 16 w + 15; T = 32, unit w = tokens
// 16 (w % 2) .. + 15, value columns 32 (w / 2) .. + 31. Tiles of K, Q and C~
// and the hand-over area are double-buffered, so one barrier per chunk
// separates producers from consumers.
//
// Value columns are held in a permuted order: row r of value block nb (the
// lane row of C~ as an A operand, the row of an output tile) is column
//   pi(nb, r) = 32 (nb / 2) + 8 (r / 4) + 4 (nb % 2) + r % 4,
// so that the lane holding rows 4 g .. 4 g + 3 of blocks 2 p and 2 p + 1 holds
// the eight consecutive output columns 32 p + 8 g .. 32 p + 8 g + 7.
// Calls f(integral_constant<int, I>) for I = B .. E - 1 in order.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

template <int T>
struct CausalFsTile {
  bf16 Ks[T][kD + kKsPad];       // keys row-major (A operand of the key projection)
  bf16x8 VtF[4][T / 32][64];     // C~ (permuted columns), chained token order per 32 keys
  bf16x8 DF[T / 32][4];          // D_K (the ones column of C~), chained order
  bf16 Qs[T][kD + kKsPad];       // queries row-major (B operand of the query projection)
  float epsq[T];                 // per query: eps / (sqrt(2/M) D_Q), or sqrt(2/M) D_Q
                                 // when the result is not renormalised
};
template <int T>
struct CausalFsSmem {
  CausalFsTile<T> tile[2];
  f32x4 num[2][4][3][T / 16][64];   // [buffer][source wave][slot][value block of the unit][lane]
  float den[2][4][3][16];           // [buffer][source wave][slot][token]
  float bq[256];                    // b'' of the head (T = 32: the query projections read it here)
  bf16x8 sel[2][64];                // T = 32: the selection fragments of the value transposes
};

// Selection matrix in loaded k order with B[k][c] = (k == 8 (c / 4) + 4 half + c % 4):
// the MFMA of value rows (A operand, k = 32 value columns of step kh) with it
// moves value column 32 kh + 8 (c / 4) + 4 half + c % 4 = pi(2 kh + half, c) to lane c.
__device__ __forceinline__ bf16x8 select_perm_frag(int half) {
  const int l = lane_id();
  const int c = l & 15;
  float v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (8 * (l >> 4) + i == 8 * (c >> 2) + 4 * half + (c & 3)) ? 1.f : 0.f;
  return Mma<bf16>::from_f32(v, 1.f);
}

// Sum over the four lanes of an aligned quad (DPP quad permutes).
__device__ __forceinline__ float quad_sum_f32(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, false));
  return v;
}

// A wave-uniform value the optimiser may not look through (it stays in scalar
// registers): keeps loop invariant code motion from hoisting loads that are
// meant to be repeated.
__device__ __forceinline__ int opaque_uniform(int x) {
  asm volatile("" : "+s"(x));
  return x;
}

// Raw buffer access (T = 32 scan): the base is a scalar resource covering the
// bytes a call may touch, the lane offset one 32-bit register, so the loop
// holds no per-lane 64-bit address (with generic pointers the compiler hoists
// base + lane offset out of the loop as a 64-bit pair per address). Word 3 of
// the resource is the 32-bit data format of raw buffer access on this family.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                           0x00020000);
}
__device__ __forceinline__ bf16x8 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off, int soff = 0) {
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, off, soff, 0));
}
__device__ __forceinline__ void buf_store8(__amdgpu_buffer_rsrc_t r, uint32_t off, bf16 *,
                                           f32x4 a, f32x4 b) {
  bf16x8 v;
  v[0] = (bf16)a[0]; v[1] = (bf16)a[1]; v[2] = (bf16)a[2]; v[3] = (bf16)a[3];
  v[4] = (bf16)b[0]; v[5] = (bf16)b[1]; v[6] = (bf16)b[2]; v[7] = (bf16)b[3];
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, off, 0, 0);
}
__device__ __forceinline__ void buf_store8(__amdgpu_buffer_rsrc_t r, uint32_t off, float *,
                                           f32x4 a, f32x4 b) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, a), r, off, 0, 0);
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, b), r, off + 16, 0, 0);
}

// Query rows of a T-token tile, row (tid mod 4T) / 4, 16 columns (T = 32:
// waves 0 and 1 load them, waves 2 and 3 take zeros).
template <int T>
__device__ __forceinline__ void load_q_rows(bf16x8 (&q)[2], const bf16 *__restrict__ Qh, int t0,
                                            int r1) {
  const int tid = threadIdx.x;
  const int lr = T == 64 ? tid >> 2 : (tid & 127) >> 2;
  if (t0 + lr < r1 && (T == 64 || tid < 4 * T)) {
    if constexpr (T == 64) {
      const bf16 *qp = Qh + (size_t)(t0 + lr) * kD + (tid & 3) * 16;
      q[0] = load_frag<bf16>(qp);
      q[1] = load_frag<bf16>(qp + 8);
    } else {
      const auto rs = buf_rsrc(Qh + (size_t)t0 * kD, T * kD * 2);
      const uint32_t off = (lr * kD + (tid & 3) * 16) * 2;
      q[0] = buf_load16(rs, off);
      q[1] = buf_load16(rs, off + 16);
    }
  } else {
    q[0] = Mma<bf16>::splat(0.f);
    q[1] = Mma<bf16>::splat(0.f);
  }
}

// Keys and values of a T-token tile in registers. T = 64: load_tile_regs.
// T = 32: every wave loads the keys of rows (tid mod 128) / 4 (waves 2 and 3
// repeat those of waves 0 and 1, for the D_K of the tokens they transpose)
// and the values of rows 16 (w % 2) + lane % 16, columns 32 (w / 2) + 8 g ..
// into v[0].
template <int T>
__device__ __forceinline__ void load_causal_tile_regs(TileRegs<bf16> &r, const bf16 *__restrict__ Kh,
                                                      const bf16 *__restrict__ Vh, int t0, int r1,
                                                      int tid) {
  if constexpr (T == 64) {
    load_tile_regs<bf16>(r, Kh, Vh, t0, r1, tid);
  } else {
    const int l = tid & 63;
    const int w = tid >> 6;
    const int lk = (tid & 127) >> 2;
    const int lv = 16 * (w & 1) + (l & 15);
    if (t0 + lk < r1) {
      const auto rs = buf_rsrc(Kh + (size_t)t0 * kD, T * kD * 2);
      const uint32_t off = (lk * kD + (tid & 3) * 16) * 2;
      r.k[0] = buf_load16(rs, off);
      r.k[1] = buf_load16(rs, off + 16);
    } else {
      r.k[0] = Mma<bf16>::splat(0.f);
      r.k[1] = Mma<bf16>::splat(0.f);
    }
    r.v[0] = t0 + lv < r1 ? buf_load16(buf_rsrc(Vh + (size_t)t0 * kD, T * kD * 2),
                                       (lv * kD + 32 * (w >> 1) + 8 * (l >> 4)) * 2)
                          : Mma<bf16>::splat(0.f);
  }
}

// Stage a prefetched tile: keys and queries row-major, D_K(t) = sqrt(2/M)
// exp(||s k_t||^2 / 2) (1 for ReLU features; 0 past r1), C~ = D_K [V 1] as
// chained-order B fragments in permuted column order (T = 64: wave w
// transposes the values of tokens 16 w ..; T = 32: of tokens 16 (w % 2) ..,
// value columns 32 (w / 2) ..), and the per-query stabiliser when eps != 0
// (the query factor when not renormalising).
template <int T, int KN, bool RN>
__device__ __forceinline__ void stage_causal_tile(CausalFsTile<T> &tl, const TileRegs<bf16> &r,
                                                  const bf16x8 (&q)[2], const bf16x8 (&sel)[2],
                                                  int t0, int r1, float s2half, float cM,
                                                  float eps) {
  using P = Mma<bf16>;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;
  const int tr = T == 64 ? tid >> 2 : (tid & 127) >> 2;
  const int cq = (tid & 3) * 16;
  const bool rows_owner = T == 64 || tid < 4 * T;   // T = 32: waves 0 and 1 store the rows
  if (rows_owner) {
    store_frag<bf16>(&tl.Ks[tr][cq], r.k[0]);
    store_frag<bf16>(&tl.Ks[tr][cq + 8], r.k[1]);
    store_frag<bf16>(&tl.Qs[tr][cq], q[0]);
    store_frag<bf16>(&tl.Qs[tr][cq + 8], q[1]);
  }
  float Dt = (t0 + tr < r1) ? 1.f : 0.f;
  if constexpr (KN == kCos) {
    float nrm = quad_sum_f32(sq_sum16(r.k));
    Dt = (t0 + tr < r1) ? cM * expf(s2half * nrm) : 0.f;
  }
  // D of tokens 16 (w mod T/16) + 4 g + j, held by the quad of lanes 16 g + 4 j
  float Dj[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) Dj[j] = __shfl(Dt, 16 * g + 4 * j);
  const int sidx = T == 64 ? w >> 1 : 0;
  const int hw = w & 1;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  auto transpose = [&](const bf16x8 &v, int kh) __attribute__((always_inline)) {
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const f32x4 c = P::mma(v, sel[half], zero4);
      bf16 *p = reinterpret_cast<bf16 *>(&tl.VtF[2 * kh + half][sidx][l]) + 4 * hw;
#pragma unroll
      for (int j = 0; j < 4; ++j) p[j] = (bf16)(c[j] * Dj[j]);
    }
  };
  if constexpr (T == 64) {
    transpose(r.v[0], 0);
    transpose(r.v[1], 1);
  } else {
    transpose(r.v[0], w >> 1);
  }
  if (c16 == 0 && (T == 64 || w < 2)) {
    bf16 *p = reinterpret_cast<bf16 *>(&tl.DF[sidx][g]) + 4 * hw;
#pragma unroll
    for (int j = 0; j < 4; ++j) p[j] = (bf16)Dj[j];
  }
  if (KN == kCos && (!RN || eps != 0.f)) {
    const float qn = quad_sum_f32(sq_sum16(q));
    const float dq = cM * expf(s2half * qn);
    if ((tid & 3) == 0 && rows_owner) tl.epsq[tr] = (t0 + tr < r1) ? (RN ? eps / dq : dq) : 0.f;
  }
}

template <typename To, int M, int KN, bool RN, bool SAVE, int T = 64>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(T == 32 ? 2 : 1))) void k_causal_fs(const bf16 *__restrict__ Q,
                                                   const bf16 *__restrict__ K,
                                                   const bf16 *__restrict__ V,
                                                   const bf16x8 *__restrict__ wfr,
                                                   const float *__restrict__ bqg,
                                                   const float *__restrict__ prefix,
                                                   To *__restrict__ out, float *__restrict__ rsave,
                                                   int H, int L, int seg_len, int nseg, float s,
                                                   float eps, float cM) {
  constexpr int MW = M / 4;          // features per wave
  constexpr int MB = MW / 16;        // 16-feature blocks per wave
  constexpr int KS = (MB + 1) / 2;   // 32-feature k-steps per wave (a lone block is zero-padded)
  constexpr int NTB = T / 16;        // 16-token blocks of a chunk
  constexpr int NKH = T / 32;        // 32-token key halves of a chunk
  constexpr int NVB = NTB;           // 16-column value blocks of an output unit
  static_assert(T == 32 || T == 64, "chunks of 32 or 64 tokens");
  using P = Mma<bf16>;
  using frag = bf16x8;
  __shared__ CausalFsSmem<T> sm;

  const int item = xcd_item(blockIdx.x, gridDim.x);
  const int bh = item / nseg;
  const int seg = item - bh * nseg;
  const int h = bh % H;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;
  const int utb = T == 64 ? w : (w & 1);   // this wave's output unit: token block,
  const int uvh = T == 64 ? 0 : (w >> 1);  // and value-column group (T = 32)
  // T = 32 runs two workgroups per CU (two waves per SIMD, at most 256 registers
  // each). M = 256 fits only in a reordered chunk: the seeds b'' stay in LDS
  // and W'' is loaded again for every chunk, a chunk starts with the previous
  // chunk's finalisation, the next tile is staged after the features, the
  // loads of the one after it go out after the contractions, and the
  // contractions run one value block at a time, each block handed over as
  // soon as it is complete. Smaller M keeps the order of the 64-token chunk,
  // which is faster where it fits.
  constexpr bool kLate = T == 32 && M > 128;
  // The contractions streamed one value block at a time (each block handed
  // over as soon as it is complete) hold far fewer partial outputs; with
  // 64-token chunks (one wave per SIMD either way) the form that first forms
  // all partials and then hands them over is 2% faster.
  constexpr bool kStream = kLate;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};

  const bf16 *Qh = Q + (size_t)bh * L * kD;
  const bf16 *Kh = K + (size_t)bh * L * kD;
  const bf16 *Vh = V + (size_t)bh * L * kD;
  To *Oh = out + (size_t)bh * L * kD;
  const float s2half = 0.5f * s * s;
  const int r0 = seg * seg_len;
  const int r1 = min(L, r0 + seg_len);

  // the first tile's loads go out first: staging waits for them alone
  TileRegs<bf16> rg;
  frag rq[2];
  load_causal_tile_regs<T>(rg, Kh, Vh, r0, r1, tid);
  load_q_rows<T>(rq, Qh, r0, r1);

  // W'' fragments of this wave's features: A operand of the query projection
  // (lane row m), B operand of the key one (lane col m); b'' per row and column
  frag wf[MB][2];
  float bk[MB];
  f32x4 bqv[MB];
  // T = 32: the fragments are loaded again for every chunk (after the previous
  // chunk's contractions), from a base the compiler may not treat as loop
  // invariant, so that they are not held across the contractions
  const frag *whead = wfr + (size_t)h * (M / 16) * 2 * 64;
  auto load_wf = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      if constexpr (kLate) {
        const auto rs = buf_rsrc(whead, (M / 16) * 2 * 64 * 16);
        const int again = opaque_uniform(0);
        wf[mb][0] = buf_load16(rs, ((w * MB + mb) * 2 * 64 + l) * 16, again);
        wf[mb][1] = buf_load16(rs, ((w * MB + mb) * 2 * 64 + 64 + l) * 16, again);
      } else {
        wf[mb][0] = whead[(w * MB + mb) * 2 * 64 + l];
        wf[mb][1] = whead[(w * MB + mb) * 2 * 64 + 64 + l];
      }
    }
  };
  load_wf();
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int mbg = w * MB + mb;
    const float *bb = bqg + (size_t)h * M + 16 * mbg;
    if constexpr (!kLate) {
      bk[mb] = bb[c16];
#pragma unroll
      for (int j = 0; j < 4; ++j) bqv[mb][j] = bb[4 * g + j];
    }
  }
  if (kLate && tid < M) sm.bq[tid] = bqg[(size_t)h * M + tid];
  // b'' of feature rows w MW + 16 mb + 4 g .. + 3 (the query projections'
  // seeds) and of feature w MW + 16 mb + c16 (the key projections')
  auto qseed = [&](int mb) __attribute__((always_inline)) {
    if constexpr (kLate)
      return *reinterpret_cast<const f32x4 *>(&sm.bq[w * MW + 16 * mb + 4 * g]);
    else
      return bqv[mb];
  };
  auto kseed = [&](int mb) __attribute__((always_inline)) {
    if constexpr (kLate)
      return sm.bq[w * MW + 16 * mb + c16];
    else
      return bk[mb];
  };

  // state rows m = w MW + 16 mb + 4 g + j, lane column c16 of block nb holding
  // value column pi(nb, c16) (block 4: the ones column in all 16 columns)
  f32x4 accS[MB][5];
  {
    const float *pre = prefix + ((size_t)bh * nseg + seg) * M * 65;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int m = w * MW + mb * 16 + 4 * g + j;
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) accS[mb][nb][j] = pre[m * 65 + perm_col(nb, c16)];
        accS[mb][4][j] = pre[m * 65 + 64];
      }
  }

  // selection fragments of the value transposes (T = 32: read from LDS at
  // each staging after the first)
  const bf16x8 sel0[2] = {select_perm_frag(0), select_perm_frag(1)};
  if (kLate && w == 0) {
    sm.sel[0][l] = sel0[0];
    sm.sel[1][l] = sel0[1];
  }
  stage_causal_tile<T, KN, RN>(sm.tile[0], rg, rq, sel0, r0, r1, s2half, cM, eps);
  if (r0 + T < r1) {
    load_causal_tile_regs<T>(rg, Kh, Vh, r0 + T, r1, tid);
    load_q_rows<T>(rq, Qh, r0 + T, r1);
  }
  __syncthreads();

  // this wave's output unit of the previous chunk: sum the four partials (its
  // own and three handed over in buffer xb), normalise, store
  f32x4 own[5];   // value blocks 0 .. NVB - 1 of the unit; [4]: the denominator
  float own_epsq = 0.f;
  auto finalize = [&](int tp, int xb) __attribute__((always_inline)) {
    f32x4 part[3][NVB];   // the other waves' partials, all loads issued together
    float pden[3];
#pragma unroll
    for (int k = 1; k < 4; ++k) {
      const int src = (w + k) & 3;         // source wave
      const int slot = (w - src - 1) & 3;  // its slot for this wave's unit
#pragma unroll
      for (int nb = 0; nb < NVB; ++nb) part[k - 1][nb] = sm.num[xb][src][slot][nb][l];
      pden[k - 1] = sm.den[xb][src][slot][c16];
    }
    f32x4 num[NVB];
#pragma unroll
    for (int nb = 0; nb < NVB; ++nb) num[nb] = own[nb] + (part[0][nb] + part[1][nb] + part[2][nb]);
    const float den = own[4][0] + (pden[0] + pden[1] + pden[2]);
    const int qt = tp + 16 * utb + c16;
    if (qt < r1) {
      const float inv = RN ? 1.0f / (den + own_epsq) : own_epsq;
#pragma unroll
      for (int pp = 0; pp < NVB / 2; ++pp)
        if constexpr (kLate)
          buf_store8(buf_rsrc(Oh + (size_t)tp * kD, T * kD * sizeof(To)),
                     ((16 * utb + c16) * kD + 32 * (uvh * (NVB / 2) + pp) + 8 * g) * sizeof(To),
                     Oh, num[2 * pp] * inv, num[2 * pp + 1] * inv);
        else
          store8(Oh + (size_t)qt * kD + 32 * (uvh * (NVB / 2) + pp) + 8 * g, num[2 * pp] * inv,
               num[2 * pp + 1] * inv);
      if constexpr (SAVE) {
        if (g == 0 && uvh == 0) rsave[(size_t)bh * L + qt] = inv;
      }
    }
  };

  // Chunk c: stage tile c + 1 (its loads were issued during chunk c - 1) and
  // load tile c + 2; form the features of chunk c; finalise chunk c - 1 (its
  // partials were handed over before the last barrier); the contractions of
  // chunk c; hand its partials over; barrier. The vector and LDS work of
  // staging and finalising overlaps the matrix work of the chunk.
  int buf = 0;
  for (int t0 = r0; t0 < r1; t0 += T, buf ^= 1) {
    const CausalFsTile<T> &tl = sm.tile[buf];
    float my_epsq;
    if constexpr (KN == kCos)
      my_epsq = (!RN || eps != 0.f) ? tl.epsq[16 * utb + c16] : 0.f;
    else
      my_epsq = RN ? eps : 1.f;
    if constexpr (kLate) {
      if (t0 > r0) finalize(t0 - T, buf ^ 1);
    } else if (t0 + T < r1) {
      stage_causal_tile<T, KN, RN>(sm.tile[buf ^ 1], rg, rq, sel0, t0 + T, r1, s2half, cM, eps);
      if (t0 + 2 * T < r1) {
        load_causal_tile_regs<T>(rg, Kh, Vh, t0 + 2 * T, r1, tid);
        load_q_rows<T>(rq, Qh, t0 + 2 * T, r1);
      }
    }

    // features of this wave's slice for the chunk's queries and keys: eight
    // projection groups (query blocks tb, then key blocks tb), software-pipelined so
    // that the matrix cores project group i + 1 while the vector unit takes the
    // cosines of group i.
    //   qB[tb][ks]  B operand: col = query 16 tb + c16, k = 32 features (chained)
    //   kA[mb][s]   A operand: lane row = feature 16 mb + c16, k = keys 32 s .. (chained)
    frag qB[NTB][KS];
    frag kA[MB][NKH];
    {
      auto load_rows = [&](auto ic, frag (&r)[2]) __attribute__((always_inline)) {
        constexpr int i = decltype(ic)::value;
        const auto &src = (i < NTB) ? tl.Qs : tl.Ks;
        r[0] = load_frag<bf16>(&src[16 * (i % NTB) + c16][8 * g]);
        r[1] = load_frag<bf16>(&src[16 * (i % NTB) + c16][32 + 8 * g]);
      };
      auto project = [&](auto ic, const frag (&r)[2], f32x4 (&pr)[MB]) __attribute__((always_inline)) {
        constexpr int i = decltype(ic)::value;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          if constexpr (i < NTB) {   // C[m][t] = W'' q_t + b''
            pr[mb] = P::mma(wf[mb][0], r[0], qseed(mb));
            pr[mb] = P::mma(wf[mb][1], r[1], pr[mb]);
          } else {                 // C[t][m] = W'' k_t + b''
            const float bb = kseed(mb);
            pr[mb] = P::mma(r[0], wf[mb][0], f32x4{bb, bb, bb, bb});
            pr[mb] = P::mma(r[1], wf[mb][1], pr[mb]);
          }
        }
      };
      f32x4 kfh[MB];   // cosines of the first key block of a pair
      auto finish = [&](auto ic, f32x4 (&pr)[MB]) __attribute__((always_inline)) {
        constexpr int i = decltype(ic)::value;
        constexpr int tb = i % NTB;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          f32x4 sd;
          if constexpr (i < NTB)
            sd = qseed(mb);
          else
            sd = f32x4{kseed(mb), kseed(mb), kseed(mb), kseed(mb)};
#pragma unroll
          for (int j = 0; j < 4; ++j) pr[mb][j] = feature<KN, P>(pr[mb][j], sd[j]);
        }
        if constexpr (i < NTB) {
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            qB[tb][ks] = P::pack(pr[2 * ks], (2 * ks + 1 < MB) ? pr[2 * ks + 1] : zero4);
        } else if constexpr ((tb & 1) == 0) {
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) kfh[mb] = pr[mb];
        } else {
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) kA[mb][tb >> 1] = P::pack(kfh[mb], pr[mb]);
        }
      };
      frag rows0[2], rows1[2];
      f32x4 pr0[MB], pr1[MB];
      load_rows(std::integral_constant<int, 0>{}, rows0);
      load_rows(std::integral_constant<int, 1>{}, rows1);
      project(std::integral_constant<int, 0>{}, rows0, pr0);
      static_for<1, 2 * NTB>([&](auto ic) __attribute__((always_inline)) {
        constexpr int i = decltype(ic)::value;
        auto &rn = (i & 1) ? rows0 : rows1;   // the buffer of group i + 1
        auto &rc = (i & 1) ? rows1 : rows0;
        auto &pc = (i & 1) ? pr1 : pr0;
        auto &pp = (i & 1) ? pr0 : pr1;
        if constexpr (i + 1 < 2 * NTB) load_rows(std::integral_constant<int, i + 1>{}, rn);
        project(ic, rc, pc);
        finish(std::integral_constant<int, i - 1>{}, pp);
        // the next group's rows first, then each projection MFMA followed by
        // three vector instructions of the previous group's epilogue, so that
        // the cosines issue while the matrix core works
        if constexpr (i + 1 < 2 * NTB) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        static_for<0, 2 * MB>([&](auto) __attribute__((always_inline)) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
        });
        __builtin_amdgcn_sched_barrier(0);
      });
      finish(std::integral_constant<int, 2 * NTB - 1>{}, pr1);
      // the features are complete here: keeps the compiler from sinking the
      // cosines past the finalisation branch, away from the projection MFMAs
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+v"(qB[tb][ks]));
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int sx = 0; sx < NKH; ++sx) asm volatile("" : "+v"(kA[mb][sx]));
    }

    if constexpr (kLate) {
      if (t0 + T < r1) {
        const bf16x8 sel[2] = {sm.sel[0][l], sm.sel[1][l]};
        stage_causal_tile<T, KN, RN>(sm.tile[buf ^ 1], rg, rq, sel, t0 + T, r1, s2half, cM, eps);
      }
    } else if (t0 > r0) {
      finalize(t0 - T, buf ^ 1);
    }

    if constexpr (kStream) {
      // the chunk's key features, one 32-token half at a time, transposed to
      // token rows on the matrix cores; then the masked P^T[t'][t] = K-hat_t' .
      // Q-hat_t over the slice for each (key half, query block) with keys up
      // to the query (the keys after it zeroed)
      frag pb[NKH][NTB];   // [half][query block]: used for tb >= 2 half
#pragma unroll
      for (int sidx = 0; sidx < NKH; ++sidx) {
        frag kT[2][KS];   // A operand: lane row = token 32 sidx + 16 tbl + c16, k = 32 features
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          f32x4 ct[2][2];
#pragma unroll
          for (int hm = 0; hm < 2; ++hm)
#pragma unroll
            for (int tbl = 0; tbl < 2; ++tbl)
              ct[tbl][hm] = (2 * ks + hm < MB)
                                ? P::mma(kA[2 * ks + hm][sidx], chained_select_frag<bf16>(tbl), zero4)
                                : zero4;
#pragma unroll
          for (int tbl = 0; tbl < 2; ++tbl) kT[tbl][ks] = P::pack(ct[tbl][0], ct[tbl][1]);
        }
#pragma unroll
        for (int tb = 2 * sidx; tb < NTB; ++tb) {
          f32x4 pt[2];
#pragma unroll
          for (int tbl = 0; tbl < 2; ++tbl) {
            const int tp = 2 * sidx + tbl;
            if (tp > tb) {
              pt[tbl] = zero4;
              continue;
            }
            pt[tbl] = P::mma(kT[tbl][0], qB[tb][0], zero4);
#pragma unroll
            for (int ks = 1; ks < KS; ++ks) pt[tbl] = P::mma(kT[tbl][ks], qB[tb][ks], pt[tbl]);
            if (tp == tb) {
#pragma unroll
              for (int j = 0; j < 4; ++j) pt[tbl][j] = (4 * g + j <= c16) ? pt[tbl][j] : 0.f;
            }
          }
          pb[sidx][tb] = P::pack(pt[0], pt[1]);
        }
      }
      // one value block at a time (the ones column last): Q-hat S with the
      // state before the chunk, plus C~^T P^T of each key half, handed over (or
      // kept when it is this wave's unit u: token block u % NTB, value blocks
      // NVB (u / NTB) ..); then the chunk's keys are folded into that block of S
      const int wu = __builtin_amdgcn_readfirstlane(w);
#pragma unroll
      for (int nb = 0; nb < 5; ++nb) {
        frag sA[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          sA[ks] = P::pack(accS[2 * ks][nb], (2 * ks + 1 < MB) ? accS[2 * ks + 1][nb] : zero4);
        frag vt[NKH];
#pragma unroll
        for (int sidx = 0; sidx < NKH; ++sidx) vt[sidx] = nb < 4 ? tl.VtF[nb][sidx][l] : tl.DF[sidx][g];
#pragma unroll
        for (int tb = 0; tb < NTB; ++tb) {
          f32x4 on = P::mma(sA[0], qB[tb][0], zero4);
#pragma unroll
          for (int ks = 1; ks < KS; ++ks) on = P::mma(sA[ks], qB[tb][ks], on);
#pragma unroll
          for (int sidx = 0; sidx < NKH; ++sidx)
            if (2 * sidx <= tb) on = P::mma(vt[sidx], pb[sidx][tb], on);
          if (nb < 4) {
            const int u = tb + NTB * (nb / NVB);
            if (u == wu)
              own[nb % NVB] = on;
            else
              sm.num[buf][w][(u - w - 1) & 3][nb % NVB][l] = on;
          } else {
#pragma unroll
            for (int u = tb; u < 4; u += NTB) {
              if (u == wu)
                own[4] = on;
              else if (g == 0)
                sm.den[buf][w][(u - w - 1) & 3][c16] = on[0];
            }
          }
        }
#pragma unroll
        for (int sidx = 0; sidx < NKH; ++sidx)
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) accS[mb][nb] = P::mma(kA[mb][sidx], vt[sidx], accS[mb][nb]);
      }
      own_epsq = my_epsq;
      if constexpr (kLate) {
        if (t0 + 2 * T < r1) {
          load_causal_tile_regs<T>(rg, Kh, Vh, t0 + 2 * T, r1, tid);
          load_q_rows<T>(rq, Qh, t0 + 2 * T, r1);
        }
        if (t0 + T < r1) load_wf();
      }

    } else {
      // partial Buf2 (value columns and the denominator) over this slice: o[nb][tb]
      // holds rows pi(nb, 4 g + j), column = token 16 tb + c16; first Q-hat S with
      // the state before the chunk
      f32x4 o[5][NTB];
#pragma unroll
      for (int nb = 0; nb < 5; ++nb) {
        frag sA[KS];   // lane row = value column, k = m
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          sA[ks] = P::pack(accS[2 * ks][nb], (2 * ks + 1 < MB) ? accS[2 * ks + 1][nb] : zero4);
#pragma unroll
        for (int tb = 0; tb < NTB; ++tb) {
          o[nb][tb] = P::mma(sA[0], qB[tb][0], zero4);
#pragma unroll
          for (int ks = 1; ks < KS; ++ks) o[nb][tb] = P::mma(sA[ks], qB[tb][ks], o[nb][tb]);
        }
      }

      // keys, one 32-token half at a time: fold into S (after the queries above
      // used it), transpose to token rows on the matrix cores, then the
      // intra-chunk part of that half: P^T[t'][t] = K-hat_t' . Q-hat_t over the
      // slice for key blocks tb' <= tb (keys after the query zeroed) and C~^T P^T
      // into o
#pragma unroll
      for (int sidx = 0; sidx < NKH; ++sidx) {
        // C~ of the half: B operand of the state update and A operand of the
        // intra-chunk product (lane = value column, k = token in chained order)
        frag vt[4];
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) vt[nb] = tl.VtF[nb][sidx][l];
        const frag df = tl.DF[sidx][g];
        frag kT[2][KS];   // A operand: lane row = token 32 sidx + 16 tbl + c16, k = 32 features
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          f32x4 ct[2][2];
#pragma unroll
          for (int hm = 0; hm < 2; ++hm) {
            const int mb = 2 * ks + hm;
            if (mb >= MB) {
              ct[0][hm] = zero4;
              ct[1][hm] = zero4;
              continue;
            }
            const frag a = kA[mb][sidx];
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) accS[mb][nb] = P::mma(a, vt[nb], accS[mb][nb]);
            accS[mb][4] = P::mma(a, df, accS[mb][4]);
#pragma unroll
            for (int tbl = 0; tbl < 2; ++tbl)
              ct[tbl][hm] = P::mma(a, chained_select_frag<bf16>(tbl), zero4);
          }
#pragma unroll
          for (int tbl = 0; tbl < 2; ++tbl) kT[tbl][ks] = P::pack(ct[tbl][0], ct[tbl][1]);
        }
#pragma unroll
        for (int tb = 2 * sidx; tb < NTB; ++tb) {
          f32x4 pt[2];
#pragma unroll
          for (int tbl = 0; tbl < 2; ++tbl) {
            const int tp = 2 * sidx + tbl;
            if (tp > tb) {
              pt[tbl] = zero4;
              continue;
            }
            pt[tbl] = P::mma(kT[tbl][0], qB[tb][0], zero4);
#pragma unroll
            for (int ks = 1; ks < KS; ++ks) pt[tbl] = P::mma(kT[tbl][ks], qB[tb][ks], pt[tbl]);
            if (tp == tb) {
#pragma unroll
              for (int j = 0; j < 4; ++j) pt[tbl][j] = (4 * g + j <= c16) ? pt[tbl][j] : 0.f;
            }
          }
          const frag pb = P::pack(pt[0], pt[1]);
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) o[nb][tb] = P::mma(vt[nb], pb, o[nb][tb]);
          o[4][tb] = P::mma(df, pb, o[4][tb]);
        }
      }

      // hand the partials of the other waves' units over; keep this wave's own
      // (unit u: token block u % NTB, value blocks NVB (u / NTB) ..)
      if constexpr (T == 64) {
#pragma unroll
        for (int nb = 0; nb < 5; ++nb)
          own[nb] = (w == 0) ? o[nb][0] : (w == 1) ? o[nb][1] : (w == 2) ? o[nb][2] : o[nb][3];
      } else {
#pragma unroll
        for (int k = 0; k < NVB; ++k)
          own[k] = (w == 0) ? o[k][0] : (w == 1) ? o[k][1] : (w == 2) ? o[NVB + k][0] : o[NVB + k][1];
        own[4] = (w & 1) ? o[4][1] : o[4][0];
      }
      own_epsq = my_epsq;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (u != w) {
          const int slot = (u - w - 1) & 3;
#pragma unroll
          for (int k = 0; k < NVB; ++k) sm.num[buf][w][slot][k][l] = o[NVB * (u / NTB) + k][u % NTB];
          if (g == 0) sm.den[buf][w][slot][c16] = o[4][u % NTB][0];
        }
      }
    }
    __syncthreads();
  }
  // the last chunk
  if (r1 > r0) finalize(r0 + T * ((r1 - r0 - 1) / T), buf ^ 1);
}

hipError_t launch_seg_scan(const Shape &sh, Dt in, float *part, int nseg, const float *state_in,
                           float *state_out, void *total_frags, hipStream_t st, float *total) {
  dim3 grid(sh.M / 32, sh.BH);
  if (in == Dt::BF16)
    hipLaunchKernelGGL(k_seg_scan<bf16>, grid, dim3(kSegScanThreads), 0, st, part, nseg, sh.M,
                       sh.Mr, state_in, state_out, (bf16 *)total_frags, total);
  else
    hipLaunchKernelGGL(k_seg_scan<float>, grid, dim3(kSegScanThreads), 0, st, part, nseg, sh.M,
                       sh.Mr, state_in, state_out, (float *)total_frags, total);
  return hipGetLastError();
}

// Calls f(integral_constant<int, KN>, bool_constant<RN>) for the shape's
// feature kernel and renormalisation.
template <typename F>
static hipError_t with_variant(const Shape &sh, F &&f) {
  using relu = std::integral_constant<int, kRelu>;
  using cosk = std::integral_constant<int, kCos>;
  if (sh.kernel == 1) return sh.renorm ? f(relu{}, std::true_type{}) : f(relu{}, std::false_type{});
  return sh.renorm ? f(cosk{}, std::true_type{}) : f(cosk{}, std::false_type{});
}

template <typename To, bool SAVE = false>
static hipError_t causal_fs_typed(const Shape &sh, const void *Q, const void *K, const void *V,
                                  const void *wfr, const float *bq, const float *prefix, void *o,
                                  int seg_len, int nseg, hipStream_t st, float *rsave = nullptr) {
  dim3 grid(nseg * sh.BH);
  return with_variant(sh, [&](auto kn, auto rn) -> hipError_t {
    constexpr int KN = decltype(kn)::value;
    constexpr bool RN = decltype(rn)::value;
    if constexpr (SAVE && !RN) {
      return hipErrorInvalidValue;
    } else {
#define FAVOR_CAUSAL_FS_LAUNCH(MM, TT)                                                      \
  hipLaunchKernelGGL((k_causal_fs<To, MM, KN, RN, SAVE, TT>), grid, dim3(256), 0, st,         \
                     (const bf16 *)Q, (const bf16 *)K, (const bf16 *)V, (const bf16x8 *)wfr,   \
                     bq, prefix, (To *)o, rsave, sh.H, sh.L, seg_len, nseg, sh.s, sh.eps,      \
                     feature_norm(sh))
#define FAVOR_CAUSAL_FS_M(TT)                                                                \
  switch (sh.M) {                                                                           \
    case 64: FAVOR_CAUSAL_FS_LAUNCH(64, TT); break;                                          \
    case 128: FAVOR_CAUSAL_FS_LAUNCH(128, TT); break;                                        \
    case 256: FAVOR_CAUSAL_FS_LAUNCH(256, TT); break;                                        \
    default: return hipErrorInvalidValue;                                                   \
  }
      if (sh.chunk == 32) {
        FAVOR_CAUSAL_FS_M(32)
      } else if (sh.chunk == 64) {
        FAVOR_CAUSAL_FS_M(64)
      } else {
        return hipErrorInvalidValue;
      }
#undef FAVOR_CAUSAL_FS_M
#undef FAVOR_CAUSAL_FS_LAUNCH
      return hipGetLastError();
    }
  });
}

// fp32 inputs: M <= 128 in one pass, M = 256 in two passes over the feature
// halves (the raw partials of the first in halves [BH][L][kHalfRow]).
template <typename T, typename To, bool SAVE = false>
static hipError_t causal_typed(const Shape &sh, const void *Q, const void *K, const void *V,
                               const void *wfr, const float *bq, const float *prefix, void *o,
                               int seg_len, int nseg, hipStream_t st, float *halves,
                               float *rsave = nullptr) {
  if (sh.chunk != 64) return hipErrorInvalidValue;   // 64-token chunks only
  dim3 grid(nseg * sh.BH);
  return with_variant(sh, [&](auto kn, auto rn) -> hipError_t {
    constexpr int KN = decltype(kn)::value;
    constexpr bool RN = decltype(rn)::value;
    if constexpr (SAVE && !RN) {
      return hipErrorInvalidValue;
    } else {
#define FAVOR_CAUSAL_LAUNCH(MM, PART, M0)                                                   \
  hipLaunchKernelGGL((k_causal<T, To, MM, KN, RN, SAVE, PART>), grid, dim3(256), 0, st,       \
                     (const T *)Q, (const T *)K, (const T *)V,                                 \
                     (const typename Mma<T>::frag *)wfr, bq, prefix, (To *)o, rsave, halves,   \
                     sh.H, sh.L, seg_len, nseg, sh.s, sh.eps, feature_norm(sh), sh.M, M0)
      switch (sh.M) {
        case 64: FAVOR_CAUSAL_LAUNCH(64, 0, 0); break;
        case 128: FAVOR_CAUSAL_LAUNCH(128, 0, 0); break;
        case 256:
          if (!halves) return hipErrorInvalidValue;
          FAVOR_CAUSAL_LAUNCH(128, 1, 0);
          FAVOR_CAUSAL_LAUNCH(128, 2, 128);
          break;
        default: return hipErrorInvalidValue;
      }
#undef FAVOR_CAUSAL_LAUNCH
      return hipGetLastError();
    }
  });
}

hipError_t launch_causal_save(const Shape &sh, Dt in, const void *Q, const void *K,
                              const void *V, const void *wfr, const float *bq,
                              const float *prefix, void *o, float *rsave, int seg_len, int nseg,
                              float *halves, hipStream_t st) {
  if (!sh.renorm) return hipErrorInvalidValue;
  if (in == Dt::BF16)
    return causal_fs_typed<bf16, true>(sh, Q, K, V, wfr, bq, prefix, o, seg_len, nseg, st, rsave);
  return causal_typed<float, float, true>(sh, Q, K, V, wfr, bq, prefix, o, seg_len, nseg, st,
                                          halves, rsave);
}

hipError_t launch_causal(const Shape &sh, Dt in, Dt out, const void *Q, const void *K,
                         const void *V, const void *wfr, const float *bq, const float *prefix,
                         void *o, int seg_len, int nseg, float *halves, hipStream_t st) {
  if (in == Dt::BF16)
    return out == Dt::BF16
               ? causal_fs_typed<bf16>(sh, Q, K, V, wfr, bq, prefix, o, seg_len, nseg, st)
               : causal_fs_typed<float>(sh, Q, K, V, wfr, bq, prefix, o, seg_len, nseg, st);
  return out == Dt::BF16 ? causal_typed<float, bf16>(sh, Q, K, V, wfr, bq, prefix, o, seg_len,
                                                     nseg, st, halves)
                         : causal_typed<float, float>(sh, Q, K, V, wfr, bq, prefix, o, seg_len,
                                                      nseg, st, halves);
}

}  // namespace favor
