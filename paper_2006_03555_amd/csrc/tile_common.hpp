// tile_common.hpp - pieces shared by the kernels that stream 64-token tiles.
//
// A 64-token tile of keys and values is staged in LDS by 256 threads:
//   Ks[64][72]     keys, row-major (A operand of the key projection, loaded order)
//   VtF[4][2][64]  C~ = D_K [V 1] without its ones column, stored as B-operand
//                  fragments of the value matrix [t x n] in chained token order
//                  (block nb of 16 value columns, token half s of the tile)
//   DF[2][4]       D_K in chained token order (the ones column of C~, scaled)
// with D_K(t) = sqrt(2/M) exp(||s k_t||^2 / 2) for rows inside the range and 0
// for rows past its end, so padded rows contribute nothing. Tiles are loaded
// into registers one tile ahead (load_tile_regs) and staged (stage_tile) into
// the other half of a double buffer, so one barrier per tile suffices.
#pragma once

#include "favor_common.hpp"

namespace favor {

constexpr int kD = 64;     // head dimension supported by the kernels
constexpr int kKsPad = 8;  // row padding of the staged key tile (elements)

template <typename T>
struct KVTile {
  using frag = typename Mma<T>::frag;
  T Ks[64][kD + kKsPad];
  frag VtF[4][2][64];
  frag DF[2][4];
};

// Global loads of one 64-token tile, held in registers until staged:
//   k[2]  keys of row tid / 4, columns 16 (tid % 4) .. + 16 (for Ks and D_K)
//   v[2]  values of row 16 w + (lane % 16) as A-operand fragments over the 64
//         value columns (loaded order: lane group g holds columns 8 g + 32 kh ..)
template <typename T>
struct TileRegs {
  typename Mma<T>::frag k[2];
  typename Mma<T>::frag v[2];
};

template <typename T>
__device__ __forceinline__ void load_tile_regs(TileRegs<T> &r, const T *__restrict__ Kh,
                                               const T *__restrict__ Vh, int t0, int r1,
                                               int tid) {
  const int l = tid & 63;
  const int rk = t0 + (tid >> 2);
  const int rv = t0 + 16 * (tid >> 6) + (l & 15);
  if (rk < r1) {
    const T *kp = Kh + (size_t)rk * kD + (tid & 3) * 16;
    r.k[0] = load_frag<T>(kp);
    r.k[1] = load_frag<T>(kp + 8);
  } else {
    r.k[0] = Mma<T>::splat(0.f);
    r.k[1] = Mma<T>::splat(0.f);
  }
  if (rv < r1) {
    const T *vp = Vh + (size_t)rv * kD + 8 * (l >> 4);
    r.v[0] = load_frag<T>(vp);
    r.v[1] = load_frag<T>(vp + 32);
  } else {
    r.v[0] = Mma<T>::splat(0.f);
    r.v[1] = Mma<T>::splat(0.f);
  }
}

// Selection matrix [32 k x 16 cols] with B[k][c] = (k == 16 half + c), as a
// B-operand fragment in loaded order: multiplying an A fragment by it moves
// value column 16 half + c of row t into lane c, rows 4 g + j (an exact
// transpose on the matrix cores; every output is 1 * v).
template <typename T>
__device__ __forceinline__ typename Mma<T>::frag select_frag(int half) {
  const int l = lane_id();
  float v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (8 * (l >> 4) + i == 16 * half + (l & 15)) ? 1.f : 0.f;
  return Mma<T>::from_f32(v, 1.f);
}

// Selection matrix in chained k order: slot i of lane group g stands for token
// 16 (i / 4) + 4 g + i % 4 of a 32-token k-step; B[k][c] = (token == 16 tbl + c).
// An MFMA of a chained K-hat^T fragment (rows = features) with it returns the
// 16 tokens of block tbl in lanes, 4 consecutive features per lane.
template <typename T>
__device__ __forceinline__ typename Mma<T>::frag chained_select_frag(int tbl) {
  const int l = lane_id();
  float v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
    v[i] = (16 * (i >> 2) + 4 * (l >> 4) + (i & 3) == 16 * tbl + (l & 15)) ? 1.f : 0.f;
  return Mma<T>::from_f32(v, 1.f);
}

// Query fragments of row t (B operand of the transposed projection): lane
// group g holds columns 8 g .. and 32 + 8 g .. ; zero past r1.
template <typename T>
__device__ __forceinline__ void load_query_frags(typename Mma<T>::frag (&qf)[2],
                                                 const T *__restrict__ Qh, int t, int r1) {
  const int g = lane_id() >> 4;
  if (t < r1) {
    qf[0] = load_frag<T>(Qh + (size_t)t * kD + 8 * g);
    qf[1] = load_frag<T>(Qh + (size_t)t * kD + 32 + 8 * g);
  } else {
    qf[0] = Mma<T>::splat(0.f);
    qf[1] = Mma<T>::splat(0.f);
  }
}

// Stage a prefetched tile into LDS: keys row-major, the value rows scaled by
// this thread's row weight a (row tid / 4) as chained-order B fragments, and
// the extra column e in place of the ones column. Wave w transposes the values
// of its 16 tokens 16 w .. 16 w + 15.
template <typename T>
__device__ __forceinline__ void stage_tile_rows(KVTile<T> &tl, const TileRegs<T> &r,
                                                const typename Mma<T>::frag (&sel)[2], float a,
                                                float e, int tid) {
  using P = Mma<T>;
  const int w = tid >> 6;
  const int l = tid & 63;
  const int g = l >> 4;
  const int c16 = l & 15;
  const int tr = tid >> 2;
  const int cq = (tid & 3) * 16;
  store_frag<T>(&tl.Ks[tr][cq], r.k[0]);
  store_frag<T>(&tl.Ks[tr][cq + 8], r.k[1]);
  // weights of rows 16 w + 4 g + j, held by lanes 16 g + 4 j of this wave
  float aj[4], ej[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    aj[j] = __shfl(a, 16 * g + 4 * j);
    ej[j] = __shfl(e, 16 * g + 4 * j);
  }
  const int sidx = w >> 1;
  const int h = w & 1;
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const f32x4 c = P::mma(r.v[kh], sel[half], f32x4{0.f, 0.f, 0.f, 0.f});
      T *p = reinterpret_cast<T *>(&tl.VtF[2 * kh + half][sidx][l]) + 4 * h;
#pragma unroll
      for (int j = 0; j < 4; ++j) p[j] = from_f32<T>(c[j] * aj[j]);
    }
  if (c16 == 0) {
    T *p = reinterpret_cast<T *>(&tl.DF[sidx][g]) + 4 * h;
#pragma unroll
    for (int j = 0; j < 4; ++j) p[j] = from_f32<T>(ej[j]);
  }
}

// Stage a prefetched tile into LDS: keys row-major, D_K(t) = sqrt(2/M)
// exp(||s k_t||^2 / 2) (1 for ReLU features; 0 past r1), and C~ = D_K [V 1] as
// chained-order B fragments.
template <typename T, int KN>
__device__ __forceinline__ void stage_tile(KVTile<T> &tl, const TileRegs<T> &r,
                                           const typename Mma<T>::frag (&sel)[2], int t0, int r1,
                                           float s2half, float cM, int tid) {
  const int tr = tid >> 2;
  float Dt = (t0 + tr < r1) ? 1.f : 0.f;
  if constexpr (KN == kCos) {
    float nrm = sq_sum16(r.k);
    nrm += __shfl_xor(nrm, 1);
    nrm += __shfl_xor(nrm, 2);
    Dt = (t0 + tr < r1) ? cM * expf(s2half * nrm) : 0.f;
  }
  stage_tile_rows<T>(tl, r, sel, Dt, Dt, tid);
}

// Key projection + features for one wave's MB m-blocks over token half sidx of
// the staged tile: kf[mb][tbl][j] = feature(W'' k_t + b'') (bC: the seeds b'' of
// the lane's feature) for token t = 32 sidx + 16 tbl + 4 g + j and feature
// m = m0 + 16 mb + (lane % 16).
template <typename T, int MB, int KN>
__device__ __forceinline__ void key_features(const KVTile<T> &tl,
                                             const typename Mma<T>::frag (&Wf)[MB][2],
                                             const f32x4 (&bC)[MB], int sidx,
                                             f32x4 (&kf)[MB][2]) {
  using P = Mma<T>;
  const int l = lane_id();
  const int g = l >> 4;
  const int c16 = l & 15;
#pragma unroll
  for (int tbl = 0; tbl < 2; ++tbl) {
    const int tb = 2 * sidx + tbl;
    const auto a0 = load_frag<T>(&tl.Ks[tb * 16 + c16][8 * g]);
    const auto a1 = load_frag<T>(&tl.Ks[tb * 16 + c16][32 + 8 * g]);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      f32x4 p = P::mma(a0, Wf[mb][0], bC[mb]);
      p = P::mma(a1, Wf[mb][1], p);
#pragma unroll
      for (int j = 0; j < 4; ++j) kf[mb][tbl][j] = feature<KN, P>(p[j], bC[mb][j]);
    }
  }
}

// Key projection + features as key_features, with the B operand (W'' for this
// wave's feature blocks) read from the head's W'' fragments in LDS and the
// accumulator seeds b'' from LDS.
template <typename T, int MB, int KN>
__device__ __forceinline__ void key_features_lds(const KVTile<T> &tl,
                                                 const typename Mma<T>::frag (*WA)[2][64],
                                                 const float *bq, int mb0, int sidx,
                                                 f32x4 (&kf)[MB][2]) {
  using P = Mma<T>;
  const int l = lane_id();
  const int g = l >> 4;
  const int c16 = l & 15;
  typename P::frag wb[MB][2];
  f32x4 bC[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    wb[mb][0] = WA[mb0 + mb][0][l];
    wb[mb][1] = WA[mb0 + mb][1][l];
    const float bb = bq[(mb0 + mb) * 16 + c16];
    bC[mb] = f32x4{bb, bb, bb, bb};
  }
#pragma unroll
  for (int tbl = 0; tbl < 2; ++tbl) {
    const int tb = 2 * sidx + tbl;
    const auto a0 = load_frag<T>(&tl.Ks[tb * 16 + c16][8 * g]);
    const auto a1 = load_frag<T>(&tl.Ks[tb * 16 + c16][32 + 8 * g]);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      f32x4 p = P::mma(a0, wb[mb][0], bC[mb]);
      p = P::mma(a1, wb[mb][1], p);
#pragma unroll
      for (int j = 0; j < 4; ++j) kf[mb][tbl][j] = feature<KN, P>(p[j], bC[mb][j]);
    }
  }
}

// Copy n fragments global -> LDS with 256 threads, all loads issued first.
template <typename F, int N>
__device__ __forceinline__ void copy_frags(F *__restrict__ dst, const F *__restrict__ src) {
  constexpr int IT = (N + 255) / 256;
  F v[IT];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int idx = it * 256 + threadIdx.x;
    if (idx < N) v[it] = src[idx];
  }
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int idx = it * 256 + threadIdx.x;
    if (idx < N) dst[idx] = v[it];
  }
}

// Workgroups are dispatched round-robin over the 8 XCDs (ids congruent mod 8
// share an XCD and its L2). Map linear id -> work item so that each XCD gets
// a contiguous range of items (consecutive tiles of the same head share the
// head's W and Buf1 in that L2). A bijection on [0, n) for any n.
__device__ __forceinline__ int xcd_item(int id, int n) {
  const int per = n >> 3;
  const int rem = n & 7;
  const int x = id & 7;
  const int k = id >> 3;
  return x * per + min(x, rem) + k;
}

// Contiguous range of work items for workgroup `id` of `nwg`: the items of
// XCD x (ids congruent to x mod 8) form one contiguous block (xcd_item), split
// evenly over that XCD's workgroups, so a workgroup's items are consecutive
// tiles of mostly one head.
__device__ __forceinline__ void xcd_range(int id, int nwg, int n, int &begin, int &end) {
  const int x = id & 7;
  const int k = id >> 3;
  const int nw = (nwg >> 3) + (x < (nwg & 7) ? 1 : 0);
  const int cnt = (n >> 3) + (x < (n & 7) ? 1 : 0);
  const int base = x * (n >> 3) + min(x, n & 7);
  begin = base + (int)((long long)k * cnt / nw);
  end = base + (int)((long long)(k + 1) * cnt / nw);
}

}  // namespace favor
