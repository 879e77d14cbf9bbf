// tile_common.hpp - pieces shared by the kernels that stream 64-token tiles.
//
// A 64-token tile of keys and values is staged in LDS by 256 threads:
//   Ks[64][72]     keys, row-major (A operand of the key projection, loaded order)
//   VtF[4][2][64]  C~ = D_K [V 1] without its ones column, stored as B-operand
//                  fragments of the value matrix [t x n] in chained token order
//                  (block nb of 16 value columns, token half s of the tile)
//   DF[2][4]       D_K in chained token order (the ones column of C~, scaled)
// with D_K(t) = sqrt(2/M) exp(||s k_t||^2 / 2) for rows inside the range and 0
// for rows past its end, so padded rows contribute nothing.
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

// Stage rows [t0, t0 + 64) of one head's K and V (row limit r1) into LDS.
// Thread tid handles row tid / 4, columns 16 (tid % 4) .. + 16.
template <typename T>
__device__ __forceinline__ void stage_kv_tile(KVTile<T> &tl, const T *__restrict__ Kh,
                                              const T *__restrict__ Vh, int t0, int r1,
                                              float s2half, float cM) {
  const int tid = threadIdx.x;
  const int tr = tid >> 2;
  const int cq = (tid & 3) * 16;
  const int row = t0 + tr;
  float kv[16], vv[16];
  if (row < r1) {
    const T *kp = Kh + (size_t)row * kD + cq;
    const T *vp = Vh + (size_t)row * kD + cq;
    load8_f32(kp, kv);
    load8_f32(kp + 8, kv + 8);
    load8_f32(vp, vv);
    load8_f32(vp + 8, vv + 8);
  } else {
#pragma unroll
    for (int k = 0; k < 16; ++k) { kv[k] = 0.f; vv[k] = 0.f; }
  }
  float nrm = 0.f;
#pragma unroll
  for (int k = 0; k < 16; ++k) nrm = fmaf(kv[k], kv[k], nrm);
  nrm += __shfl_xor(nrm, 1);
  nrm += __shfl_xor(nrm, 2);
  const float Dt = (row < r1) ? cM * expf(s2half * nrm) : 0.f;
  store_frag<T>(&tl.Ks[tr][cq], Mma<T>::from_f32(kv, 1.f));
  store_frag<T>(&tl.Ks[tr][cq + 8], Mma<T>::from_f32(kv + 8, 1.f));
  const int sidx = tr >> 5;
  const int r = tr & 31;
  const int gg = chained_group(r);
  const int sl = chained_slot(r);
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int n = cq + k;
    T *p = reinterpret_cast<T *>(&tl.VtF[n >> 4][sidx][(n & 15) + 16 * gg]);
    p[sl] = from_f32<T>(vv[k] * Dt);
  }
  if ((tid & 3) == 0) reinterpret_cast<T *>(&tl.DF[sidx][gg])[sl] = from_f32<T>(Dt);
}

// Key projection + features for one wave's MB m-blocks over token half sidx of
// the staged tile: kf[mb][tbl][j] = cos(2 pi (W'' k_t + b'')) for token
// t = 32 sidx + 16 tbl + 4 g + j and feature m = m0 + 16 mb + (lane % 16).
template <typename T, int MB>
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
      for (int j = 0; j < 4; ++j) kf[mb][tbl][j] = P::cos_rev(p[j]);
    }
  }
}

// Load W'' = (s / 2 pi) W as B-operand fragments (lane col m, loaded d order)
// and b'' = b / 2 pi as accumulator seeds for m = m0 + 16 mb + lane % 16.
template <typename T, int MB>
__device__ __forceinline__ void load_w_bfrags(const float *__restrict__ Wh,
                                              const float *__restrict__ bh, int m0, float ws,
                                              typename Mma<T>::frag (&Wf)[MB][2],
                                              f32x4 (&bC)[MB]) {
  const int l = lane_id();
  const int g = l >> 4;
  const int c16 = l & 15;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int m = m0 + mb * 16 + c16;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      float v[8];
      load8_f32(Wh + (size_t)m * kD + ks * 32 + 8 * g, v);
      Wf[mb][ks] = Mma<T>::from_f32(v, ws);
    }
    const float bb = bh[m] * kInv2Pi;
    bC[mb] = f32x4{bb, bb, bb, bb};
  }
}

// Fill W'' A-operand fragments (lane row m, loaded d order) for all M rows and
// b'' into LDS, cooperatively.
template <typename T, int M>
__device__ __forceinline__ void fill_w_afrags(typename Mma<T>::frag (*WA)[2][64], float *bq,
                                              const float *__restrict__ Wh,
                                              const float *__restrict__ bh, float ws) {
  for (int idx = threadIdx.x; idx < (M / 16) * 2 * 64; idx += blockDim.x) {
    const int mb = idx >> 7;
    const int ks = (idx >> 6) & 1;
    const int ll = idx & 63;
    const int m = mb * 16 + (ll & 15);
    float v[8];
    load8_f32(Wh + (size_t)m * kD + ks * 32 + 8 * (ll >> 4), v);
    WA[mb][ks][ll] = Mma<T>::from_f32(v, ws);
  }
  for (int idx = threadIdx.x; idx < M; idx += blockDim.x) bq[idx] = bh[idx] * kInv2Pi;
}

}  // namespace favor
