// kernels.hpp - host-side launchers of the FAVOR kernels (internal to libfavor).
#pragma once

#include <cmath>

#include <hip/hip_runtime.h>

#include "../../include/favor.h"
#include <stddef.h>
#include <stdint.h>

namespace favor {

enum class Dt { F32 = 0, BF16 = 1 };

// Bytes of one k32 operand fragment for element type dt (8 elements).
inline int frag_bytes(Dt dt) { return dt == Dt::BF16 ? 16 : 32; }

// Shape and scalars of one call; pointers are device pointers.
struct Shape {
  int BH;        // B * H
  int H;         // heads (W and b are per head)
  int L;
  int M;         // rows the kernels work on: 64, 128 or 256 (M_r rounded up)
  int Mr;        // features drawn (a multiple of 16); rows M_r .. M - 1 are padding
  float s;       // input scale
  float eps;     // denominator stabiliser
  int kernel;    // 0 Gaussian-kernel (cos) features, 1 ReLU features
  int renorm;    // 1 divide by D-hat, 0 return the numerator Q' K'^T V
  float keps;    // ReLU: added to every feature
  int chunk;     // tokens per step of the causal scan: 64, or 32 (bf16 inputs)
};

// Scales of the projection W'' = ws W and of its seed b'' = bs b for the
// shape's feature kernel: cos takes revolutions (s / 2 pi, 1 / 2 pi); ReLU
// features carry 1 / sqrt(M) and no phase.
// sqrt(2 / M) of the cos features' D factor, for the M_r features drawn (a
// kernel argument, so that it stays in a scalar register).
inline float feature_norm(const Shape &sh) { return sqrtf(2.0f / (float)sh.Mr); }

inline void feature_scales(const Shape &sh, float &ws, float &bs) {
  if (sh.kernel == 1) {
    ws = sh.s / sqrtf((float)sh.Mr);
    bs = 0.f;
  } else {
    ws = sh.s * 0.15915494309189535f;
    bs = 0.15915494309189535f;
  }
}

hipError_t launch_orf_draw(uint64_t seed, int n_heads, int M, int kind, float *W, float *b,
                           hipStream_t st);

hipError_t launch_feature_map(const Shape &sh, Dt in, Dt out, const void *X, const float *W,
                              const float *b, void *Xp, hipStream_t st);

// Groups of four waves in one k_kside workgroup (two groups share each SIMD and
// one partial per row range): bf16 inputs with M >= 128 use two.
constexpr int kside_groups(Dt in, int M) { return in == Dt::BF16 && M >= 128 ? 2 : 1; }

// K side: per (head, row range) partial Buf1 = K'^T [V 1] -> part [BH][nsplit][M][65].
// Builds W'' = (s / 2 pi) W from W, b itself and stores the fragments
// [H][M/16][2][64] (element type of `in`) and b'' = b / 2 pi [H][M] of every
// head into wfr, bq for the launches that follow.
hipError_t launch_kside(const Shape &sh, Dt in, const void *K, const void *V, const float *W,
                        const float *b, void *wfr, float *bq, float *part, int rows_per_split,
                        int nsplit, hipStream_t st);

// Sum the partials of each head and write Buf1^T as Q-side operand fragments.
hipError_t launch_finalize(const Shape &sh, Dt in, const float *part, int nsplit, void *frags,
                           hipStream_t st);

// Q side: out = (Q' Buf1)[:, :d] / ((Q' Buf1)[:, d] + eps), Q' rebuilt on the fly.
hipError_t launch_qside(const Shape &sh, Dt in, Dt out, const void *Q, const void *wfr,
                        const float *bq, const void *frags, void *o, hipStream_t st);

// In-place exclusive scan of segment partials (plus state_in); writes state_out
// (state_in + total) and, if non-null, the total of this call's tokens as the
// Q-side Buf1^T fragments (the layout launch_finalize writes; element type of
// `in`) and as an aggregate total [BH][M][65] fp32.
hipError_t launch_seg_scan(const Shape &sh, Dt in, float *part, int nseg, const float *state_in,
                           float *state_out, void *total_frags, hipStream_t st,
                           float *total = nullptr);

// Forward passes that also write each row's 1 / (D-hat + eps) in units of the
// unscaled features (rsave [BH][L]) for the backward pass; renormalised shapes
// and out dtype = in dtype only.
hipError_t launch_qside_save(const Shape &sh, Dt in, const void *Q, const void *wfr,
                             const float *bq, const void *frags, void *o, float *rsave,
                             hipStream_t st);
hipError_t launch_causal_save(const Shape &sh, Dt in, const void *Q, const void *K,
                              const void *V, const void *wfr, const float *bq,
                              const float *prefix, void *o, float *rsave, int seg_len, int nseg,
                              float *halves, hipStream_t st);

// Backward pass. k_kside's weighted mode: part [BH][nsplit][M][65] = sum over
// each row range of Q-hat_t^T [aux_t.x dout_t, aux_t.y].
hipError_t launch_kside_agg(const Shape &sh, Dt in, const void *Q, const void *dout,
                            const float *W, const float *b, const float2 *aux, float *part,
                            int rows_per_split, int nsplit, hipStream_t st);

// Pointers of one backward launch (device; unused ones may be null).
struct BwdArgs {
  const void *Q, *K, *V, *dout, *out;
  const float *rsave;    // [BH][L] 1 / (D-hat + eps) (renormalised)
  const void *wfr;       // W'' fragments written by k_kside
  const float *bq;       // b''
  const float *W;        // [H][M][d]
  const float *state;    // dQ: Buf1 [BH][M][65] or segment prefixes [BH][nseg][M][65];
                         // dK, dV: dBuf1 or segment suffixes, same layouts
  void *dQ, *dK, *dV;
  float2 *aux;           // [BH][L] (alpha, alpha u_d)
  int seg_len, nseg;     // causal: the segments of the forward plan
};
// accumulate (causal only): add onto dQ instead of overwriting it.
hipError_t launch_bwd_dq(const Shape &sh, Dt in, bool causal, const BwdArgs &a, hipStream_t st,
                         bool accumulate = false);
hipError_t launch_bwd_dkv(const Shape &sh, Dt in, bool causal, const BwdArgs &a, hipStream_t st);
// Fixed-order sum of split partials [BH][ns][M][65] -> [BH][M][65].
hipError_t launch_sum_splits(const Shape &sh, const float *part, int ns, float *dst,
                             hipStream_t st);
// In-place exclusive suffix scan over chunks plus dsout; the total plus dsout to dsin.
// bias (nullable, [BH][M][65]): added to every suffix but not to dsin.
hipError_t launch_suffix_scan(const Shape &sh, float *part, int nch, const float *dsout,
                              float *dsin, hipStream_t st, const float *bias = nullptr);

// Causal chunk scan of each segment starting from its prefix state. halves:
// [BH][L][68] fp32 scratch for fp32 inputs at M = 256 (two feature-half
// passes), else unused (may be null).
hipError_t launch_causal(const Shape &sh, Dt in, Dt out, const void *Q, const void *K,
                         const void *V, const void *wfr, const float *bq, const float *prefix,
                         void *o, int seg_len, int nseg, float *halves, hipStream_t st);

}  // namespace favor

namespace favor {

// Kernel ids for the per-launch timing facility (favor_timing_*).
enum KernelId {
  kKerOrfDraw = 0,
  kKerFeatureMap,
  kKerKside,
  kKerFinalize,
  kKerQside,
  kKerSegScan,
  kKerCausal,
  kKerSumSplits,
  kKerBwdDq,
  kKerBwdAgg,
  kKerSuffixScan,
  kKerBwdDkv,
  kNumKernels
};
const char *kernel_name(int k);

// Records msg as the calling thread's favor_last_error text and returns st.
favor_status report(favor_status st, const char *msg);

// Brackets one launch with pooled HIP events on `st` while timing is enabled.
class LaunchTimer {
 public:
  LaunchTimer(int kernel, hipStream_t st);
  ~LaunchTimer();
  LaunchTimer(const LaunchTimer &) = delete;
  LaunchTimer &operator=(const LaunchTimer &) = delete;

 private:
  int kernel_;
  hipStream_t st_;
  hipEvent_t begin_ = nullptr;
};

}  // namespace favor
