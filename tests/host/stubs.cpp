// stubs.cpp - CPU-only stand-ins for the device side of libfavor, so that the
// host layer (favor_api.cpp, timing.cpp) can be built with g++ under address
// and undefined-behaviour sanitizers and driven by the descriptor fuzzer.
// Every launcher records that it ran and checks the arguments the host layer
// hands it for internal consistency; the few HIP runtime calls the host layer
// makes are answered here, so nothing touches a GPU.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

#include "../../paper_2006_03555_amd/csrc/kernels.hpp"

int g_launches = 0;

namespace {

void require(bool ok, const char *what) {
  if (!ok) {
    std::fprintf(stderr, "inconsistent launch arguments: %s\n", what);
    std::abort();
  }
}

void shape_ok(const favor::Shape &sh) {
  require(sh.BH > 0 && sh.H > 0 && sh.BH % sh.H == 0, "B*H a positive multiple of H");
  require(sh.L > 0, "L > 0 when launching");
  require(sh.M == 64 || sh.M == 128 || sh.M == 256, "padded M");
  require(sh.Mr > 0 && sh.Mr <= sh.M && sh.Mr % 16 == 0, "M drawn");
}

void plan_ok(const favor::Shape &sh, int rows, int nseg) {
  require(rows > 0 && rows % 64 == 0, "rows per split a positive multiple of 64");
  require(nseg > 0 && (long long)rows * nseg >= sh.L && (long long)rows * (nseg - 1) < sh.L,
          "splits cover L exactly once");
}

hipError_t ran() {
  ++g_launches;
  return hipSuccess;
}

}  // namespace

namespace favor {

hipError_t launch_orf_draw(uint64_t, int n_heads, int M, int, float *W, float *b, hipStream_t) {
  require(n_heads > 0 && M > 0 && W && b, "draw arguments");
  return ran();
}
hipError_t launch_feature_map(const Shape &sh, Dt, Dt, const void *X, const float *W,
                              const float *b, void *Xp, hipStream_t) {
  shape_ok(sh);
  require(X && W && b && Xp, "feature map pointers");
  return ran();
}
hipError_t launch_kside(const Shape &sh, Dt, const void *K, const void *V, const float *W,
                        const float *b, void *wfr, float *bq, float *part, int rows, int nsplit,
                        hipStream_t) {
  shape_ok(sh);
  plan_ok(sh, rows, nsplit);
  require(K && V && W && b && wfr && bq && part, "key pass pointers");
  return ran();
}
hipError_t launch_finalize(const Shape &sh, Dt, const float *part, int nsplit, void *frags,
                           hipStream_t) {
  shape_ok(sh);
  require(part && frags && nsplit > 0, "finalize");
  return ran();
}
hipError_t launch_qside(const Shape &sh, Dt, Dt, const void *Q, const void *wfr, const float *bq,
                        const void *frags, void *o, hipStream_t) {
  shape_ok(sh);
  require(Q && wfr && bq && frags && o, "query pass pointers");
  return ran();
}
hipError_t launch_seg_scan(const Shape &sh, Dt, float *part, int nseg, const float *, float *,
                           void *, hipStream_t, float *) {
  require(sh.BH > 0, "segment scan heads");
  require((part == nullptr) == (nseg == 0), "segment scan partials");
  return ran();
}
hipError_t launch_qside_save(const Shape &sh, Dt, const void *Q, const void *wfr, const float *bq,
                             const void *frags, void *o, float *rsave, hipStream_t) {
  shape_ok(sh);
  require(Q && wfr && bq && frags && o && rsave && sh.renorm, "saving query pass");
  return ran();
}
hipError_t launch_causal_save(const Shape &sh, Dt, const void *Q, const void *K, const void *V,
                              const void *wfr, const float *bq, const float *prefix, void *o,
                              float *rsave, int seg_len, int nseg, float *, hipStream_t) {
  shape_ok(sh);
  plan_ok(sh, seg_len, nseg);
  require(Q && K && V && wfr && bq && prefix && o && rsave && sh.renorm, "saving causal pass");
  return ran();
}
hipError_t launch_causal(const Shape &sh, Dt, Dt, const void *Q, const void *K, const void *V,
                         const void *wfr, const float *bq, const float *prefix, void *o,
                         int seg_len, int nseg, float *, hipStream_t) {
  shape_ok(sh);
  plan_ok(sh, seg_len, nseg);
  require(Q && K && V && wfr && bq && prefix && o, "causal pass pointers");
  return ran();
}
hipError_t launch_kside_agg(const Shape &sh, Dt, const void *Q, const void *dout, const float *W,
                            const float *b, const float2 *aux, float *part, int rows,
                            int nsplit, hipStream_t) {
  shape_ok(sh);
  plan_ok(sh, rows, nsplit);
  require(Q && dout && W && b && aux && part, "weighted key pass pointers");
  return ran();
}
hipError_t launch_bwd_dq(const Shape &sh, Dt, bool causal, const BwdArgs &a, hipStream_t,
                         bool accumulate) {
  shape_ok(sh);
  require(a.Q && a.dout && a.out && a.rsave && a.W && a.state && a.dQ && a.aux, "dQ pass");
  require(causal || !accumulate, "only the causal dQ pass adds onto dQ");
  if (causal) plan_ok(sh, a.seg_len, a.nseg);
  return ran();
}
hipError_t launch_bwd_dkv(const Shape &sh, Dt, bool causal, const BwdArgs &a, hipStream_t) {
  shape_ok(sh);
  require(a.K && a.V && a.W && a.state && a.dK && a.dV, "dK dV pass");
  if (causal) plan_ok(sh, a.seg_len, a.nseg);
  return ran();
}
hipError_t launch_sum_splits(const Shape &sh, const float *part, int ns, float *dst, hipStream_t) {
  shape_ok(sh);
  require(part && dst && ns > 0, "sum of splits");
  return ran();
}
hipError_t launch_suffix_scan(const Shape &sh, float *part, int nch, const float *, float *dsin,
                              hipStream_t, const float *bias) {
  require(sh.BH > 0 && nch >= 0 && (nch > 0 || dsin), "suffix scan");
  require(!bias || (part && nch > 0), "suffix bias without suffixes");
  return ran();
}

}  // namespace favor

// The HIP runtime calls of the host layer (timing and error strings).
extern "C" {
const char *hipGetErrorString(hipError_t) { return "stubbed HIP error"; }
hipError_t hipEventCreate(hipEvent_t *e) {
  *e = reinterpret_cast<hipEvent_t>(new int(0));
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
hipError_t hipEventElapsedTime(float *ms, hipEvent_t, hipEvent_t) {
  *ms = 0.f;
  return hipSuccess;
}
}
