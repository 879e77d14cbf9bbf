// favor_api.cpp - the C ABI of libfavor: argument validation, workspace
// sizing, launch planning and dispatch to the kernels. Validation is plain
// host code that touches no device, so a bad call never launches anything.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include "../../include/favor.h"
#include "kernels.hpp"

namespace {

thread_local std::string g_last_error;

favor_status fail(favor_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

favor_status ok() {
  g_last_error.clear();
  return FAVOR_OK;
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// The integer a caller stored in an enum-typed field or argument. A C caller
// may pass any int there, and in C++ reading an enum object that holds a value
// outside its enumerators is undefined, so validation reads the bytes.
static_assert(sizeof(favor_dtype) == sizeof(int) && sizeof(favor_rf_kind) == sizeof(int),
              "the enums of the C ABI are int-sized");
int raw_enum(const void *p) {
  int v;
  std::memcpy(&v, p, sizeof v);
  return v;
}

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Rows the kernels work on for M features: 64, 128 or 256 (the rows past M are
// padding with zero features).
int padded_m(int M) { return M <= 64 ? 64 : M <= 128 ? 128 : 256; }

constexpr int kTargetWorkgroups = 512;  // two waves of workgroups over 256 CUs
// the causal pass with 64-token chunks holds a whole compute unit per
// workgroup (LDS and registers), so its segments are sized for one workgroup
// per CU; with 32-token chunks two workgroups share a CU
constexpr int kCausalWorkgroups = 256;
constexpr int kMinRowsPerSplit = 256;
// Causal segments may be shorter: on short sequences more segments keep more
// CUs busy, and a segment of two 64-token chunks still amortises the scan's
// prologue (measured: the causal call 10-23% and its gradients 25-32% faster at
// L <= 1024 for 32 heads; longer sequences keep the workgroup target's segments)
constexpr int kMinRowsPerSegment = 128;
// Longest sequence per head (and longest causal segment): the kernels index
// tokens with 32-bit integers and step past the end by up to two tiles.
constexpr int kMaxL = 1 << 30;
// Tokens per step of the causal scan: 64 by default (four 16-token matrix-core
// blocks in the intra-chunk product); bf16 inputs also take 32.
constexpr int kChunk = 64;
constexpr int kChunkSmall = 32;

// The chunk length a call runs with: the descriptor's, or by default 32 for
// bf16 inputs with at most 128 feature rows (two workgroups per CU scan those
// faster) and 64 otherwise.
int chunk_len(const favor_desc *g) {
  if (g->chunk != 0) return g->chunk;
  return g->in_dtype == FAVOR_BF16 && padded_m(g->M) <= 128 ? kChunkSmall : kChunk;
}

enum Op {
  kOpFeatureMap = 0,
  kOpBidir = 1,
  kOpCausal = 2,
  kOpBoth = 3,
  kOpBidirBackward = 4,
  kOpCausalBackward = 5,
  kOpBothBackward = 6
};

favor_status validate(const favor_desc *g, int op) {
  if (!g) return fail(FAVOR_ERR_INVALID_ARGUMENT, "descriptor is NULL");
  if (op < kOpFeatureMap || op > kOpBothBackward)
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "unknown operation %d", op);
  if (g->B < 0 || g->H < 0 || g->L < 0)
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "negative size B=%d H=%d L=%d", g->B, g->H, g->L);
  if (g->d <= 0 || g->M <= 0)
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "d=%d and M=%d must be positive", g->d, g->M);
  const int in_dt = raw_enum(&g->in_dtype), out_dt = raw_enum(&g->out_dtype);
  if (in_dt != FAVOR_F32 && in_dt != FAVOR_BF16)
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "unknown in_dtype %d", in_dt);
  if (out_dt != FAVOR_F32 && out_dt != FAVOR_BF16)
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "unknown out_dtype %d", out_dt);
  if (!std::isfinite(g->input_scale))
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "input_scale must be finite");
  if (!std::isfinite(g->denom_eps) || g->denom_eps < 0.f)
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "denom_eps must be finite and >= 0");
  if (g->kernel != FAVOR_KERNEL_SOFTMAX && g->kernel != FAVOR_KERNEL_RELU)
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "unknown kernel %d", (int)g->kernel);
  if (g->no_renormalize != 0 && g->no_renormalize != 1)
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "no_renormalize must be 0 or 1");
  if (g->kernel == FAVOR_KERNEL_RELU && (!std::isfinite(g->kernel_eps) || g->kernel_eps < 0.f))
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "kernel_eps must be finite and >= 0");
  if (g->chunk < 0) return fail(FAVOR_ERR_INVALID_ARGUMENT, "chunk=%d is negative", g->chunk);
  if (g->segment < 0 || g->segment % 64 != 0)
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "segment=%d must be a non-negative multiple of 64",
                g->segment);
  if (g->L > kMaxL) return fail(FAVOR_ERR_UNSUPPORTED, "L=%d exceeds 2^30", g->L);
  if (g->chunk != 0 && g->chunk != kChunk && g->chunk != kChunkSmall)
    return fail(FAVOR_ERR_UNSUPPORTED, "chunk=%d not supported (T = 64 or 32)", g->chunk);
  if (g->chunk == kChunkSmall && in_dt != FAVOR_BF16 &&
      (op == kOpCausal || op == kOpBoth || op == kOpCausalBackward || op == kOpBothBackward))
    return fail(FAVOR_ERR_UNSUPPORTED, "chunk=32 needs bf16 inputs (the fp32 scan takes T = 64)");
  if (g->segment > kMaxL)
    return fail(FAVOR_ERR_UNSUPPORTED, "segment=%d exceeds 2^30", g->segment);
  if (g->d != 64) return fail(FAVOR_ERR_UNSUPPORTED, "d=%d not supported (d = 64)", g->d);
  if (g->M % 16 != 0 || g->M > 256)
    return fail(FAVOR_ERR_UNSUPPORTED, "M=%d not supported (a multiple of 16, at most 256)",
                g->M);
  const long long bh = (long long)g->B * g->H;
  if (bh > 65535) return fail(FAVOR_ERR_UNSUPPORTED, "B*H=%lld exceeds 65535", bh);
  if (op == kOpBidirBackward || op == kOpCausalBackward || op == kOpBothBackward) {
    if (g->out_dtype != g->in_dtype)
      return fail(FAVOR_ERR_UNSUPPORTED, "the backward pass needs out_dtype == in_dtype");
  }
  return FAVOR_OK;
}

// Backward workspace: the forward plan's buffers (split or segment
// partials, Buf1^T fragments, W'', b''), then the recomputed output and row
// reciprocals, the per-row (alpha, alpha u_d), the aggregated q-hat (x) u~
// partials and, bidirectional, Buf1 and dBuf1 as plain [M][65] arrays.
struct BwdPlan {
  int BH = 0;
  int nsplit = 0;
  int rows_per_split = 0;
  size_t part = 0, frags = 0, wfr = 0, bq = 0, out = 0, rsave = 0, aux = 0, part2 = 0,
         buf1 = 0, dbuf1 = 0, halves = 0;
  size_t total = 0;
};

// Workspace: [ split partials | Buf1^T fragments (bidir, both) | W'' fragments | b'' |
//              Buf1 as an fp32 aggregate (both) |
//              feature-half partials (causal and both, fp32 inputs at M > 128) ]
// A backward call given the workspace of a forward call reads the partials
// (split partials, or segment prefixes after the scan), W'', b'' and the
// both-directions total from these offsets.
struct Plan {
  int BH = 0;
  int nsplit = 0;         // bidir: K-side splits; causal and both: segments
  int rows_per_split = 0;
  size_t part_bytes = 0;
  size_t frag_bytes = 0;  // bidir and both
  size_t wfr_bytes = 0;
  size_t bq_bytes = 0;
  size_t sum_bytes = 0;   // both: [BH][M][65] fp32, Buf1 = the scan's total
  size_t half_bytes = 0;  // [BH][L][68] fp32: the first feature half's raw row results
  size_t total = 0;
};

// Pointers into a forward call's workspace (plan p).
struct FwdBufs {
  float *part, *bq, *sum, *halves;
  void *frags, *wfr;
};
FwdBufs carve_fwd(const Plan &p, void *ws) {
  char *c = static_cast<char *>(ws);
  FwdBufs f;
  f.part = reinterpret_cast<float *>(c);
  c += p.part_bytes;
  f.frags = c;
  c += p.frag_bytes;
  f.wfr = c;
  c += p.wfr_bytes;
  f.bq = reinterpret_cast<float *>(c);
  c += p.bq_bytes;
  f.sum = p.sum_bytes ? reinterpret_cast<float *>(c) : nullptr;
  c += p.sum_bytes;
  f.halves = p.half_bytes ? reinterpret_cast<float *>(c) : nullptr;
  return f;
}

Plan make_plan(const favor_desc *g, int op) {
  const bool causal = (op != kOpBidir);
  Plan p;
  p.BH = g->B * g->H;
  if (p.BH == 0 || g->L == 0) return p;
  // L and segment are at most 2^30 (validated), so these stay within int
  const int tiles = (g->L + 63) / 64;
  int rows;
  if (causal && g->segment > 0) {
    rows = g->segment;
  } else {
    // a two-group k_kside workgroup fills a CU by itself
    const favor::Dt in = g->in_dtype == FAVOR_BF16 ? favor::Dt::BF16 : favor::Dt::F32;
    const int target = !causal ? kTargetWorkgroups / favor::kside_groups(in, padded_m(g->M))
                       : chunk_len(g) == kChunkSmall ? 2 * kCausalWorkgroups
                                                     : kCausalWorkgroups;
    int want = (target + p.BH - 1) / p.BH;
    int max_split = tiles / ((causal ? kMinRowsPerSegment : kMinRowsPerSplit) / 64);
    if (max_split < 1) max_split = 1;
    if (want > max_split) want = max_split;
    if (want < 1) want = 1;
    rows = 64 * ((tiles + want - 1) / want);
  }
  p.rows_per_split = rows;
  p.nsplit = (int)(((long long)g->L + rows - 1) / rows);
  const int M = padded_m(g->M);
  p.part_bytes = round_up((size_t)p.BH * p.nsplit * M * 65 * sizeof(float), 256);
  const int fb = g->in_dtype == FAVOR_BF16 ? 16 : 32;
  if (op != kOpCausal) p.frag_bytes = round_up((size_t)p.BH * 5 * (M / 32) * 64 * fb, 256);
  p.wfr_bytes = round_up((size_t)g->H * (M / 16) * 2 * 64 * fb, 256);
  p.bq_bytes = round_up((size_t)g->H * M * sizeof(float), 256);
  if (op == kOpBoth) p.sum_bytes = round_up((size_t)p.BH * M * 65 * sizeof(float), 256);
  if (causal && g->in_dtype == FAVOR_F32 && M > 128)
    p.half_bytes = round_up((size_t)p.BH * g->L * 68 * sizeof(float), 256);
  p.total = p.part_bytes + p.frag_bytes + p.wfr_bytes + p.bq_bytes + p.sum_bytes + p.half_bytes;
  return p;
}

BwdPlan make_bwd_plan(const favor_desc *g, bool causal) {
  BwdPlan p;
  p.BH = g->B * g->H;
  if (p.BH == 0 || g->L == 0) return p;
  const size_t elt = g->in_dtype == FAVOR_BF16 ? 2 : 4;
  const int M = padded_m(g->M);
  const size_t agg = (size_t)M * 65 * sizeof(float);
  // the forward plan's splits (bidirectional) or segments (causal)
  const Plan f = make_plan(g, causal ? kOpCausal : kOpBidir);
  p.rows_per_split = f.rows_per_split;
  p.nsplit = f.nsplit;
  const int fb = g->in_dtype == FAVOR_BF16 ? 16 : 32;
  p.part = round_up((size_t)p.BH * p.nsplit * agg, 256);
  p.frags = causal ? 0 : round_up((size_t)p.BH * 5 * (M / 32) * 64 * fb, 256);
  p.wfr = round_up((size_t)g->H * (M / 16) * 2 * 64 * fb, 256);
  p.bq = round_up((size_t)g->H * M * sizeof(float), 256);
  p.out = round_up((size_t)p.BH * g->L * 64 * elt, 256);
  p.rsave = round_up((size_t)p.BH * g->L * sizeof(float), 256);
  p.aux = round_up((size_t)p.BH * g->L * 2 * sizeof(float), 256);
  p.part2 = p.part;
  p.buf1 = causal ? 0 : round_up((size_t)p.BH * agg, 256);
  p.dbuf1 = p.buf1;
  p.halves = f.half_bytes;   // the recomputed causal pass of fp32 inputs at M > 128
  p.total = p.part + p.frags + p.wfr + p.bq + p.out + p.rsave + p.aux + p.part2 + p.buf1 +
            p.dbuf1 + p.halves;
  return p;
}

favor::Shape shape_of(const favor_desc *g) {
  favor::Shape sh;
  sh.BH = g->B * g->H;
  sh.H = g->H;
  sh.L = g->L;
  sh.M = padded_m(g->M);
  sh.Mr = g->M;
  sh.s = g->input_scale;
  sh.eps = g->denom_eps;
  sh.kernel = g->kernel;
  sh.renorm = g->no_renormalize ? 0 : 1;
  sh.keps = g->kernel == FAVOR_KERNEL_RELU ? g->kernel_eps : 0.f;
  sh.chunk = chunk_len(g);
  return sh;
}

favor::Dt dt_of(favor_dtype d) { return d == FAVOR_BF16 ? favor::Dt::BF16 : favor::Dt::F32; }

favor_status check_ptr(const void *p, const char *name, bool needed) {
  if (!needed) return FAVOR_OK;
  if (!p) return fail(FAVOR_ERR_INVALID_ARGUMENT, "%s is NULL", name);
  if (!aligned(p, 16)) return fail(FAVOR_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", name);
  return FAVOR_OK;
}

// A forward call's optional row_scale output.
favor_status check_row_scale(const favor_desc *g, const void *rs, const char *name) {
  if (!rs || g->no_renormalize) return FAVOR_OK;
  if (!aligned(rs, 4)) return fail(FAVOR_ERR_INVALID_ARGUMENT, "%s is not 4-byte aligned", name);
  if (g->out_dtype != g->in_dtype)
    return fail(FAVOR_ERR_UNSUPPORTED, "%s needs out_dtype == in_dtype", name);
  return FAVOR_OK;
}

favor_status device_result(hipError_t e, const char *what) {
  if (e != hipSuccess)
    return fail(FAVOR_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

#define FAVOR_TRY(expr)                   \
  do {                                    \
    favor_status st__ = (expr);           \
    if (st__ != FAVOR_OK) return st__;    \
  } while (0)

}  // namespace

namespace favor {

// Records msg as the calling thread's favor_last_error text and returns st.
favor_status report(favor_status st, const char *msg) { return fail(st, "%s", msg); }

}  // namespace favor

extern "C" {

int32_t favor_abi_version(void) { return FAVOR_ABI_VERSION; }

const char *favor_last_error(void) { return g_last_error.c_str(); }

const char *favor_status_string(favor_status s) {
  switch (s) {
    case FAVOR_OK: return "FAVOR_OK";
    case FAVOR_ERR_INVALID_ARGUMENT: return "FAVOR_ERR_INVALID_ARGUMENT";
    case FAVOR_ERR_UNSUPPORTED: return "FAVOR_ERR_UNSUPPORTED";
    case FAVOR_ERR_WORKSPACE_TOO_SMALL: return "FAVOR_ERR_WORKSPACE_TOO_SMALL";
    case FAVOR_ERR_DEVICE: return "FAVOR_ERR_DEVICE";
  }
  return "FAVOR_ERR_UNKNOWN";
}

favor_status favor_validate_desc(const favor_desc *g, int op) {
  FAVOR_TRY(validate(g, op));
  return ok();
}

size_t favor_backward_workspace_size(const favor_desc *g, int causal) {
  const int op = causal == 2 ? kOpBothBackward : (causal ? kOpCausalBackward : kOpBidirBackward);
  if (validate(g, op) != FAVOR_OK) return 0;
  if (op == kOpBothBackward) return make_bwd_plan(g, false).total + make_bwd_plan(g, true).total;
  return make_bwd_plan(g, causal != 0).total;
}

size_t favor_workspace_size(const favor_desc *g, int causal) {
  const int op = causal == 2 ? kOpBoth : (causal ? kOpCausal : kOpBidir);
  if (validate(g, op) != FAVOR_OK) return 0;
  return make_plan(g, op).total;
}

favor_status favor_orf_draw(uint64_t seed, int32_t n_heads, int32_t M, int32_t d,
                            favor_rf_kind kind, float *W, float *b, hipStream_t stream) {
  if (n_heads < 0) return fail(FAVOR_ERR_INVALID_ARGUMENT, "n_heads=%d is negative", n_heads);
  if (M <= 0 || d <= 0) return fail(FAVOR_ERR_INVALID_ARGUMENT, "M=%d d=%d must be positive", M, d);
  const int k = raw_enum(&kind);
  if (k != FAVOR_RF_ORTHO_CHI && k != FAVOR_RF_ORTHO_FIXED && k != FAVOR_RF_IID &&
      k != FAVOR_RF_HADAMARD && k != FAVOR_RF_GIVENS)
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "unknown random-feature kind %d", k);
  if (d != 64) return fail(FAVOR_ERR_UNSUPPORTED, "d=%d not supported (d = 64)", d);
  if (M > 4096) return fail(FAVOR_ERR_UNSUPPORTED, "M=%d exceeds 4096", M);
  if (n_heads > 65535) return fail(FAVOR_ERR_UNSUPPORTED, "n_heads=%d exceeds 65535", n_heads);
  if (n_heads == 0) return ok();
  if (!W || !b) return fail(FAVOR_ERR_INVALID_ARGUMENT, "W and b must be non-NULL");
  if (!aligned(W, 16) || !aligned(b, 4))
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "W must be 16-byte and b 4-byte aligned");
  hipError_t e;
  {
    favor::LaunchTimer t(favor::kKerOrfDraw, stream);
    e = favor::launch_orf_draw(seed, n_heads, M, k, W, b, stream);
  }
  return device_result(e, "favor_orf_draw launch");
}

favor_status favor_feature_map(const favor_desc *g, const void *X, const float *W,
                               const float *b, void *Xprime, hipStream_t stream) {
  FAVOR_TRY(validate(g, kOpFeatureMap));
  const bool work = (long long)g->B * g->H * g->L > 0;
  FAVOR_TRY(check_ptr(X, "X", work));
  FAVOR_TRY(check_ptr(W, "W", work));
  FAVOR_TRY(check_ptr(b, "b", work));
  FAVOR_TRY(check_ptr(Xprime, "Xprime", work));
  if (!work) return ok();
  hipError_t e;
  {
    favor::LaunchTimer t(favor::kKerFeatureMap, stream);
    e = favor::launch_feature_map(shape_of(g), dt_of(g->in_dtype), dt_of(g->out_dtype), X, W, b,
                                  Xprime, stream);
  }
  return device_result(e, "favor_feature_map launch");
}

favor_status favor_attn_bidir(const favor_desc *g, const void *Q, const void *K,
                              const void *V, const float *W, const float *b, void *out,
                              void *ws, size_t ws_bytes, hipStream_t stream) {
  return favor_attn_bidir_save(g, Q, K, V, W, b, out, nullptr, ws, ws_bytes, stream);
}

favor_status favor_attn_bidir_save(const favor_desc *g, const void *Q, const void *K,
                                   const void *V, const float *W, const float *b, void *out,
                                   float *row_scale, void *ws, size_t ws_bytes,
                                   hipStream_t stream) {
  FAVOR_TRY(validate(g, kOpBidir));
  FAVOR_TRY(check_row_scale(g, row_scale, "row_scale"));
  const Plan p = make_plan(g, kOpBidir);
  const bool work = p.total > 0;
  FAVOR_TRY(check_ptr(Q, "Q", work));
  FAVOR_TRY(check_ptr(K, "K", work));
  FAVOR_TRY(check_ptr(V, "V", work));
  FAVOR_TRY(check_ptr(W, "W", work));
  FAVOR_TRY(check_ptr(b, "b", work));
  FAVOR_TRY(check_ptr(out, "out", work));
  if (!work) return ok();
  if (!ws) return fail(FAVOR_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (!aligned(ws, 256)) return fail(FAVOR_ERR_INVALID_ARGUMENT, "workspace is not 256-byte aligned");
  if (ws_bytes < p.total)
    return fail(FAVOR_ERR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes, p.total);
  const favor::Shape sh = shape_of(g);
  const favor::Dt in = dt_of(g->in_dtype);
  hipStream_t st = stream;
  const FwdBufs f = carve_fwd(p, ws);
  float *part = f.part;
  void *frags = f.frags;
  void *wfr = f.wfr;
  float *bq = f.bq;
  hipError_t e;
  {
    favor::LaunchTimer t(favor::kKerKside, st);
    e = favor::launch_kside(sh, in, K, V, W, b, wfr, bq, part, p.rows_per_split, p.nsplit, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_bidir key pass");
  {
    favor::LaunchTimer t(favor::kKerFinalize, st);
    e = favor::launch_finalize(sh, in, part, p.nsplit, frags, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_bidir reduction");
  {
    favor::LaunchTimer t(favor::kKerQside, st);
    if (row_scale && sh.renorm)
      e = favor::launch_qside_save(sh, in, Q, wfr, bq, frags, out, row_scale, st);
    else
      e = favor::launch_qside(sh, in, dt_of(g->out_dtype), Q, wfr, bq, frags, out, st);
  }
  return device_result(e, "favor_attn_bidir query pass");
}

favor_status favor_attn_causal(const favor_desc *g, const void *Q, const void *K,
                               const void *V, const float *W, const float *b, void *out,
                               const float *state_in, float *state_out, void *ws,
                               size_t ws_bytes, hipStream_t stream) {
  return favor_attn_causal_save(g, Q, K, V, W, b, out, state_in, state_out, nullptr, ws,
                                ws_bytes, stream);
}

favor_status favor_attn_causal_save(const favor_desc *g, const void *Q, const void *K,
                                    const void *V, const float *W, const float *b, void *out,
                                    const float *state_in, float *state_out, float *row_scale,
                                    void *ws, size_t ws_bytes, hipStream_t stream) {
  FAVOR_TRY(validate(g, kOpCausal));
  FAVOR_TRY(check_row_scale(g, row_scale, "row_scale"));
  const Plan p = make_plan(g, kOpCausal);
  const bool work = p.total > 0;
  const bool heads = (long long)g->B * g->H > 0;
  FAVOR_TRY(check_ptr(Q, "Q", work));
  FAVOR_TRY(check_ptr(K, "K", work));
  FAVOR_TRY(check_ptr(V, "V", work));
  FAVOR_TRY(check_ptr(W, "W", work));
  FAVOR_TRY(check_ptr(b, "b", work));
  FAVOR_TRY(check_ptr(out, "out", work));
  if (state_in && !aligned(state_in, 16))
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "state_in is not 16-byte aligned");
  if (state_out && !aligned(state_out, 16))
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "state_out is not 16-byte aligned");
  const favor::Shape sh = shape_of(g);
  hipStream_t st = stream;
  if (!work) {
    // no tokens: the carried state passes through unchanged
    if (heads && state_out) {
      hipError_t e;
      {
        favor::LaunchTimer t(favor::kKerSegScan, st);
        e = favor::launch_seg_scan(sh, favor::Dt::F32, nullptr, 0, state_in, state_out, nullptr,
                                   st);
      }
      return device_result(e, "favor_attn_causal state copy");
    }
    return ok();
  }
  if (!ws) return fail(FAVOR_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (!aligned(ws, 256)) return fail(FAVOR_ERR_INVALID_ARGUMENT, "workspace is not 256-byte aligned");
  if (ws_bytes < p.total)
    return fail(FAVOR_ERR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes, p.total);
  const favor::Dt in = dt_of(g->in_dtype);
  const FwdBufs f = carve_fwd(p, ws);
  float *part = f.part;
  void *wfr = f.wfr;
  float *bq = f.bq;
  float *halves = f.halves;
  hipError_t e;
  {
    favor::LaunchTimer t(favor::kKerKside, st);
    e = favor::launch_kside(sh, in, K, V, W, b, wfr, bq, part, p.rows_per_split, p.nsplit, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_causal segment aggregates");
  {
    favor::LaunchTimer t(favor::kKerSegScan, st);
    e = favor::launch_seg_scan(sh, in, part, p.nsplit, state_in, state_out, nullptr, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_causal segment scan");
  {
    favor::LaunchTimer t(favor::kKerCausal, st);
    if (row_scale && sh.renorm)
      e = favor::launch_causal_save(sh, in, Q, K, V, wfr, bq, part, out, row_scale,
                                    p.rows_per_split, p.nsplit, halves, st);
    else
      e = favor::launch_causal(sh, in, dt_of(g->out_dtype), Q, K, V, wfr, bq, part, out,
                               p.rows_per_split, p.nsplit, halves, st);
  }
  return device_result(e, "favor_attn_causal chunk scan");
}

favor_status favor_attn_both(const favor_desc *g, const void *Q, const void *K, const void *V,
                             const float *W, const float *b, void *out_bidir, void *out_causal,
                             const float *state_in, float *state_out, float *row_scale_bidir,
                             float *row_scale_causal, void *ws, size_t ws_bytes,
                             hipStream_t stream) {
  FAVOR_TRY(validate(g, kOpBoth));
  FAVOR_TRY(check_row_scale(g, row_scale_bidir, "row_scale_bidir"));
  FAVOR_TRY(check_row_scale(g, row_scale_causal, "row_scale_causal"));
  const Plan p = make_plan(g, kOpBoth);
  const bool work = p.total > 0;
  const bool heads = (long long)g->B * g->H > 0;
  FAVOR_TRY(check_ptr(Q, "Q", work));
  FAVOR_TRY(check_ptr(K, "K", work));
  FAVOR_TRY(check_ptr(V, "V", work));
  FAVOR_TRY(check_ptr(W, "W", work));
  FAVOR_TRY(check_ptr(b, "b", work));
  FAVOR_TRY(check_ptr(out_bidir, "out_bidir", work));
  FAVOR_TRY(check_ptr(out_causal, "out_causal", work));
  if (state_in && !aligned(state_in, 16))
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "state_in is not 16-byte aligned");
  if (state_out && !aligned(state_out, 16))
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "state_out is not 16-byte aligned");
  const favor::Shape sh = shape_of(g);
  hipStream_t st = stream;
  if (!work) {
    if (heads && state_out) {
      hipError_t e;
      {
        favor::LaunchTimer t(favor::kKerSegScan, st);
        e = favor::launch_seg_scan(sh, favor::Dt::F32, nullptr, 0, state_in, state_out, nullptr,
                                   st);
      }
      return device_result(e, "favor_attn_both state copy");
    }
    return ok();
  }
  if (!ws) return fail(FAVOR_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (!aligned(ws, 256)) return fail(FAVOR_ERR_INVALID_ARGUMENT, "workspace is not 256-byte aligned");
  if (ws_bytes < p.total)
    return fail(FAVOR_ERR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes, p.total);
  const favor::Dt in = dt_of(g->in_dtype);
  const favor::Dt out = dt_of(g->out_dtype);
  const FwdBufs f = carve_fwd(p, ws);
  float *part = f.part;
  void *frags = f.frags;
  void *wfr = f.wfr;
  float *bq = f.bq;
  float *halves = f.halves;
  hipError_t e;
  {
    favor::LaunchTimer t(favor::kKerKside, st);
    e = favor::launch_kside(sh, in, K, V, W, b, wfr, bq, part, p.rows_per_split, p.nsplit, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_both segment aggregates");
  {
    // the segment scan also writes the total over the sequence (Buf1) as Q-side fragments
    favor::LaunchTimer t(favor::kKerSegScan, st);
    e = favor::launch_seg_scan(sh, in, part, p.nsplit, state_in, state_out, frags, st, f.sum);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_both segment scan");
  {
    favor::LaunchTimer t(favor::kKerQside, st);
    if (row_scale_bidir && sh.renorm)
      e = favor::launch_qside_save(sh, in, Q, wfr, bq, frags, out_bidir, row_scale_bidir, st);
    else
      e = favor::launch_qside(sh, in, out, Q, wfr, bq, frags, out_bidir, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_both bidirectional query pass");
  {
    favor::LaunchTimer t(favor::kKerCausal, st);
    if (row_scale_causal && sh.renorm)
      e = favor::launch_causal_save(sh, in, Q, K, V, wfr, bq, part, out_causal,
                                    row_scale_causal, p.rows_per_split, p.nsplit, halves, st);
    else
      e = favor::launch_causal(sh, in, out, Q, K, V, wfr, bq, part, out_causal,
                               p.rows_per_split, p.nsplit, halves, st);
  }
  return device_result(e, "favor_attn_both chunk scan");
}

}  // extern "C"

namespace {

// Carve the backward workspace.
struct BwdBufs {
  float *part, *bq, *rsave, *part2, *buf1, *dbuf1, *halves;
  void *frags, *wfr, *out;
  float2 *aux;
};

BwdBufs carve(const BwdPlan &p, void *ws) {
  char *c = static_cast<char *>(ws);
  BwdBufs b;
  b.part = reinterpret_cast<float *>(c);
  c += p.part;
  b.frags = c;
  c += p.frags;
  b.wfr = c;
  c += p.wfr;
  b.bq = reinterpret_cast<float *>(c);
  c += p.bq;
  b.out = c;
  c += p.out;
  b.rsave = reinterpret_cast<float *>(c);
  c += p.rsave;
  b.aux = reinterpret_cast<float2 *>(c);
  c += p.aux;
  b.part2 = reinterpret_cast<float *>(c);
  c += p.part2;
  b.buf1 = reinterpret_cast<float *>(c);
  c += p.buf1;
  b.dbuf1 = reinterpret_cast<float *>(c);
  c += p.dbuf1;
  b.halves = p.halves ? reinterpret_cast<float *>(c) : nullptr;
  return b;
}

// The forward call's output and row scales, when the caller passes them.
favor_status check_saved(const favor_desc *g, const void *out, const float *rs, bool &saved) {
  if ((out == nullptr) != (rs == nullptr))
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "out and row_scale are passed together or not at all");
  saved = out != nullptr && !g->no_renormalize;
  if (saved && (!aligned(out, 16) || !aligned(rs, 4)))
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "out must be 16-byte, row_scale 4-byte aligned");
  return FAVOR_OK;
}

// A forward call's workspace offered to a backward call: fwd_op names the call
// that left it (0 none, kOpBidir, kOpCausal, kOpBoth); allowed lists the
// forward calls whose workspace holds what this backward call reads.
favor_status check_forward_ws(const void *fwd_ws, int fwd_op, int allowed_a, int allowed_b) {
  if (fwd_op == 0) {
    if (fwd_ws) return fail(FAVOR_ERR_INVALID_ARGUMENT, "fwd_ws given with fwd_op 0");
    return FAVOR_OK;
  }
  if (fwd_op != allowed_a && fwd_op != allowed_b)
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "fwd_op %d does not name a forward call this "
                                            "backward call can read", fwd_op);
  if (!fwd_ws) return fail(FAVOR_ERR_INVALID_ARGUMENT, "fwd_op %d without fwd_ws", fwd_op);
  if (!aligned(fwd_ws, 256))
    return fail(FAVOR_ERR_INVALID_ARGUMENT, "fwd_ws is not 256-byte aligned");
  return FAVOR_OK;
}

favor_status check_workspace(const void *ws, size_t ws_bytes, size_t need) {
  if (!ws) return fail(FAVOR_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (!aligned(ws, 256)) return fail(FAVOR_ERR_INVALID_ARGUMENT, "workspace is not 256-byte aligned");
  if (ws_bytes < need)
    return fail(FAVOR_ERR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes, need);
  return FAVOR_OK;
}

}  // namespace

extern "C" {

favor_status favor_attn_bidir_backward(const favor_desc *g, const void *Q, const void *K,
                                       const void *V, const float *W, const float *b,
                                       const void *dout, const void *out_fwd,
                                       const float *row_scale, const void *fwd_ws, int32_t fwd_op,
                                       void *dQ, void *dK, void *dV, void *ws, size_t ws_bytes,
                                       hipStream_t stream) {
  FAVOR_TRY(validate(g, kOpBidirBackward));
  bool saved = false;
  FAVOR_TRY(check_saved(g, out_fwd, row_scale, saved));
  FAVOR_TRY(check_forward_ws(fwd_ws, fwd_op, kOpBidir, kOpBoth));
  const BwdPlan p = make_bwd_plan(g, false);
  const bool work = p.total > 0;
  const void *in_ptrs[] = {Q, K, V, W, b, dout, dQ, dK, dV};
  const char *names[] = {"Q", "K", "V", "W", "b", "dout", "dQ", "dK", "dV"};
  for (int i = 0; i < 9; ++i) FAVOR_TRY(check_ptr(in_ptrs[i], names[i], work));
  if (!work) return ok();
  FAVOR_TRY(check_workspace(ws, ws_bytes, p.total));
  const favor::Shape sh = shape_of(g);
  const favor::Dt in = dt_of(g->in_dtype);
  hipStream_t st = stream;
  const BwdBufs w = carve(p, ws);
  hipError_t e;
  // the key side of the forward pass: Buf1 with the W'' fragments and b'', read
  // from the forward call's workspace or recomputed; then the normalised output
  // with each row's reciprocal unless saved
  void *wfr = w.wfr, *frags = w.frags;
  float *bq = w.bq, *part = w.part, *buf1 = w.buf1;
  bool have_frags = false;
  if (fwd_op != 0) {
    const FwdBufs f = carve_fwd(make_plan(g, fwd_op), const_cast<void *>(fwd_ws));
    wfr = f.wfr;
    bq = f.bq;
    frags = f.frags;
    have_frags = true;
    if (fwd_op == kOpBoth) buf1 = f.sum;
    else part = f.part;
  } else {
    favor::LaunchTimer t(favor::kKerKside, st);
    e = favor::launch_kside(sh, in, K, V, W, b, wfr, bq, part, p.rows_per_split, p.nsplit, st);
    if (e != hipSuccess) return device_result(e, "favor_attn_bidir_backward key pass");
  }
  if (sh.renorm && !saved) {
    if (!have_frags) {
      favor::LaunchTimer t(favor::kKerFinalize, st);
      e = favor::launch_finalize(sh, in, part, p.nsplit, frags, st);
      if (e != hipSuccess) return device_result(e, "favor_attn_bidir_backward reduction");
    }
    {
      favor::LaunchTimer t(favor::kKerQside, st);
      e = favor::launch_qside_save(sh, in, Q, wfr, bq, frags, w.out, w.rsave, st);
    }
    if (e != hipSuccess) return device_result(e, "favor_attn_bidir_backward query pass");
  }
  if (buf1 == w.buf1) {
    favor::LaunchTimer t(favor::kKerSumSplits, st);
    e = favor::launch_sum_splits(sh, part, p.nsplit, w.buf1, st);
    if (e != hipSuccess) return device_result(e, "favor_attn_bidir_backward Buf1");
  }
  favor::BwdArgs a{Q,  K,  V,  dout, saved ? out_fwd : w.out, saved ? row_scale : w.rsave,
                   wfr, bq, W, buf1, dQ, dK, dV, w.aux, p.rows_per_split, p.nsplit};
  {
    favor::LaunchTimer t(favor::kKerBwdDq, st);
    e = favor::launch_bwd_dq(sh, in, false, a, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_bidir_backward query gradients");
  {
    favor::LaunchTimer t(favor::kKerBwdAgg, st);
    e = favor::launch_kside_agg(sh, in, Q, dout, W, b, w.aux, w.part2, p.rows_per_split,
                                p.nsplit, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_bidir_backward dBuf1 partials");
  {
    favor::LaunchTimer t(favor::kKerSumSplits, st);
    e = favor::launch_sum_splits(sh, w.part2, p.nsplit, w.dbuf1, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_bidir_backward dBuf1");
  a.state = w.dbuf1;
  {
    favor::LaunchTimer t(favor::kKerBwdDkv, st);
    e = favor::launch_bwd_dkv(sh, in, false, a, st);
  }
  return device_result(e, "favor_attn_bidir_backward key and value gradients");
}

favor_status favor_attn_causal_backward(const favor_desc *g, const void *Q, const void *K,
                                        const void *V, const float *W, const float *b,
                                        const float *state_in, const void *dout,
                                        const void *out_fwd, const float *row_scale,
                                        const void *fwd_ws, int32_t fwd_op,
                                        const float *dstate_out, void *dQ, void *dK, void *dV,
                                        float *dstate_in, void *ws, size_t ws_bytes,
                                        hipStream_t stream) {
  FAVOR_TRY(validate(g, kOpCausalBackward));
  bool saved = false;
  FAVOR_TRY(check_saved(g, out_fwd, row_scale, saved));
  FAVOR_TRY(check_forward_ws(fwd_ws, fwd_op, kOpCausal, kOpBoth));
  const BwdPlan p = make_bwd_plan(g, true);
  const bool work = p.total > 0;
  const bool heads = (long long)g->B * g->H > 0;
  const void *in_ptrs[] = {Q, K, V, W, b, dout, dQ, dK, dV};
  const char *names[] = {"Q", "K", "V", "W", "b", "dout", "dQ", "dK", "dV"};
  for (int i = 0; i < 9; ++i) FAVOR_TRY(check_ptr(in_ptrs[i], names[i], work));
  const void *st_ptrs[] = {state_in, dstate_out, dstate_in};
  const char *st_names[] = {"state_in", "dstate_out", "dstate_in"};
  for (int i = 0; i < 3; ++i)
    if (st_ptrs[i] && !aligned(st_ptrs[i], 16))
      return fail(FAVOR_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", st_names[i]);
  const favor::Shape sh = shape_of(g);
  hipStream_t st = stream;
  hipError_t e;
  if (!work) {
    // no tokens: the state gradient passes through unchanged
    if (heads && dstate_in) {
      {
        favor::LaunchTimer t(favor::kKerSuffixScan, st);
        e = favor::launch_suffix_scan(sh, nullptr, 0, dstate_out, dstate_in, st);
      }
      return device_result(e, "favor_attn_causal_backward state gradient copy");
    }
    return ok();
  }
  FAVOR_TRY(check_workspace(ws, ws_bytes, p.total));
  const favor::Dt in = dt_of(g->in_dtype);
  const BwdBufs w = carve(p, ws);
  // the forward pass as favor_attn_causal runs it: the segment prefixes (plus
  // state_in) with the W'' fragments and b'', read from the forward call's
  // workspace (where its scan left them) or recomputed; then the output with
  // each row's reciprocal unless saved
  void *wfr = w.wfr;
  float *bq = w.bq, *prefix = w.part;
  if (fwd_op != 0) {
    const FwdBufs f = carve_fwd(make_plan(g, fwd_op), const_cast<void *>(fwd_ws));
    wfr = f.wfr;
    bq = f.bq;
    prefix = f.part;
  } else {
    {
      favor::LaunchTimer t(favor::kKerKside, st);
      e = favor::launch_kside(sh, in, K, V, W, b, wfr, bq, prefix, p.rows_per_split, p.nsplit,
                              st);
    }
    if (e != hipSuccess) return device_result(e, "favor_attn_causal_backward segment aggregates");
    {
      favor::LaunchTimer t(favor::kKerSegScan, st);
      e = favor::launch_seg_scan(sh, in, prefix, p.nsplit, state_in, nullptr, nullptr, st);
    }
    if (e != hipSuccess) return device_result(e, "favor_attn_causal_backward segment prefixes");
  }
  if (sh.renorm && !saved) {
    favor::LaunchTimer t(favor::kKerCausal, st);
    e = favor::launch_causal_save(sh, in, Q, K, V, wfr, bq, prefix, w.out, w.rsave,
                                  p.rows_per_split, p.nsplit, w.halves, st);
    if (e != hipSuccess) return device_result(e, "favor_attn_causal_backward forward pass");
  }
  favor::BwdArgs a{Q,  K,  V,  dout, saved ? out_fwd : w.out, saved ? row_scale : w.rsave,
                   wfr, bq, W, prefix, dQ, dK, dV, w.aux, p.rows_per_split, p.nsplit};
  {
    favor::LaunchTimer t(favor::kKerBwdDq, st);
    e = favor::launch_bwd_dq(sh, in, true, a, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_causal_backward query gradients");
  {
    favor::LaunchTimer t(favor::kKerBwdAgg, st);
    e = favor::launch_kside_agg(sh, in, Q, dout, W, b, w.aux, w.part2, p.rows_per_split,
                                p.nsplit, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_causal_backward row aggregates");
  {
    favor::LaunchTimer t(favor::kKerSuffixScan, st);
    e = favor::launch_suffix_scan(sh, w.part2, p.nsplit, dstate_out, dstate_in, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_causal_backward suffix states");
  a.state = w.part2;
  {
    favor::LaunchTimer t(favor::kKerBwdDkv, st);
    e = favor::launch_bwd_dkv(sh, in, true, a, st);
  }
  return device_result(e, "favor_attn_causal_backward key and value gradients");
}

favor_status favor_attn_both_backward(const favor_desc *g, const void *Q, const void *K,
                                      const void *V, const float *W, const float *b,
                                      const float *state_in, const void *dout_bidir,
                                      const void *dout_causal, const void *out_bidir,
                                      const float *row_scale_bidir, const void *out_causal,
                                      const float *row_scale_causal, const void *fwd_ws,
                                      int32_t fwd_op, const float *dstate_out, void *dQ,
                                      void *dK, void *dV, float *dstate_in, void *ws,
                                      size_t ws_bytes, hipStream_t stream) {
  FAVOR_TRY(validate(g, kOpBothBackward));
  bool saved_b = false, saved_c = false;
  FAVOR_TRY(check_saved(g, out_bidir, row_scale_bidir, saved_b));
  FAVOR_TRY(check_saved(g, out_causal, row_scale_causal, saved_c));
  FAVOR_TRY(check_forward_ws(fwd_ws, fwd_op, kOpBoth, kOpBoth));
  const BwdPlan pb = make_bwd_plan(g, false), pc = make_bwd_plan(g, true);
  const bool work = pb.total > 0;
  const bool heads = (long long)g->B * g->H > 0;
  const void *in_ptrs[] = {Q, K, V, W, b, dout_bidir, dout_causal, dQ, dK, dV};
  const char *names[] = {"Q", "K", "V", "W", "b", "dout_bidir", "dout_causal", "dQ", "dK", "dV"};
  for (int i = 0; i < 10; ++i) FAVOR_TRY(check_ptr(in_ptrs[i], names[i], work));
  const void *st_ptrs[] = {state_in, dstate_out, dstate_in};
  const char *st_names[] = {"state_in", "dstate_out", "dstate_in"};
  for (int i = 0; i < 3; ++i)
    if (st_ptrs[i] && !aligned(st_ptrs[i], 16))
      return fail(FAVOR_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", st_names[i]);
  const favor::Shape sh = shape_of(g);
  hipStream_t st = stream;
  hipError_t e;
  if (!work) {
    // no tokens: the state gradient passes through unchanged
    if (heads && dstate_in) {
      {
        favor::LaunchTimer t(favor::kKerSuffixScan, st);
        e = favor::launch_suffix_scan(sh, nullptr, 0, dstate_out, dstate_in, st);
      }
      return device_result(e, "favor_attn_both_backward state gradient copy");
    }
    return ok();
  }
  FAVOR_TRY(check_workspace(ws, ws_bytes, pb.total + pc.total));
  const favor::Dt in = dt_of(g->in_dtype);
  const BwdBufs wb = carve(pb, ws);
  const BwdBufs wc = carve(pc, static_cast<char *>(ws) + pb.total);
  // the forward quantities of favor_attn_both: the segment prefixes (plus
  // state_in), Buf1 as a plain aggregate and as Q-side fragments, W'' and b'',
  // read from the forward call's workspace or recomputed as that call computes
  // them; then each direction's output and row reciprocals unless saved
  void *wfr = wc.wfr, *frags = wb.frags;
  float *bq = wc.bq, *prefix = wc.part, *buf1 = wb.buf1;
  if (fwd_op != 0) {
    const FwdBufs f = carve_fwd(make_plan(g, kOpBoth), const_cast<void *>(fwd_ws));
    wfr = f.wfr;
    bq = f.bq;
    prefix = f.part;
    frags = f.frags;
    buf1 = f.sum;
  } else {
    {
      favor::LaunchTimer t(favor::kKerKside, st);
      e = favor::launch_kside(sh, in, K, V, W, b, wfr, bq, prefix, pc.rows_per_split, pc.nsplit,
                              st);
    }
    if (e != hipSuccess) return device_result(e, "favor_attn_both_backward segment aggregates");
    {
      favor::LaunchTimer t(favor::kKerSegScan, st);
      e = favor::launch_seg_scan(sh, in, prefix, pc.nsplit, state_in, nullptr, frags, st, buf1);
    }
    if (e != hipSuccess) return device_result(e, "favor_attn_both_backward segment prefixes");
  }
  if (sh.renorm && !saved_b) {
    favor::LaunchTimer t(favor::kKerQside, st);
    e = favor::launch_qside_save(sh, in, Q, wfr, bq, frags, wb.out, wb.rsave, st);
    if (e != hipSuccess) return device_result(e, "favor_attn_both_backward bidirectional pass");
  }
  if (sh.renorm && !saved_c) {
    favor::LaunchTimer t(favor::kKerCausal, st);
    e = favor::launch_causal_save(sh, in, Q, K, V, wfr, bq, prefix, wc.out, wc.rsave,
                                  pc.rows_per_split, pc.nsplit, wc.halves, st);
    if (e != hipSuccess) return device_result(e, "favor_attn_both_backward causal pass");
  }
  // bidirectional: dQ of its rows, then dBuf1 = sum of q-hat (x) u~ over every row
  favor::BwdArgs ab{Q,   K,   V,   dout_bidir, saved_b ? out_bidir : wb.out,
                    saved_b ? row_scale_bidir : wb.rsave, wfr, bq, W, buf1, dQ, dK, dV,
                    wb.aux, pb.rows_per_split, pb.nsplit};
  {
    favor::LaunchTimer t(favor::kKerBwdDq, st);
    e = favor::launch_bwd_dq(sh, in, false, ab, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_both_backward bidirectional dQ");
  {
    favor::LaunchTimer t(favor::kKerBwdAgg, st);
    e = favor::launch_kside_agg(sh, in, Q, dout_bidir, W, b, wb.aux, wb.part2, pb.rows_per_split,
                                pb.nsplit, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_both_backward dBuf1 partials");
  {
    favor::LaunchTimer t(favor::kKerSumSplits, st);
    e = favor::launch_sum_splits(sh, wb.part2, pb.nsplit, wb.dbuf1, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_both_backward dBuf1");
  // causal: its dQ added onto the bidirectional one; the suffix aggregates with
  // dBuf1 added (every key sees every row in the bidirectional direction), so
  // one key pass gives dK and dV of both directions
  favor::BwdArgs ac{Q,   K,   V,   dout_causal, saved_c ? out_causal : wc.out,
                    saved_c ? row_scale_causal : wc.rsave, wfr, bq, W, prefix, dQ, dK, dV,
                    wc.aux, pc.rows_per_split, pc.nsplit};
  {
    favor::LaunchTimer t(favor::kKerBwdDq, st);
    e = favor::launch_bwd_dq(sh, in, true, ac, st, /*accumulate=*/true);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_both_backward causal dQ");
  {
    favor::LaunchTimer t(favor::kKerBwdAgg, st);
    e = favor::launch_kside_agg(sh, in, Q, dout_causal, W, b, wc.aux, wc.part2,
                                pc.rows_per_split, pc.nsplit, st);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_both_backward row aggregates");
  {
    favor::LaunchTimer t(favor::kKerSuffixScan, st);
    e = favor::launch_suffix_scan(sh, wc.part2, pc.nsplit, dstate_out, dstate_in, st, wb.dbuf1);
  }
  if (e != hipSuccess) return device_result(e, "favor_attn_both_backward suffix states");
  ac.state = wc.part2;
  {
    favor::LaunchTimer t(favor::kKerBwdDkv, st);
    e = favor::launch_bwd_dkv(sh, in, true, ac, st);
  }
  return device_result(e, "favor_attn_both_backward key and value gradients");
}

}  // extern "C"
