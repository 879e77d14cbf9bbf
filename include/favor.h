/*
 * favor.h - C ABI of libfavor, FAVOR attention (Fast Attention Via Orthogonal
 * Random features, arXiv 2006.03555) for AMD MI355X (gfx950).
 *
 * Every tensor argument is a DEVICE pointer owned by the caller; the library
 * never allocates, frees or retains device memory (scratch is the caller's
 * workspace; the one exception is the static scratch array each GPU holds for
 * favor_attn_both_noalloc). Every call is asynchronous: work is enqueued on `stream`
 * (NULL = the default stream) and nothing waits.
 *
 * Errors: arguments are validated completely before anything is launched. On
 * failure a call returns a non-zero favor_status, writes no output and records
 * a message retrievable with favor_last_error() (per thread). A failed launch
 * returns FAVOR_ERR_DEVICE. Numerical outcomes are not errors: a denominator
 * D-hat that is zero gives IEEE Inf/NaN rows exactly as the formulas do.
 *
 * Layouts (row-major, contiguous, 16-byte aligned):
 *   Q, K, V, out   [B][H][L][d]      in_dtype (out: out_dtype)
 *   W              [H][M][d]  float  rows omega_m of the random-feature matrix
 *   b              [H][M]     float  phases b_m
 *   X' (features)  [B][H][L][M]      out_dtype
 *   state          [B][H][M][d+1] float, column d holds sum_j K'_j (the "1" column)
 * One draw (W, b) per head is shared by every batch entry.
 *
 * Supported: d = 64; M a multiple of 16 from 16 to 256 (the kernels work on M
 * rounded up to 64, 128 or 256 rows, the rows past M being padding whose
 * features are zero, so every array above keeps M; the causal scan with F32
 * inputs and M > 128 runs as two passes over the feature halves);
 * 0 <= L <= 2^30 (any length, ragged tails handled; L = 0 is a no-op); B, H >= 0,
 * B*H <= 65535; in_dtype F32 or BF16; out_dtype F32 or BF16. F32 inputs use
 * fp32 matrix cores and an accurately rounded cosine; BF16 inputs use bf16
 * matrix cores with fp32 accumulation, the hardware cosine and bf16 features.
 */
#ifndef FAVOR_H
#define FAVOR_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__)
#define FAVOR_API __attribute__((visibility("default")))
#else
#define FAVOR_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* The HIP runtime's stream handle (the same declaration as in
 * hip/hip_runtime_api.h, so either header may come first). NULL is the default
 * stream. */
struct ihipStream_t;
typedef struct ihipStream_t *hipStream_t;

typedef enum {
  FAVOR_OK = 0,
  FAVOR_ERR_INVALID_ARGUMENT = 1,  /* null/misaligned pointer, negative size, bad enum */
  FAVOR_ERR_UNSUPPORTED = 2,       /* valid but not implemented (d, M, dtype combo)    */
  FAVOR_ERR_WORKSPACE_TOO_SMALL = 3,
  FAVOR_ERR_DEVICE = 4             /* a HIP launch or runtime call failed               */
} favor_status;

typedef enum { FAVOR_F32 = 0, FAVOR_BF16 = 1 } favor_dtype;

typedef enum {
  FAVOR_RF_ORTHO_CHI = 0,   /* R-ORF blocks, rows scaled by independent chi_d norms (default) */
  FAVOR_RF_ORTHO_FIXED = 1, /* R-ORF blocks, every row scaled to norm sqrt(d)                  */
  FAVOR_RF_IID = 2,         /* unstructured i.i.d. N(0, I_d) rows                              */
  FAVOR_RF_HADAMARD = 3,    /* H-ORF blocks sqrt(d) H D3 H D2 H D1 (Sec. 2.4 (2))              */
  FAVOR_RF_GIVENS = 4       /* G-ORF blocks sqrt(d) G_1 ... G_K, K = 2 d log2 d (Sec. 2.4 (2)) */
} favor_rf_kind;

/* Feature kernel (Sec. 2.2, Eq. interesting):
 *   SOFTMAX  Gaussian-kernel features for softmax attention (Sec. 2.3):
 *            phi(x)_m = exp(||x~||^2 / 2) sqrt(2/M) cos(omega_m . x~ + b_m)
 *   RELU     generalized attention with f = ReLU, g = h = 1 (the paper's
 *            "Performer-ReLU", App. B): phi(x)_m = ReLU(omega_m . x~) / sqrt(M)
 *            + kernel_eps; the phases b are not used. */
typedef enum { FAVOR_KERNEL_SOFTMAX = 0, FAVOR_KERNEL_RELU = 1 } favor_kernel;

typedef struct {
  int32_t B, H, L, d, M;
  favor_dtype in_dtype;     /* Q, K, V (and X for the feature map) */
  favor_dtype out_dtype;    /* out, X'                             */
  float input_scale;        /* x~ = input_scale * x. d^-1/4 evaluates the paper's
                               exp(Q K^T / sqrt d) (Sec. 2.1) on the given Q, K.  */
  float denom_eps;          /* added to D-hat before dividing; 0 = Algorithm 1      */
  int32_t chunk;            /* causal chunk length T: tokens per step of the
                               prefix-sum scan (Sec. 2.5.1): 64 (four 16-token
                               matrix-core blocks in the intra-chunk product) or,
                               for bf16 inputs, 32; 0 = library default: 32 for
                               bf16 inputs with M <= 128, else 64. Other values,
                               and 32 with fp32 inputs in a causal call, return
                               FAVOR_ERR_UNSUPPORTED. The result is the same sum
                               in another grouping                                 */
  int32_t kernel;           /* favor_kernel; 0 (zero-initialised) = SOFTMAX         */
  int32_t no_renormalize;   /* 0 = out = Buf3 / (buf4 + denom_eps) (Algorithm 1);
                               1 = out = Buf3 = Q' K'^T V ("renormalize_attention"
                               off, App. B; denom_eps is then unused)             */
  float kernel_eps;         /* RELU: added to every feature (App. B kernel_epsilon,
                               default 1e-3); ignored for SOFTMAX                  */
  int32_t segment;          /* causal: tokens per segment, the stretch of the
                               sequence one workgroup scans chunk by chunk from
                               the aggregate of the segments before it (a multiple
                               of 64, at most 2^30); 0 = library default (about one
                               workgroup per compute unit with T = 64, two with
                               T = 32)                                             */
} favor_desc;

/*
 * favor_orf_draw - draw the random-feature matrix W [n_heads][M][d] and phases
 * b [n_heads][M] (Sec. 2.3 for the Gaussian-kernel features, Sec. 2.4 for the
 * orthogonal R-ORF construction).
 *
 * For each head h and block k < ceil(M/d): a d x d matrix of N(0,1) entries has
 * its rows orthonormalised in order by Gram-Schmidt (the orthogonal factor
 * with positive triangular diagonal); row m = k d + r is scaled by rho_m (kind
 * CHI: the norm of an independent N(0, I_d) vector; FIXED: sqrt(d)); the first
 * M stacked rows are kept. IID kind keeps the raw Gaussian rows. b_m = 2 pi u_m.
 * HADAMARD: block k = sqrt(d) H D3 H D2 H D1 with the normalised Sylvester-
 * Hadamard matrix H[i][j] = (-1)^popcount(i & j) / sqrt(d) and diagonals D_t of
 * signs: element (3 k + t) d + c of purpose 3 is +1 when its 32-bit word is
 * below 2^31, else -1. GIVENS: block k = sqrt(d) G_1 ... G_K, K = 2 d log2 d;
 * G_t rotates the (i, j) plane by theta (row vectors: v_i <- cos v_i + sin v_j,
 * v_j <- -sin v_i + cos v_j), from words x0, x1, x2 of call k K + t of purpose 4:
 * i = (x0 d) >> 32, j' = (x1 (d - 1)) >> 32, j = j' + [j' >= i],
 * theta = 2 pi (x2 + 0.5) 2^-32. Both are orthogonal with rows of norm sqrt(d).
 *
 * Random numbers: Philox4x64-10 (Salmon et al., SC'11), key (seed, 0), counter
 * (i, h, purpose, 0) with purpose 0 = Gaussian blocks, 1 = chi-norm Gaussians,
 * 2 = phases, 3 = Hadamard signs, 4 = Givens rotations. Call i yields four 64-bit words w0..w3, i.e. eight 32-bit words
 * x[2j] = low(wj), x[2j+1] = high(wj); stream element n is word n % 8 of call
 * n / 8; u = (x + 0.5) 2^-32; Gaussians by Box-Muller from uniform pairs
 * (u[2p], u[2p+1]): sqrt(-2 ln u[2p]) * (cos, sin)(2 pi u[2p+1]). Gaussian
 * element of block k, row r, column c: n = (k d + r) d + c; chi vector of row
 * m: n = m d + c; phase of row m: n = m. Uniforms, Gaussians and phases are
 * computed in fp32; the orthogonalisation, norms and scaling in fp64.
 *
 * Requires n_heads >= 0, d = 64, 1 <= M <= 4096. W, b: device, fp32; W 16-byte
 * aligned, b 4-byte aligned.
 */
FAVOR_API favor_status favor_orf_draw(uint64_t seed, int32_t n_heads, int32_t M, int32_t d,
                            favor_rf_kind kind, float *W, float *b, hipStream_t stream);

/*
 * favor_feature_map - X' = D_X X-hat, the paper's Q' = D_Q Q-hat (Sec. 2.3,
 * Eqs. dqdk and qkprime) with Gaussian-kernel features (c = sqrt 2, f = cos):
 *   X'[l][m] = exp(||x~_l||^2 / 2) * sqrt(2/M) * cos(omega_m . x~_l + b_m),
 *   x~_l = input_scale * X[l];
 * with g->kernel = FAVOR_KERNEL_RELU the generalized-attention features
 *   X'[l][m] = max(omega_m . x~_l, 0) / sqrt(M) + g->kernel_eps   (b unused).
 * X [B][H][L][d] in g->in_dtype -> Xprime [B][H][L][M] in g->out_dtype.
 * g->denom_eps, g->chunk and g->no_renormalize are ignored.
 */
FAVOR_API favor_status favor_feature_map(const favor_desc *g, const void *X, const float *W,
                               const float *b, void *Xprime, hipStream_t stream);

/*
 * favor_workspace_size - bytes of device workspace favor_attn_bidir (causal = 0),
 * favor_attn_causal (causal = 1, or any value other than 0 and 2) or
 * favor_attn_both (causal = 2) needs for descriptor g; 0 if g is invalid.
 * The workspace must be 256-byte aligned; its contents on entry do not matter.
 */
FAVOR_API size_t favor_workspace_size(const favor_desc *g, int causal);

/*
 * favor_attn_bidir - bidirectional FAVOR (Sec. 2.5, Algorithm 1):
 *   C = [V 1_L], Buf1 = K'^T C (M x (d+1)), Buf2 = Q' Buf1,
 *   out = diag(buf4 + denom_eps)^-1 Buf3 with [Buf3 buf4] = Buf2,
 * where Q', K' are the feature maps of favor_feature_map for g->kernel. With
 * g->no_renormalize = 1 the result is Buf3 itself. The L x L matrix Q' K'^T and
 * the L x M features are never stored. Deterministic (no atomics).
 */
FAVOR_API favor_status favor_attn_bidir(const favor_desc *g, const void *Q, const void *K,
                              const void *V, const float *W, const float *b, void *out,
                              void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * favor_attn_bidir_save - favor_attn_bidir that also writes, for the backward
 * pass, row_scale [B][H][L] fp32 (nullable): each row's 1 / (buf4 + denom_eps)
 * in units of the features without D_Q sqrt(2/M). Needs out_dtype == in_dtype;
 * row_scale is not written without renormalisation.
 */
FAVOR_API favor_status favor_attn_bidir_save(const favor_desc *g, const void *Q, const void *K,
                                             const void *V, const float *W, const float *b,
                                             void *out, float *row_scale, void *ws,
                                             size_t ws_bytes, hipStream_t stream);

/*
 * favor_attn_causal - unidirectional FAVOR by prefix sums (Sec. 2.5.1, Eq.
 * cumsum): row i of the result is (G^PS_i)^T Q'_i normalised as in Algorithm 1
 * (not normalised with g->no_renormalize = 1; features as for favor_attn_bidir),
 * G^PS_i = S_0 + sum_{j <= i} K'_j C_j^T (keys up to and including i). The
 * prefix tensor is never stored: workgroups scan chunks of tokens carrying an
 * M x (d+1) fp32 state.
 * state_in  (nullable) [B][H][M][d+1] fp32: S_0, the aggregate of earlier tokens.
 * state_out (nullable) [B][H][M][d+1] fp32: receives S_0 + sum over all L tokens,
 * so a long sequence can be processed in pieces. Deterministic (no atomics).
 */
FAVOR_API favor_status favor_attn_causal(const favor_desc *g, const void *Q, const void *K,
                               const void *V, const float *W, const float *b, void *out,
                               const float *state_in, float *state_out,
                               void *ws, size_t ws_bytes, hipStream_t stream);

/* favor_attn_causal_save - favor_attn_causal that also writes row_scale, as
 * favor_attn_bidir_save does. */
FAVOR_API favor_status favor_attn_causal_save(const favor_desc *g, const void *Q,
                                              const void *K, const void *V, const float *W,
                                              const float *b, void *out, const float *state_in,
                                              float *state_out, float *row_scale, void *ws,
                                              size_t ws_bytes, hipStream_t stream);

/*
 * favor_attn_both - both directions over the same Q, K, V in one call: the
 * results of favor_attn_bidir (out_bidir) and favor_attn_causal (out_causal,
 * with state_in / state_out as there; state_in affects the causal output only).
 * The bidirectional Buf1 = K'^T [V 1] is the causal aggregate over the whole
 * sequence (G^PS_L of Eq. cumsum), so one pass over the keys serves both:
 * the key features are built once per segment and the segment scan also
 * returns the total. Workspace: favor_workspace_size(g, 2). Deterministic.
 * row_scale_bidir, row_scale_causal (nullable): as for favor_attn_bidir_save.
 */
FAVOR_API favor_status favor_attn_both(const favor_desc *g, const void *Q, const void *K,
                                       const void *V, const float *W, const float *b,
                                       void *out_bidir, void *out_causal,
                                       const float *state_in, float *state_out,
                                       float *row_scale_bidir, float *row_scale_causal,
                                       void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * favor_attn_both_noalloc - favor_attn_both for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same arguments without ws / ws_bytes, and the same
 * results. The workspace is a static array of favor_noalloc_scratch_bytes()
 * bytes (32 MiB) that each GPU the library runs on holds from the first load of
 * the library's code there until the process ends; nothing is allocated or
 * freed by the call. A call whose favor_workspace_size(g, 2) exceeds it returns
 * FAVOR_ERR_WORKSPACE_TOO_SMALL and launches nothing. Every call on one GPU uses
 * that GPU's one array: calls that overlap on one GPU (concurrent streams,
 * threads) race on it and must be serialised by the caller. The array needs no
 * clearing (the kernels overwrite what they read). The current device is the
 * one whose array is used (the stream must belong to it).
 */
FAVOR_API favor_status favor_attn_both_noalloc(const favor_desc *g, const void *Q,
                                               const void *K, const void *V, const float *W,
                                               const float *b, void *out_bidir,
                                               void *out_causal, const float *state_in,
                                               float *state_out, float *row_scale_bidir,
                                               float *row_scale_causal, hipStream_t stream);

/* Size in bytes of favor_attn_both_noalloc's static scratch array. */
FAVOR_API size_t favor_noalloc_scratch_bytes(void);

/*
 * Backward pass (the paper trains through FAVOR and benchmarks its backward
 * pass, Sec. 4.1): gradients of a loss with respect to Q, K, V given
 * dout = dLoss/dout, for the same descriptor, inputs and features as the
 * forward call. Algorithm 1 and Eq. cumsum are taken in reverse:
 *   [dBuf3 dbuf4] from the normalisation (dBuf3 = dout / (buf4 + eps), dbuf4 =
 *   -(dout . out) / (buf4 + eps); dout and 0 without renormalisation),
 *   dQ' = dBuf2 Buf1^T, dBuf1 = Q'^T dBuf2, dK' = C dBuf1^T, dV = (K' dBuf1)[:, :d],
 * then through the feature maps. The forward quantities are recomputed (nothing
 * from the forward call is needed); W and b receive no gradient.
 * dout, dQ, dK, dV: [B][H][L][d] in in_dtype; out_dtype must equal in_dtype
 * (FAVOR_ERR_UNSUPPORTED otherwise). Every supported M; with fp32 inputs the
 * gradient kernels take 128 (bidirectional) or 64 (causal) features at a time
 * and add the slices' parts into dQ, dK, dV in a fixed order. Deterministic
 * (no atomics). dQ, dK, dV are written in full (ragged tails included).
 * Workspace: favor_backward_workspace_size(g, causal) bytes, 256-byte aligned
 * (causal: 0 bidirectional, 1 causal, 2 both directions in one call).
 * out and row_scale (both nullable, both or neither): the forward call's output
 * and row_scale for the same inputs, features and descriptor; given, the backward
 * skips recomputing them (their recomputation otherwise runs inside the call).
 * Not read without renormalisation.
 * fwd_ws, fwd_op: the workspace a forward call left behind and which call that
 * was (1 favor_attn_bidir or favor_attn_bidir_save, 2 favor_attn_causal or
 * favor_attn_causal_save, 3 favor_attn_both), or NULL and 0. The forward call must have had the same
 * descriptor, K, V, W, b (and, causal, the same state_in), completed in stream
 * order before, and its workspace must be unchanged since. Given, the backward
 * reads Buf1 (bidirectional: 1 or 3) or the segment prefixes (causal: 2 or 3),
 * the W'' fragments and b'' from it instead of recomputing them; fwd_ws is only
 * read. Other fwd_op values, or fwd_ws without fwd_op, are
 * FAVOR_ERR_INVALID_ARGUMENT.
 */
FAVOR_API size_t favor_backward_workspace_size(const favor_desc *g, int causal);

/* favor_attn_bidir_backward - gradients of favor_attn_bidir. */
FAVOR_API favor_status favor_attn_bidir_backward(const favor_desc *g, const void *Q,
                                                 const void *K, const void *V, const float *W,
                                                 const float *b, const void *dout,
                                                 const void *out, const float *row_scale,
                                                 const void *fwd_ws, int32_t fwd_op,
                                                 void *dQ, void *dK, void *dV, void *ws,
                                                 size_t ws_bytes, hipStream_t stream);

/*
 * favor_attn_causal_backward - gradients of favor_attn_causal (Eq. cumsum):
 * dQ'_i = G^PS_i dBuf2_i with the prefix aggregate, and with the suffix
 * R_j = dstate_out + sum_{i >= j} Q'_i dBuf2_i^T: dK'_j = R_j C_j,
 * dV_j = (R_j^T K'_j)[:d]. state_in (nullable) as in the forward call;
 * dstate_out (nullable) [B][H][M][d+1] fp32: the gradient reaching state_out;
 * dstate_in (nullable) [B][H][M][d+1] fp32: receives the gradient of state_in
 * (R_1), so a sequence processed in pieces is differentiated piece by piece
 * from the last. L = 0 copies dstate_out (or zeros) to dstate_in.
 */
FAVOR_API favor_status favor_attn_causal_backward(const favor_desc *g, const void *Q,
                                                  const void *K, const void *V, const float *W,
                                                  const float *b, const float *state_in,
                                                  const void *dout, const void *out,
                                                  const float *row_scale, const void *fwd_ws,
                                                  int32_t fwd_op, const float *dstate_out,
                                                  void *dQ, void *dK,
                                                  void *dV, float *dstate_in, void *ws,
                                                  size_t ws_bytes, hipStream_t stream);

/*
 * favor_attn_both_backward - gradients of favor_attn_both: of a loss that depends
 * on both outputs, given dout_bidir and dout_causal (Algorithm 1 and Eq. cumsum
 * in reverse, as the two calls above). dQ, dK, dV receive the sums of the two
 * directions' gradients. The key side is one pass: the bidirectional dBuf1 is
 * the aggregate every key of the sequence sees, so it is added to each key's
 * causal suffix R_j before dK'_j = R_j C_j and dV_j = (R_j^T K'_j)[:d]; dQ of the
 * causal direction is added onto the bidirectional one (bf16: one more
 * rounding). out_bidir with row_scale_bidir, and out_causal with
 * row_scale_causal: each pair nullable, both or neither, as the forward call
 * saved them. fwd_ws, fwd_op: a favor_attn_both call's workspace and 3, or NULL
 * and 0. state_in, dstate_out, dstate_in as for favor_attn_causal_backward
 * (dstate_in receives the causal direction's state gradient only; the
 * bidirectional output does not depend on state_in). Workspace:
 * favor_backward_workspace_size(g, 2) bytes, 256-byte aligned. Other
 * conditions and errors as for the two calls above.
 */
FAVOR_API favor_status favor_attn_both_backward(const favor_desc *g, const void *Q,
                                                const void *K, const void *V, const float *W,
                                                const float *b, const float *state_in,
                                                const void *dout_bidir, const void *dout_causal,
                                                const void *out_bidir,
                                                const float *row_scale_bidir,
                                                const void *out_causal,
                                                const float *row_scale_causal,
                                                const void *fwd_ws, int32_t fwd_op,
                                                const float *dstate_out, void *dQ, void *dK,
                                                void *dV, float *dstate_in, void *ws,
                                                size_t ws_bytes, hipStream_t stream);

/* Host-only validation of a descriptor for an operation (0 feature map,
 * 1 bidirectional, 2 causal, 3 both, 4 bidirectional backward, 5 causal
 * backward, 6 backward of both directions); launches nothing and touches no
 * device. */
FAVOR_API favor_status favor_validate_desc(const favor_desc *g, int op);

FAVOR_API const char *favor_status_string(favor_status s);

/* Detail of the last failure on the calling thread ("" if none). */
FAVOR_API const char *favor_last_error(void);

/*
 * Per-kernel timing for benchmarks. While enabled, every kernel the library
 * launches is bracketed by two HIP events recorded on the launch stream (the
 * events come from a pool; nothing is allocated on the device). Reading
 * waits for the recorded events and returns, for kernel id k, the summed
 * milliseconds and launch count since the last reset. Ids run from 0 to
 * favor_timing_num_kernels() - 1; favor_timing_kernel_name(k) names them.
 * Not thread-safe with respect to concurrent launches from several threads.
 */
FAVOR_API favor_status favor_timing_enable(int on);
FAVOR_API favor_status favor_timing_reset(void);
FAVOR_API int32_t favor_timing_num_kernels(void);
FAVOR_API const char *favor_timing_kernel_name(int32_t k);
FAVOR_API favor_status favor_timing_read(int32_t k, double *ms, int64_t *count);

/*
 * Measurement probes for roofline reports (not part of the method): one launch
 * of 512 workgroups of 256 threads (two per CU) in which every wave issues
 * iters x 8 independent v_mfma_f32_16x16x32_bf16 (kind 0), every lane
 * evaluates iters x 8 independent hardware cosines (kind 1), or every lane
 * projects iters tokens onto M = 256 H-ORF rows the structured way, four blocks
 * of three 64-point Walsh-Hadamard transforms with sign flips in registers
 * (kind 2; the O(M log d) apply of Sec. 2.4, against which the dense matrix-core
 * projection of kind 0 is compared). Timing a launch and dividing
 * favor_probe_work(kind, iters) (FLOP for kind 0, cosines for kind 1, tokens
 * for kind 2) by its duration gives the rate this GPU reaches. sink: a device
 * buffer of at least 512 floats (never written for the probe's inputs).
 */
FAVOR_API favor_status favor_probe(int32_t kind, int32_t iters, float *sink, hipStream_t stream);
FAVOR_API double favor_probe_work(int32_t kind, int32_t iters);

/* ABI version of this header; bumped on any incompatible change. */
FAVOR_API int32_t favor_abi_version(void);

#define FAVOR_ABI_VERSION 7

#ifdef __cplusplus
}
#endif

#endif /* FAVOR_H */
