"""FAVOR attention in fp64, step by step as the paper states it.

Test infrastructure only (see ``oracle/__init__``).

Shapes: Q, K, V are [..., L, d] (leading axes are batch and head); W is
[H, M, d] and b is [H, M], one draw per head shared across the batch. When the
inputs carry a head axis (axis -3) W and b broadcast over it.

Readings of points the paper leaves open:
  * Gaussian-kernel features use omega ~ N(0, I_d) acting on the scaled input
    x~ = s x (s = input_scale; s = d^-1/4 gives the paper's exp(QK^T / sqrt d)).
    With s = d^-1/4 this is the same as omega ~ N(0, sigma^-2 I) on raw x with
    sigma = d^1/4; the printed "N(0, sigma^2 I)" contradicts Bochner's theorem
    and the paper's own Theorem 1, which uses N(0, I_d) on d^-1/4-scaled inputs.
  * "ortho_scaling = 0.0" (App. B) is read as chi_d-distributed row norms, which
    keeps each row's Gaussian marginal (Sec. 2.4) and so stays unbiased.
  * The stabiliser is added to the denominator D-hat; 0 reproduces Algorithm 1.
  * Algorithm 1's "Result in R^{L x L}" is read as R^{L x d}; the prefix-sum
    row is (G^PS_i)^T Q'_i in R^{d+1}; the cumsum index runs over j.
  * Generalized attention with f = ReLU (Sec. 2.2, Eq. interesting; the
    "Performer-ReLU" default of App. B): g = h = 1 (no D_Q, D_K), c = 1, b = 0,
    and the kernel stabiliser ("kernel_epsilon", App. B) added to every feature:
    phi(x)_m = ReLU(omega_m . x~) / sqrt(M) + kernel_eps. The same R-ORF rows W
    serve both kernels; the phases b are not used by ReLU features.
  * "renormalize_attention" (App. B) switches the final D-hat^-1 of Algorithm 1:
    off returns Buf3 = Q' K'^T V itself.
"""
import numpy as np

from . import philox

RF_ORTHO_CHI = 0     # R-ORF blocks, rows scaled by independent chi_d norms
RF_ORTHO_FIXED = 1   # R-ORF blocks, rows scaled to sqrt(d)
RF_IID = 2           # unstructured Gaussian rows
RF_HADAMARD = 3      # H-ORF blocks sqrt(d) H D3 H D2 H D1 (Sec. 2.4)
RF_GIVENS = 4        # G-ORF blocks sqrt(d) G_1 ... G_K, K = 2 d log2 d rotations (Sec. 2.4)

KERNEL_SOFTMAX = 0   # Gaussian-kernel features (cos), softmax attention
KERNEL_RELU = 1      # generalized attention with f = ReLU


def gram_schmidt_rows(G):
    """Orthonormalise the rows of a square matrix in order (Sec. 2.4, R-ORFs).

    Modified Gram-Schmidt in fp64: row i loses its components along rows
    0..i-1 already orthonormalised, then is normalised. The result is the
    unique orthogonal factor whose triangular factor has a positive diagonal.
    """
    G = np.array(G, dtype=np.float64)
    n = G.shape[0]
    Qr = np.zeros_like(G)
    for i in range(n):
        r = G[i].copy()
        for j in range(i):
            r -= np.dot(Qr[j], r) * Qr[j]
        Qr[i] = r / np.linalg.norm(r)
    return Qr


def hadamard(d):
    """Normalised Sylvester-Hadamard matrix: H[i][j] = (-1)^popcount(i & j) / sqrt(d)."""
    i = np.arange(d)
    bits = np.bitwise_and.outer(i, i)
    par = np.zeros_like(bits)
    while np.any(bits):
        par ^= bits & 1
        bits >>= 1
    return (1.0 - 2.0 * par) / np.sqrt(d)


def hadamard_signs(seed, head, blk, d):
    """The three Rademacher diagonals of block blk: element (3 blk + t) d + c of
    stream SIGNS is +1 when its 32-bit word is below 2^31, else -1. Shape [3, d]."""
    n = (3 * blk + 3) * d
    w = philox.words32(seed, head, philox.PURPOSE_SIGNS, n)[3 * blk * d:].reshape(3, d)
    return np.where(w < np.uint64(1 << 31), 1.0, -1.0)


def hadamard_block(seed, head, blk, d):
    """H-ORF block (Sec. 2.4 (2); the random Hadamard construction it cites):
    sqrt(d) H D3 H D2 H D1 with Rademacher diagonals D_t. Orthogonal rows of norm sqrt(d)."""
    H = hadamard(d)
    D = hadamard_signs(seed, head, blk, d)
    return np.sqrt(d) * (H * D[2]) @ (H * D[1]) @ (H * D[0])


def givens_params(seed, head, blk, d, K):
    """Rotation t of block blk from call blk K + t of stream GIVENS (words x0, x1, x2):
    i = floor(x0 d / 2^32), j' = floor(x1 (d - 1) / 2^32), j = j' + [j' >= i],
    theta = 2 pi (x2 + 0.5) 2^-32."""
    n = (blk * K + K) * 8
    w = philox.words32(seed, head, philox.PURPOSE_GIVENS, n)[blk * K * 8:].reshape(K, 8)
    i = (w[:, 0] * np.uint64(d)) >> np.uint64(32)
    jp = (w[:, 1] * np.uint64(d - 1)) >> np.uint64(32)
    j = jp + (jp >= i)
    theta = 2.0 * np.pi * (w[:, 2].astype(np.float64) + 0.5) * 2.0 ** -32
    return i.astype(np.int64), j.astype(np.int64), theta


def givens_count(d):
    """Rotations per G-ORF block: 2 d log2 d."""
    return 2 * d * int(round(np.log2(d)))


def givens_block(seed, head, blk, d, K=None):
    """G-ORF block (Sec. 2.4 (2); Kac's random walk of the Givens construction it
    cites): sqrt(d) G_1 G_2 ... G_K, G_t the rotation by theta_t in the (i_t, j_t)
    plane (G[i][i] = G[j][j] = cos, G[i][j] = -sin, G[j][i] = sin); K = 2 d log2 d
    rotations, O(M log d) numbers for M rows as the paper counts (d log2 d leaves the
    entries visibly non-Gaussian, fourth moment ~5.5; twice that mixes them, ~3.0)."""
    if K is None:
        K = givens_count(d)
    i, j, theta = givens_params(seed, head, blk, d, K)
    B = np.eye(d)
    for t in range(K):
        c, s = np.cos(theta[t]), np.sin(theta[t])
        bi, bj = B[:, i[t]].copy(), B[:, j[t]].copy()
        B[:, i[t]] = c * bi + s * bj       # row vector v <- v G_t
        B[:, j[t]] = -s * bi + c * bj
    return np.sqrt(d) * B


def orf_draw(seed, n_heads, M, d, kind=RF_ORTHO_CHI, heads=None):
    """Random-feature matrix W [H, M, d] and phases b [H, M] (Secs. 2.3-2.4).

    heads: optional list of head indices; W and b then hold only those heads, in
    that order (each head is drawn from its own streams, so a head's rows do
    not depend on the others).

    For each head and each d x d block k < ceil(M/d): a Gaussian block (Philox
    stream, purpose ORF, row-major element index (k d + r) d + c) has its rows
    orthonormalised by Gram-Schmidt; row m = k d + r is then scaled by rho_m,
    the norm of an independent N(0, I_d) vector (purpose CHI, elements
    m d .. m d + d - 1). The blocks are stacked and the first M rows kept.
    b_m = 2 pi u_m with u_m uniform (purpose PHASE, element m).
    FIXED kind uses rho = sqrt(d); IID kind keeps the raw Gaussian rows.
    HADAMARD and GIVENS kinds use the structured orthogonal blocks (rows of norm
    sqrt(d)) in place of the Gram-Schmidt ones.
    """
    nblk = -(-M // d)
    hs = list(range(n_heads)) if heads is None else list(heads)
    W = np.zeros((len(hs), M, d), dtype=np.float64)
    b = np.zeros((len(hs), M), dtype=np.float64)
    for i, h in enumerate(hs):
        g = philox.gaussians(seed, h, philox.PURPOSE_ORF, nblk * d * d).reshape(nblk, d, d)
        rows = []
        for k in range(nblk):
            if kind == RF_IID:
                rows.append(g[k])
            elif kind == RF_HADAMARD:
                rows.append(hadamard_block(seed, h, k, d))
            elif kind == RF_GIVENS:
                rows.append(givens_block(seed, h, k, d))
            else:
                rows.append(gram_schmidt_rows(g[k]))
        Wh = np.concatenate(rows, axis=0)[:M]
        if kind == RF_ORTHO_CHI:
            chi = philox.gaussians(seed, h, philox.PURPOSE_CHI, M * d).reshape(M, d)
            rho = np.sqrt(np.sum(chi * chi, axis=1))
            Wh = Wh * rho[:, None]
        elif kind == RF_ORTHO_FIXED:
            Wh = Wh * np.sqrt(d)
        W[i] = Wh
        b[i] = 2.0 * np.pi * philox.uniforms(seed, h, philox.PURPOSE_PHASE, M)
    return W, b


def _per_head(W, b, X):
    """Broadcast W [H,M,d], b [H,M] against X [..., H, L, d]."""
    W = np.asarray(W, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if X.ndim >= 3:
        return W, b[..., None, :]          # W [H,M,d], b [H,1,M]
    return W[0], b[0][None, :]             # single head, X [L, d]


def feature_map(X, W, b, input_scale):
    """X' = D_X X-hat (Sec. 2.3, Eqs. dqdk and qkprime), X [..., L, d] -> [..., L, M].

    x~ = s x; X-hat = sqrt(2/M) cos(W x~ + b) (Gaussian-kernel features, c = sqrt 2,
    f = cos); D_X = diag(exp(||x~||^2 / 2)), which is the paper's exp(||x||^2 / r)
    with r = 2 sqrt(d) when s = d^-1/4.
    """
    X = np.asarray(X, dtype=np.float64)
    W, bb = _per_head(W, b, X)
    M = W.shape[-2]
    Xs = input_scale * X
    proj = np.matmul(Xs, np.swapaxes(W, -1, -2))                # [..., L, M]
    Xhat = np.sqrt(2.0 / M) * np.cos(proj + bb)
    D = np.exp(0.5 * np.sum(Xs * Xs, axis=-1))                  # [..., L]
    return D[..., None] * Xhat


def feature_map_relu(X, W, input_scale, kernel_eps=1e-3):
    """Generalized-attention features with f = ReLU (Sec. 2.2, Eqs. interesting and
    qkprime with g = h = 1, c = 1, b = 0): X [..., L, d] -> [..., L, M],
    phi(x)_m = ReLU(omega_m . x~) / sqrt(M) + kernel_eps, x~ = s x.
    """
    X = np.asarray(X, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    if X.ndim < 3:
        W = W[0]
    M = W.shape[-2]
    proj = np.matmul(input_scale * X, np.swapaxes(W, -1, -2))   # [..., L, M]
    return np.maximum(proj, 0.0) / np.sqrt(M) + kernel_eps


def features(X, W, b, input_scale, kernel=KERNEL_SOFTMAX, kernel_eps=1e-3):
    """Q' or K' for the chosen kernel (softmax: feature_map; ReLU: feature_map_relu)."""
    if kernel == KERNEL_RELU:
        return feature_map_relu(X, W, input_scale, kernel_eps)
    return feature_map(X, W, b, input_scale)


def _with_ones(V):
    """C = [V 1_L] (Algorithm 1)."""
    V = np.asarray(V, dtype=np.float64)
    ones = np.ones(V.shape[:-1] + (1,), dtype=np.float64)
    return np.concatenate([V, ones], axis=-1)


def attn_bidir_features(Qp, Kp, V, denom_eps=0.0, renormalize=True):
    """Algorithm 1, bidirectional branch, given Q' and K'.

    Buf1 = K'^T C, Buf2 = Q' Buf1, [Buf3 buf4] = Buf2, return diag(buf4)^-1 Buf3
    (Buf3 itself when renormalize is off).
    """
    C = _with_ones(V)
    d = C.shape[-1] - 1
    Buf1 = np.matmul(np.swapaxes(Kp, -1, -2), C)                # [..., M, d+1]
    Buf2 = np.matmul(Qp, Buf1)                                  # [..., L, d+1]
    Buf3, buf4 = Buf2[..., :d], Buf2[..., d]
    if not renormalize:
        return Buf3
    return Buf3 / (buf4 + denom_eps)[..., None]


def attn_bidir(Q, K, V, W, b, input_scale, denom_eps=0.0, kernel=KERNEL_SOFTMAX,
               kernel_eps=1e-3, renormalize=True):
    """Bidirectional FAVOR (Sec. 2.5, Algorithm 1)."""
    Qp = features(Q, W, b, input_scale, kernel, kernel_eps)
    Kp = features(K, W, b, input_scale, kernel, kernel_eps)
    return attn_bidir_features(Qp, Kp, V, denom_eps, renormalize)


def attn_causal_features(Qp, Kp, V, denom_eps=0.0, state_in=None, renormalize=True):
    """Unidirectional FAVOR by sequential prefix aggregation (Sec. 2.5.1, Eq. cumsum;
    the O(Md + Ld + ML)-space variant of Sec. 2.6).

    For i = 1..L: G^PS_i = G^PS_{i-1} + K'_i C_i^T, Buf2_i = (G^PS_i)^T Q'_i;
    then normalise as in Algorithm 1. Vectorised over the leading axes only.
    Returns (out [..., L, d], G^PS_L [..., M, d+1]); state_in, if given, is the
    aggregate carried in from earlier tokens (G^PS_0).
    """
    C = _with_ones(V)
    L = C.shape[-2]
    d = C.shape[-1] - 1
    M = Kp.shape[-1]
    S = np.zeros(Kp.shape[:-2] + (M, d + 1), dtype=np.float64)
    if state_in is not None:
        S = S + np.asarray(state_in, dtype=np.float64)
    Buf2 = np.zeros(C.shape, dtype=np.float64)
    for i in range(L):
        S += Kp[..., i, :, None] * C[..., i, None, :]
        Buf2[..., i, :] = np.einsum("...m,...mp->...p", Qp[..., i, :], S)
    Buf3, buf4 = Buf2[..., :d], Buf2[..., d]
    if not renormalize:
        return Buf3, S
    return Buf3 / (buf4 + denom_eps)[..., None], S


def attn_causal(Q, K, V, W, b, input_scale, denom_eps=0.0, state_in=None,
                kernel=KERNEL_SOFTMAX, kernel_eps=1e-3, renormalize=True):
    """Unidirectional FAVOR (Algorithm 1, prefix-sum branch). Returns (out, state)."""
    Qp = features(Q, W, b, input_scale, kernel, kernel_eps)
    Kp = features(K, W, b, input_scale, kernel, kernel_eps)
    return attn_causal_features(Qp, Kp, V, denom_eps, state_in, renormalize)


def attn_explicit(Q, K, V, W, b, input_scale, causal, denom_eps=0.0, kernel=KERNEL_SOFTMAX,
                  kernel_eps=1e-3, renormalize=True):
    """The L x L estimator itself: A-hat = Q' K'^T (Eq. unbiased_attention_estimation),
    masked by tril (diagonal included) when causal, then D-hat^-1 A-hat V with
    D-hat = diag(A-hat 1_L) (A-hat V itself when renormalize is off). Only for small L."""
    Qp = features(Q, W, b, input_scale, kernel, kernel_eps)
    Kp = features(K, W, b, input_scale, kernel, kernel_eps)
    Ahat = np.matmul(Qp, np.swapaxes(Kp, -1, -2))
    if causal:
        Ahat = np.tril(Ahat)
    AV = np.matmul(Ahat, np.asarray(V, dtype=np.float64))
    if not renormalize:
        return AV
    Dhat = np.sum(Ahat, axis=-1)
    return AV / (Dhat + denom_eps)[..., None]


def softmax_attn(Q, K, V, input_scale, causal):
    """Exact attention (Sec. 2.1, Eqs. attnorm and uattnorm) on x~ = s x:
    A = exp(Q~ K~^T), tril(A) when causal (diagonal included), D^-1 A V.
    Evaluated as a row-max-shifted softmax, which leaves D^-1 A unchanged."""
    Qs = input_scale * np.asarray(Q, dtype=np.float64)
    Ks = input_scale * np.asarray(K, dtype=np.float64)
    logits = np.matmul(Qs, np.swapaxes(Ks, -1, -2))
    if causal:
        L = logits.shape[-1]
        mask = np.tril(np.ones((L, L), dtype=bool))
        logits = np.where(mask, logits, -np.inf)
    logits = logits - np.max(logits, axis=-1, keepdims=True)
    A = np.exp(logits)
    return np.matmul(A, np.asarray(V, dtype=np.float64)) / np.sum(A, axis=-1)[..., None]
