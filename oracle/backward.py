"""Gradients of FAVOR attention in fp64: the steps of Algorithm 1 and of the
prefix-sum form (Eq. cumsum) taken in reverse order (Sec. 2.5; the paper
benchmarks the backward pass, Sec. 4.1, and trains through it).

Test infrastructure only (see ``oracle/__init__``).

Every function takes the upstream gradient dout = dLoss/dout [..., L, d] and
returns the gradients of the same loss with respect to the inputs. The forward
quantities are recomputed with ``oracle.favor`` (nothing is saved).

Notation as in Algorithm 1: C = [V 1], Buf1 = K'^T C, Buf2 = Q' Buf1,
[Buf3 buf4] = Buf2, out = Buf3 / (buf4 + eps) (Buf3 itself when not
renormalised). Feature derivatives (x~ = s x, theta_m = omega_m . x~ + b_m):
  softmax  phi_m = exp(||x~||^2/2) sqrt(2/M) cos(theta_m):
           d phi_m / d x~ = phi_m x~ - exp(||x~||^2/2) sqrt(2/M) sin(theta_m) omega_m
  ReLU     phi_m = ReLU(omega_m . x~) / sqrt(M) + kernel_eps:
           d phi_m / d x~ = [omega_m . x~ > 0] omega_m / sqrt(M)
           (the derivative at a zero projection is taken as 0)
and d/dx = s d/dx~.
"""
import numpy as np

from . import favor


def _per_head(W, b, X):
    W = np.asarray(W, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if X.ndim >= 3:
        return W, b[..., None, :]
    return W[0], b[0][None, :]


def feature_map_vjp(X, W, b, input_scale, dXp):
    """Gradient with respect to X of sum(dXp * X') for the softmax features
    (Sec. 2.3, Eqs. dqdk and qkprime). X [..., L, d], dXp [..., L, M]."""
    X = np.asarray(X, dtype=np.float64)
    dXp = np.asarray(dXp, dtype=np.float64)
    W, bb = _per_head(W, b, X)
    M = W.shape[-2]
    s = input_scale
    Xs = s * X
    theta = np.matmul(Xs, np.swapaxes(W, -1, -2)) + bb          # [..., L, M]
    D = np.exp(0.5 * np.sum(Xs * Xs, axis=-1))[..., None]        # [..., L, 1]
    phi = D * np.sqrt(2.0 / M) * np.cos(theta)
    radial = np.sum(dXp * phi, axis=-1, keepdims=True) * Xs      # sum_m dphi_m phi_m x~
    angular = np.matmul(dXp * D * np.sqrt(2.0 / M) * np.sin(theta), W)
    return s * (radial - angular)


def feature_map_relu_vjp(X, W, input_scale, dXp):
    """Gradient with respect to X of sum(dXp * X') for ReLU features (Sec. 2.2)."""
    X = np.asarray(X, dtype=np.float64)
    dXp = np.asarray(dXp, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    if X.ndim < 3:
        W = W[0]
    M = W.shape[-2]
    s = input_scale
    proj = np.matmul(s * X, np.swapaxes(W, -1, -2))
    gate = (proj > 0.0).astype(np.float64)
    return s * np.matmul(dXp * gate / np.sqrt(M), W)


def features_vjp(X, W, b, input_scale, dXp, kernel=favor.KERNEL_SOFTMAX):
    if kernel == favor.KERNEL_RELU:
        return feature_map_relu_vjp(X, W, input_scale, dXp)
    return feature_map_vjp(X, W, b, input_scale, dXp)


def _dbuf2(Buf2, dout, denom_eps, renormalize):
    """Gradient of the final step of Algorithm 1 with respect to Buf2 = [Buf3 buf4]."""
    d = Buf2.shape[-1] - 1
    Buf3, buf4 = Buf2[..., :d], Buf2[..., d]
    if not renormalize:
        return np.concatenate([dout, np.zeros(dout.shape[:-1] + (1,))], axis=-1)
    den = (buf4 + denom_eps)[..., None]
    dBuf3 = dout / den
    dbuf4 = -np.sum(dout * Buf3, axis=-1, keepdims=True) / (den * den)
    return np.concatenate([dBuf3, dbuf4], axis=-1)


def attn_bidir_backward(Q, K, V, W, b, input_scale, dout, denom_eps=0.0,
                        kernel=favor.KERNEL_SOFTMAX, kernel_eps=1e-3, renormalize=True):
    """Gradients (dQ, dK, dV) of bidirectional FAVOR (Algorithm 1), steps reversed:
    dBuf2 from the normalisation; Buf2 = Q' Buf1 gives dQ' = dBuf2 Buf1^T and
    dBuf1 = Q'^T dBuf2; Buf1 = K'^T C gives dK' = C dBuf1^T and dC = K' dBuf1
    (dV = its first d columns); then the feature maps."""
    V = np.asarray(V, dtype=np.float64)
    dout = np.asarray(dout, dtype=np.float64)
    d = V.shape[-1]
    Qp = favor.features(Q, W, b, input_scale, kernel, kernel_eps)
    Kp = favor.features(K, W, b, input_scale, kernel, kernel_eps)
    C = np.concatenate([V, np.ones(V.shape[:-1] + (1,))], axis=-1)
    Buf1 = np.matmul(np.swapaxes(Kp, -1, -2), C)
    Buf2 = np.matmul(Qp, Buf1)
    dBuf2 = _dbuf2(Buf2, dout, denom_eps, renormalize)
    dQp = np.matmul(dBuf2, np.swapaxes(Buf1, -1, -2))
    dBuf1 = np.matmul(np.swapaxes(Qp, -1, -2), dBuf2)
    dKp = np.matmul(C, np.swapaxes(dBuf1, -1, -2))
    dC = np.matmul(Kp, dBuf1)
    dQ = features_vjp(Q, W, b, input_scale, dQp, kernel)
    dK = features_vjp(K, W, b, input_scale, dKp, kernel)
    return dQ, dK, dC[..., :d]


def attn_causal_backward(Q, K, V, W, b, input_scale, dout, denom_eps=0.0, state_in=None,
                         dstate_out=None, kernel=favor.KERNEL_SOFTMAX, kernel_eps=1e-3,
                         renormalize=True):
    """Gradients of unidirectional FAVOR by prefix sums (Eq. cumsum), by sequential
    aggregation in both directions (the O(Md + Ld + ML)-space form of Sec. 2.6).

    Forward: G_i = S_0 + sum_{j <= i} K'_j C_j^T, Buf2_i = G_i^T Q'_i, state_out = G_L.
    Backward: dQ'_i = G_i dBuf2_i; with R_j = dstate_out + sum_{i >= j} Q'_i dBuf2_i^T
    (a suffix sum, j = L..1), dK'_j = R_j C_j and dC_j = R_j^T K'_j; dstate_in = R_1.
    Returns (dQ, dK, dV, dstate_in [..., M, d+1])."""
    V = np.asarray(V, dtype=np.float64)
    dout = np.asarray(dout, dtype=np.float64)
    d = V.shape[-1]
    L = V.shape[-2]
    Qp = favor.features(Q, W, b, input_scale, kernel, kernel_eps)
    Kp = favor.features(K, W, b, input_scale, kernel, kernel_eps)
    M = Kp.shape[-1]
    C = np.concatenate([V, np.ones(V.shape[:-1] + (1,))], axis=-1)
    G = np.zeros(Kp.shape[:-2] + (M, d + 1))
    if state_in is not None:
        G = G + np.asarray(state_in, dtype=np.float64)
    dBuf2 = np.zeros(C.shape)
    dQp = np.zeros(Qp.shape)
    for i in range(L):
        G = G + Kp[..., i, :, None] * C[..., i, None, :]
        Buf2_i = np.einsum("...m,...mp->...p", Qp[..., i, :], G)
        dBuf2[..., i, :] = _dbuf2(Buf2_i[..., None, :], dout[..., i, None, :], denom_eps,
                                  renormalize)[..., 0, :]
        dQp[..., i, :] = np.einsum("...mp,...p->...m", G, dBuf2[..., i, :])
    R = np.zeros(Kp.shape[:-2] + (M, d + 1))
    if dstate_out is not None:
        R = R + np.asarray(dstate_out, dtype=np.float64)
    dKp = np.zeros(Kp.shape)
    dC = np.zeros(C.shape)
    for j in range(L - 1, -1, -1):
        R = R + Qp[..., j, :, None] * dBuf2[..., j, None, :]
        dKp[..., j, :] = np.einsum("...mp,...p->...m", R, C[..., j, :])
        dC[..., j, :] = np.einsum("...mp,...m->...p", R, Kp[..., j, :])
    dQ = features_vjp(Q, W, b, input_scale, dQp, kernel)
    dK = features_vjp(K, W, b, input_scale, dKp, kernel)
    return dQ, dK, dC[..., :d], R
