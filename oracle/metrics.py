"""Parity metrics for FAVOR outputs (test infrastructure only).

FAVOR outputs are ratios of two signed sums of products (Algorithm 1:
diag(buf4)^-1 Buf3), so an elementwise |delta| / |ref| is meaningless for
entries that pass near zero. Two gates are used instead, both max over rows:

  E_row   max_i ||out_i - ref_i||_inf / ||ref_i||_inf
  E_cond  max_{i,k} |out_ik - ref_ik| / sigma_ik with
          sigma_ik = (S_ik + |ref_ik| S_i,d) / |D-hat_i|,
          S = |Q'| (|K'|^T |C|)  (bidirectional) or its prefix analogue
          (causal), D-hat_i = Buf2_i,d the denominator of row i (plus the
          stabiliser when one is used). sigma is the first-order
          forward-error scale of a ratio of two sums of products: if every
          factor Q'_im, K'_jm, C_jk (and every carried-state entry) is
          perturbed by a relative amount of at most delta, the output moves
          by at most 3 delta sigma_ik to first order, so E_cond is the error
          in units of the working precision's unit roundoff times the
          problem's condition.

For the causal form with a carried state S_0 (Sec. 2.5.1, Eq. cumsum: the
prefix aggregate is S_0 plus the sum over keys j <= i), the carried state is
part of both sums: S_i = |Q'_i| (|S_0| + sum_{j<=i} |K'_j| |C_j|^T) and
D-hat_i = Q'_i . (S_0[:, d] + sum_{j<=i} K'_j).

Without renormalisation the output is Buf3 itself, a plain sum of products,
and sigma_ik = S_ik (err_cond_numerator).
"""
import numpy as np


def err_row(out, ref):
    """max over rows of ||out_i - ref_i||_inf / ||ref_i||_inf (rows = last axis)."""
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.max(np.abs(out - ref), axis=-1)
    den = np.max(np.abs(ref), axis=-1)
    return float(np.max(num / den)) if num.size else 0.0


def error_scale(Qp, Kp, V, causal, state_in=None):
    """(S, D-hat): the absolute-value sums S [..., L, d+1] and the signed
    denominator D-hat [..., L] (Buf2[..., d] of Algorithm 1, or of the prefix
    form with the carried state state_in [..., M, d+1] included)."""
    V = np.asarray(V, dtype=np.float64)
    Qp = np.asarray(Qp, dtype=np.float64)
    Kp = np.asarray(Kp, dtype=np.float64)
    C = np.concatenate([V, np.ones(V.shape[:-1] + (1,))], axis=-1)
    aQ, aK, aC = np.abs(Qp), np.abs(Kp), np.abs(C)
    d = V.shape[-1]
    if not causal:
        S = np.matmul(aQ, np.matmul(np.swapaxes(aK, -1, -2), aC))
        den = np.matmul(Qp, np.matmul(np.swapaxes(Kp, -1, -2), C[..., d:]))[..., 0]
        return S, den
    # prefix analogue: the same sums over keys j <= i plus the carried state
    L = C.shape[-2]
    M = Kp.shape[-1]
    S = np.empty(C.shape)
    den = np.empty(C.shape[:-1])
    acc = np.zeros(Kp.shape[:-2] + (M, d + 1))
    accd = np.zeros(Kp.shape[:-2] + (M,))
    if state_in is not None:
        st = np.asarray(state_in, dtype=np.float64)
        acc = acc + np.abs(st)
        accd = accd + st[..., :, d]
    for i in range(L):
        acc += aK[..., i, :, None] * aC[..., i, None, :]
        accd += Kp[..., i, :]
        S[..., i, :] = np.einsum("...m,...mp->...p", aQ[..., i, :], acc)
        den[..., i] = np.einsum("...m,...m->...", Qp[..., i, :], accd)
    return S, den


def err_cond(out, ref, S, den):
    """E_cond = max |out - ref| / sigma, sigma = (S[:d] + |ref| S[d]) / |den|.
    den is the row denominator (D-hat, plus the stabiliser if one is used); its
    sign does not matter."""
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = ref.shape[-1]
    sigma = (S[..., :d] + np.abs(ref) * S[..., d:d + 1]) / np.abs(den)[..., None]
    return float(np.max(np.abs(out - ref) / sigma)) if ref.size else 0.0


def err_cond_numerator(out, ref, S):
    """E_cond for the unnormalised result Buf3: max |out - ref| / S[..., :d]."""
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = ref.shape[-1]
    return float(np.max(np.abs(out - ref) / S[..., :d])) if ref.size else 0.0


def kappa(S, den):
    """Per-row condition number kappa_i = S_i,d / |D-hat_i|: how much the
    denominator cancels (1 for non-negative features)."""
    return S[..., -1] / np.abs(den)


# ---------------------------------------------------------------- gradients
def _abs_features_vjp(X, W, b, input_scale, A, kernel, kernel_eps):
    """The feature-map vector-Jacobian product of oracle.backward evaluated on
    absolute values: every product's factors replaced by their magnitudes and
    the difference of the radial and angular terms by their sum."""
    from . import favor
    X = np.asarray(X, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    s = abs(input_scale)
    Wh = W if X.ndim >= 3 else W[0]
    M = Wh.shape[-2]
    if kernel == favor.KERNEL_RELU:
        proj = np.matmul(input_scale * X, np.swapaxes(Wh, -1, -2))
        gate = (proj > 0.0).astype(np.float64)
        return s * np.matmul(A * gate / np.sqrt(M), np.abs(Wh))
    b = np.asarray(b, dtype=np.float64)
    bb = b[..., None, :] if X.ndim >= 3 else b[0][None, :]
    Xs = input_scale * X
    theta = np.matmul(Xs, np.swapaxes(Wh, -1, -2)) + bb
    D = np.exp(0.5 * np.sum(Xs * Xs, axis=-1))[..., None]
    phi = D * np.sqrt(2.0 / M) * np.abs(np.cos(theta))
    radial = np.sum(A * phi, axis=-1, keepdims=True) * np.abs(Xs)
    angular = np.matmul(A * D * np.sqrt(2.0 / M) * np.abs(np.sin(theta)), np.abs(Wh))
    return s * (radial + angular)


def grad_error_scale(Q, K, V, W, b, input_scale, dout, causal, denom_eps=0.0, state_in=None,
                     dstate_out=None, kernel=0, kernel_eps=1e-3, renormalize=True):
    """First-order error scales (A_dQ, A_dK, A_dV) of the gradients of Algorithm 1
    (Sec. 2.5) or of the prefix-sum form (Sec. 2.5.1, Eq. cumsum), entry by entry.

    The steps of oracle.backward are evaluated on absolute values (a running
    error bound): Q', K', C, the carried state and dstate_out by their
    magnitudes; the output gradient dBuf2_i = [dout_i, -(dout_i . out_i)] /
    (D-hat_i + eps) by [|dout_i|, |dout_i| . (|out_i| + sigma_i)] / |D-hat_i + eps|
    times (1 + kappa_i), where sigma_i is the output's error scale (E_cond) and
    kappa_i = S_i,d / |D-hat_i + eps| the relative error scale of the
    denominator ([|dout_i|, 0] without renormalisation); the sums over keys or
    queries then add magnitudes, and the feature VJP adds the magnitudes of its
    radial and angular terms. A rounding or perturbation of relative size delta
    in every factor moves each gradient entry by O(delta) times this scale, and
    it is never below the gradient's own magnitude. Where a gradient cancels
    (a single key: the renormalised output is v_1 whatever the query, so its
    gradient is 0; the difference v_j - out_i of nearly equal rows) the scale
    stays at the size of the terms that cancel."""
    from . import favor
    V = np.asarray(V, dtype=np.float64)
    dout = np.asarray(dout, dtype=np.float64)
    d = V.shape[-1]
    L = V.shape[-2]
    Qp = favor.features(Q, W, b, input_scale, kernel, kernel_eps)
    Kp = favor.features(K, W, b, input_scale, kernel, kernel_eps)
    M = Kp.shape[-1]
    C = np.concatenate([V, np.ones(V.shape[:-1] + (1,))], axis=-1)
    aQ, aK, aC = np.abs(Qp), np.abs(Kp), np.abs(C)
    ad = np.abs(dout)
    # forward: Buf2 (signed) and its magnitude sums S, row by row
    S, den = error_scale(Qp, Kp, V, causal, state_in=state_in if causal else None)
    if causal:
        Buf2 = np.empty(C.shape)
        G = np.zeros(Kp.shape[:-2] + (M, d + 1))
        if state_in is not None:
            G = G + np.asarray(state_in, dtype=np.float64)
        for i in range(L):
            G = G + Kp[..., i, :, None] * C[..., i, None, :]
            Buf2[..., i, :] = np.einsum("...m,...mp->...p", Qp[..., i, :], G)
    else:
        Buf2 = np.matmul(Qp, np.matmul(np.swapaxes(Kp, -1, -2), C))
    if renormalize:
        den = (den + denom_eps)[..., None]
        kap = (S[..., d:] + abs(denom_eps)) / np.abs(den)
        out = Buf2[..., :d] / den
        sig = (S[..., :d] + np.abs(out) * S[..., d:]) / np.abs(den)
        a3 = ad / np.abs(den)
        a4 = np.sum(ad * (np.abs(out) + sig), axis=-1, keepdims=True) / np.abs(den)
        adB = np.concatenate([a3, a4], axis=-1) * (1.0 + kap)
    else:
        adB = np.concatenate([ad, np.zeros(ad.shape[:-1] + (1,))], axis=-1)
    if causal:
        AdQp = np.empty(Qp.shape)
        G = np.zeros(Kp.shape[:-2] + (M, d + 1))
        if state_in is not None:
            G = G + np.abs(np.asarray(state_in, dtype=np.float64))
        for i in range(L):
            G = G + aK[..., i, :, None] * aC[..., i, None, :]
            AdQp[..., i, :] = np.einsum("...mp,...p->...m", G, adB[..., i, :])
        R = np.zeros(Kp.shape[:-2] + (M, d + 1))
        if dstate_out is not None:
            R = R + np.abs(np.asarray(dstate_out, dtype=np.float64))
        AdKp = np.empty(Kp.shape)
        AdC = np.empty(C.shape)
        for j in range(L - 1, -1, -1):
            R = R + aQ[..., j, :, None] * adB[..., j, None, :]
            AdKp[..., j, :] = np.einsum("...mp,...p->...m", R, aC[..., j, :])
            AdC[..., j, :] = np.einsum("...mp,...m->...p", R, aK[..., j, :])
    else:
        aB1 = np.matmul(np.swapaxes(aK, -1, -2), aC)
        AdQp = np.matmul(adB, np.swapaxes(aB1, -1, -2))
        adB1 = np.matmul(np.swapaxes(aQ, -1, -2), adB)
        AdKp = np.matmul(aC, np.swapaxes(adB1, -1, -2))
        AdC = np.matmul(aK, adB1)
    AdQ = _abs_features_vjp(Q, W, b, input_scale, AdQp, kernel, kernel_eps)
    AdK = _abs_features_vjp(K, W, b, input_scale, AdKp, kernel, kernel_eps)
    return AdQ, AdK, AdC[..., :d]


def err_grad_rows(got, ref, scale):
    """max over rows i of ||got_i - ref_i||_inf / ||scale_i||_inf: the row's
    error in units of its first-order error scale (grad_error_scale)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if not ref.size:
        return 0.0
    num = np.max(np.abs(got - ref), axis=-1)
    den = np.max(np.asarray(scale, dtype=np.float64), axis=-1)
    return float(np.max(num / den))
