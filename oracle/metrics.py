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
