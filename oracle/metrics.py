"""Parity metrics for FAVOR outputs (test infrastructure only).

FAVOR outputs are ratios of two signed sums of products (Algorithm 1:
diag(buf4)^-1 Buf3), so an elementwise |delta| / |ref| is meaningless for
entries that pass near zero. Two gates are used instead, both max over rows:

  E_row   max_i ||out_i - ref_i||_inf / ||ref_i||_inf
  E_cond  max_{i,k} |out_ik - ref_ik| / sigma_ik with
          sigma_ik = (S_ik + |ref_ik| S_i,d) / |Buf2_i,d|,
          S = |Q'| (|K'|^T |C|)  (bidirectional) or its prefix analogue
          (causal). sigma is the first-order forward-error scale of a ratio of
          two sums of products, so E_cond is the error in units of the working
          precision's unit roundoff times the problem's condition.

Without renormalisation the output is Buf3 itself, a plain sum of products,
and sigma_ik = S_ik (err_cond_numerator).
"""
import numpy as np


def err_row(out, ref):
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.max(np.abs(out - ref), axis=-1)
    den = np.max(np.abs(ref), axis=-1)
    return float(np.max(num / den)) if num.size else 0.0


def error_scale(Qp, Kp, V, causal, state_in_abs=None):
    """(S, |Buf2[..., d]|): the absolute-value sums and the denominator magnitude."""
    V = np.asarray(V, dtype=np.float64)
    C = np.concatenate([V, np.ones(V.shape[:-1] + (1,))], axis=-1)
    aQ, aK, aC = np.abs(Qp), np.abs(Kp), np.abs(C)
    d = V.shape[-1]
    if not causal:
        S = np.matmul(aQ, np.matmul(np.swapaxes(aK, -1, -2), aC))
        den = np.matmul(Qp, np.matmul(np.swapaxes(Kp, -1, -2), C[..., d:]))[..., 0]
    else:
        # prefix analogue, computed with cumulative sums over tokens
        L = C.shape[-2]
        M = Kp.shape[-1]
        S = np.empty(C.shape)
        den = np.empty(C.shape[:-1])
        acc = np.zeros(Kp.shape[:-2] + (M, d + 1))
        accd = np.zeros(Kp.shape[:-2] + (M,))
        if state_in_abs is not None:
            acc = acc + np.abs(state_in_abs)
        for i in range(L):
            acc += aK[..., i, :, None] * aC[..., i, None, :]
            accd += Kp[..., i, :]
            S[..., i, :] = np.einsum("...m,...mp->...p", aQ[..., i, :], acc)
            den[..., i] = np.einsum("...m,...m->...", Qp[..., i, :], accd)
    return S, np.abs(den)


def err_cond(out, ref, S, den_abs):
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = ref.shape[-1]
    sigma = (S[..., :d] + np.abs(ref) * S[..., d:d + 1]) / den_abs[..., None]
    return float(np.max(np.abs(out - ref) / sigma)) if ref.size else 0.0


def err_cond_numerator(out, ref, S):
    """E_cond for the unnormalised result Buf3: max |out - ref| / S[..., :d]."""
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = ref.shape[-1]
    return float(np.max(np.abs(out - ref) / S[..., :d])) if ref.size else 0.0
