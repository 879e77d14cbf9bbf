"""Pins of the parity metrics (oracle/metrics.py) against what they are defined to
measure, independently of the formulas inside them.

Algorithm 1 (Sec. 2.5) computes out_ik = N_ik / D_i with N_ik = sum over terms
Q'_im K'_jm C_jk (C = [V 1]) and D_i the same sum over the column C_jd = 1; the
prefix form (Sec. 2.5.1, Eq. cumsum) takes the keys j <= i and adds the carried
state S_0: terms Q'_im S_0[m, k]. The error scale S_ik is by definition the sum
of the absolute values of those terms, and D-hat_i the signed sum for column d.
The pins enumerate the terms one by one in plain Python loops, build the exact
case where the first-order bound is attained, and check the bound on random
perturbations.
"""
import itertools

import numpy as np
import pytest

from oracle import favor, metrics


def _terms(Qp, Kp, V, i, k, causal, state_in=None):
    """Every product term of Buf2[i, k] (column k = d is the denominator)."""
    L, d = V.shape
    M = Qp.shape[1]
    C = lambda j, c: 1.0 if c == d else V[j, c]
    out = []
    for j in range(L):
        if causal and j > i:
            continue
        for m in range(M):
            out.append(Qp[i, m] * Kp[j, m] * C(j, k))
    if causal and state_in is not None:
        for m in range(M):
            out.append(Qp[i, m] * state_in[m, k])
    return out


def _brute(Qp, Kp, V, causal, state_in=None):
    L, d = V.shape
    S = np.zeros((L, d + 1))
    den = np.zeros(L)
    num = np.zeros((L, d + 1))
    for i, k in itertools.product(range(L), range(d + 1)):
        t = _terms(Qp, Kp, V, i, k, causal, state_in)
        S[i, k] = sum(abs(x) for x in t)
        num[i, k] = sum(t)
    den[:] = num[:, d]
    return S, den, num


def _signed_case(seed, L=6, M=5, d=3):
    rng = np.random.default_rng(seed)
    Qp = rng.normal(size=(L, M))
    Kp = rng.normal(size=(L, M))
    V = rng.normal(size=(L, d))
    st = rng.normal(size=(M, d + 1)) * 3.0
    return Qp, Kp, V, st


def test_err_row_hand_example():
    ref = np.array([[1.0, -2.0, 0.5], [0.1, 0.2, -0.4]])
    out = np.array([[1.1, -2.0, 0.5], [0.1, 0.25, -0.4]])
    # row 0: 0.1 / 2 = 0.05; row 1: 0.05 / 0.4 = 0.125
    assert metrics.err_row(out, ref) == pytest.approx(0.125, rel=1e-12)
    assert metrics.err_row(ref, ref) == 0.0
    assert metrics.err_row(np.zeros((0, 3)), np.zeros((0, 3))) == 0.0


def test_err_cond_hand_example():
    # one row, d = 2: S = [4, 2, 5], D-hat = -2 (sign must not matter)
    ref = np.array([[1.0, -3.0]])
    out = np.array([[1.5, -3.0 + 0.17]])
    S = np.array([[4.0, 2.0, 5.0]])
    # sigma = (S_k + |ref_k| * 5) / 2 = [(4 + 5) / 2, (2 + 15) / 2] = [4.5, 8.5]
    want = max(0.5 / 4.5, 0.17 / 8.5)
    assert metrics.err_cond(out, ref, S, np.array([-2.0])) == pytest.approx(want, rel=1e-12)
    assert metrics.err_cond(out, ref, S, np.array([2.0])) == pytest.approx(want, rel=1e-12)
    assert metrics.err_cond_numerator(out, ref, S) == pytest.approx(max(0.5 / 4, 0.17 / 2),
                                                                   rel=1e-12)
    S_b = np.array([[4.0, 2.0, 5.0]])
    assert metrics.kappa(S_b, np.array([-2.0]))[0] == pytest.approx(2.5)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_error_scale_bidir_is_sum_of_absolute_terms(seed):
    Qp, Kp, V, _ = _signed_case(seed)
    S, den = metrics.error_scale(Qp, Kp, V, causal=False)
    Sb, denb, num = _brute(Qp, Kp, V, causal=False)
    np.testing.assert_allclose(S, Sb, rtol=1e-13, atol=0)
    np.testing.assert_allclose(den, denb, rtol=1e-12, atol=1e-14)
    # the denominator is Algorithm 1's buf4: out * D-hat = Buf3
    out = favor.attn_bidir_features(Qp, Kp, V)
    np.testing.assert_allclose(out * den[:, None], num[:, :-1], rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("with_state", [False, True])
def test_error_scale_causal_is_sum_of_absolute_terms(seed, with_state):
    Qp, Kp, V, st = _signed_case(seed)
    st = st if with_state else None
    S, den = metrics.error_scale(Qp, Kp, V, causal=True, state_in=st)
    Sb, denb, num = _brute(Qp, Kp, V, causal=True, state_in=st)
    np.testing.assert_allclose(S, Sb, rtol=1e-13, atol=0)
    np.testing.assert_allclose(den, denb, rtol=1e-12, atol=1e-13)
    out, _ = favor.attn_causal_features(Qp, Kp, V, state_in=st)
    np.testing.assert_allclose(out * den[:, None], num[:, :-1], rtol=1e-10, atol=1e-12)


def test_error_scale_batched_matches_per_head():
    rng = np.random.default_rng(5)
    B, H, L, M, d = 2, 3, 7, 4, 2
    Qp, Kp = rng.normal(size=(2, B, H, L, M))
    V = rng.normal(size=(B, H, L, d))
    st = rng.normal(size=(B, H, M, d + 1))
    for causal in (False, True):
        S, den = metrics.error_scale(Qp, Kp, V, causal, state_in=st if causal else None)
        for bi, hi in itertools.product(range(B), range(H)):
            Sb, denb, _ = _brute(Qp[bi, hi], Kp[bi, hi], V[bi, hi], causal,
                                 st[bi, hi] if causal else None)
            np.testing.assert_allclose(S[bi, hi], Sb, rtol=1e-13)
            np.testing.assert_allclose(den[bi, hi], denb, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("causal,with_state", [(False, False), (True, False), (True, True)])
def test_first_order_bound_is_attained_for_positive_terms(causal, with_state):
    """Non-negative features, values and state: |terms| = terms, so S = Buf2 and
    sigma_ik = 2 out_ik. Scaling every value entry (V and the state's value
    columns) by (1 + delta) scales out by exactly (1 + delta), hence
    E_cond = delta / 2 exactly. A denominator that leaves out part of the sum
    (e.g. the carried state) makes sigma too large and E_cond smaller."""
    rng = np.random.default_rng(11)
    L, M, d = 9, 6, 4
    Qp = rng.uniform(0.1, 1.0, size=(L, M))
    Kp = rng.uniform(0.1, 1.0, size=(L, M))
    V = rng.uniform(0.5, 2.0, size=(L, d))
    st = rng.uniform(0.0, 40.0, size=(M, d + 1)) if with_state else None
    delta = 1e-3
    if causal:
        ref, _ = favor.attn_causal_features(Qp, Kp, V, state_in=st)
        st2 = None if st is None else np.concatenate([st[:, :d] * (1 + delta), st[:, d:]], 1)
        out, _ = favor.attn_causal_features(Qp, Kp, V * (1 + delta), state_in=st2)
    else:
        ref = favor.attn_bidir_features(Qp, Kp, V)
        out = favor.attn_bidir_features(Qp, Kp, V * (1 + delta))
    S, den = metrics.error_scale(Qp, Kp, V, causal, state_in=st)
    assert metrics.err_cond(out, ref, S, den) == pytest.approx(delta / 2, rel=1e-9)
    assert np.allclose(metrics.kappa(S, den), 1.0)


@pytest.mark.parametrize("causal,with_state", [(False, False), (True, False), (True, True)])
def test_random_relative_perturbations_stay_within_three_delta(causal, with_state):
    """Every factor of every term perturbed by a relative amount of at most delta
    (signed features, so D-hat cancels): |out - ref| <= 3 delta sigma to first
    order. An error scale that is too small (a dropped term, a wrong sign in
    D-hat) breaks the bound on some seed."""
    delta = 1e-6
    worst = 0.0
    for seed in range(20):
        rng = np.random.default_rng(100 + seed)
        L, M, d = 8, 6, 3
        Qp = rng.normal(size=(L, M))
        Kp = rng.normal(size=(L, M))
        V = rng.normal(size=(L, d))
        st = rng.normal(size=(M, d + 1)) * 2.0 if with_state else None
        pert = lambda a: a * (1 + delta * rng.uniform(-1, 1, size=a.shape))
        # every term Q_im K_jm C_jk: perturbing Q', K' and V covers all three
        # factors except the exact ones column, which the kernels keep exact
        if causal:
            ref, _ = favor.attn_causal_features(Qp, Kp, V, state_in=st)
            out, _ = favor.attn_causal_features(pert(Qp), pert(Kp), pert(V),
                                                state_in=None if st is None else pert(st))
        else:
            ref = favor.attn_bidir_features(Qp, Kp, V)
            out = favor.attn_bidir_features(pert(Qp), pert(Kp), pert(V))
        S, den = metrics.error_scale(Qp, Kp, V, causal, state_in=st)
        e = metrics.err_cond(out, ref, S, den)
        assert e <= 3 * delta * (1 + 1e-3), (seed, e)
        worst = max(worst, e)
    # and the bound is not vacuous: some row reaches a sizeable part of it
    assert worst >= 0.1 * delta


def test_carried_state_enters_the_denominator():
    """A large carried state dominates D-hat: the metric's denominator must be
    the full prefix denominator, which the explicit sum over the state's column
    d plus the keys gives."""
    rng = np.random.default_rng(3)
    L, M, d = 4, 8, 2
    Qp = np.abs(rng.normal(size=(L, M)))
    Kp = np.abs(rng.normal(size=(L, M)))
    V = rng.normal(size=(L, d))
    st = np.zeros((M, d + 1))
    st[:, d] = 200.0
    _, den = metrics.error_scale(Qp, Kp, V, causal=True, state_in=st)
    want = [Qp[i] @ (st[:, d] + Kp[:i + 1].sum(0)) for i in range(L)]
    np.testing.assert_allclose(den, want, rtol=1e-13)


# ---------------------------------------------------------------- gradients
from oracle import backward as bw  # noqa: E402


def _grad_case(seed, L=9, M=8, d=4, B=1, H=2):
    rng = np.random.default_rng(seed)
    Q = rng.normal(size=(B, H, L, d)) * 0.5
    K = rng.normal(size=(B, H, L, d)) * 0.5
    V = rng.normal(size=(B, H, L, d))
    dout = rng.normal(size=(B, H, L, d))
    W, b = favor.orf_draw(seed, H, M, d)
    return Q, K, V, dout, W, b


def _grads(Q, K, V, W, b, dout, causal, **kw):
    if causal:
        return bw.attn_causal_backward(Q, K, V, W, b, 1.0, dout, **kw)[:3]
    return bw.attn_bidir_backward(Q, K, V, W, b, 1.0, dout, **kw)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("kernel,renorm,eps", [(favor.KERNEL_SOFTMAX, True, 0.0),
                                               (favor.KERNEL_SOFTMAX, True, 0.3),
                                               (favor.KERNEL_SOFTMAX, False, 0.0),
                                               (favor.KERNEL_RELU, True, 0.0)])
def test_grad_scale_bounds_relative_perturbations(causal, kernel, renorm, eps, monkeypatch):
    """Perturb every factor the contractions multiply (the features Q', K', the
    values V and the output gradient) by a relative amount of at most delta: each
    gradient row moves by at most a small multiple of delta times its error scale,
    in particular on the rows whose gradient cancels (the first causal row, whose
    exact dQ is 0 with renormalisation)."""
    delta = 1e-6
    worst = 0.0
    for seed in range(6):
        Q, K, V, dout, W, b = _grad_case(seed)
        kw = dict(kernel=kernel, renormalize=renorm, denom_eps=eps)
        ref = _grads(Q, K, V, W, b, dout, causal, **kw)
        scale = metrics.grad_error_scale(Q, K, V, W, b, 1.0, dout, causal, **kw)
        for r, a in zip(ref, scale):
            assert np.all(a >= np.abs(r) * (1 - 1e-12))
        rng = np.random.default_rng(seed + 50)
        real = favor.features
        monkeypatch.setattr(favor, "features", lambda *a, **k: (
            lambda f: f * (1 + delta * rng.uniform(-1, 1, size=f.shape)))(real(*a, **k)))
        pert = lambda x: x * (1 + delta * rng.uniform(-1, 1, size=x.shape))
        got = _grads(Q, K, pert(V), W, b, pert(dout), causal, **kw)
        monkeypatch.setattr(favor, "features", real)
        for g, r, a in zip(got, ref, scale):
            e = metrics.err_grad_rows(g, r, a)
            assert e <= 4 * delta, e
            worst = max(worst, e)
    assert worst >= 0.02 * delta


@pytest.mark.parametrize("causal", [False, True])
def test_grad_scale_of_values_for_positive_terms(causal):
    """Non-negative features (ReLU with kernel_eps > 0 on any input), values and
    output gradient: dV_j = sum_i dout_i (Q'_i . K'_j) / D-hat_i has no
    cancellation and kappa = 1, so its scale is exactly (1 + kappa) |dV| = 2 dV."""
    rng = np.random.default_rng(2)
    B, H, L, M, d = 1, 1, 7, 8, 3
    Q = rng.normal(size=(B, H, L, d))
    K = rng.normal(size=(B, H, L, d))
    V = rng.uniform(0.5, 2.0, size=(B, H, L, d))
    dout = rng.uniform(0.1, 1.0, size=(B, H, L, d))
    W, b = favor.orf_draw(4, H, M, d)
    kw = dict(kernel=favor.KERNEL_RELU, kernel_eps=0.05)
    dV = _grads(Q, K, V, W, b, dout, causal, **kw)[2]
    AdV = metrics.grad_error_scale(Q, K, V, W, b, 1.0, dout, causal, **kw)[2]
    assert np.all(dV > 0)
    np.testing.assert_allclose(AdV, 2 * dV, rtol=1e-12)


def test_grad_scale_single_key_rows_keep_the_size_of_their_terms():
    """With one key (L = 1) the renormalised output is v_1 whatever q and k are:
    dQ and dK vanish in exact arithmetic, yet their error scale is the size of
    the terms that cancel, comparable to that of dV."""
    Q, K, V, dout, W, b = _grad_case(7, L=1)
    dQ, dK, dV = _grads(Q, K, V, W, b, dout, False)
    AdQ, AdK, AdV = metrics.grad_error_scale(Q, K, V, W, b, 1.0, dout, False)
    assert np.max(np.abs(dQ)) <= 1e-12 * np.max(AdQ)
    assert np.max(np.abs(dK)) <= 1e-12 * np.max(AdK)
    assert np.min(AdQ.max(axis=-1)) > 1e-3 * np.max(AdV)


def test_grad_scale_bounds_perturbations_with_carried_states(monkeypatch):
    """The causal form with a carried state and a gradient reaching state_out:
    both enter the prefix and suffix aggregates, and their magnitudes enter the
    scale; perturbing them with the other factors stays within the bound."""
    delta = 1e-6
    for seed in range(4):
        Q, K, V, dout, W, b = _grad_case(seed)
        rng = np.random.default_rng(seed + 80)
        S0 = rng.normal(size=(1, 2, 8, 5)) * 100.0
        dS = rng.normal(size=(1, 2, 8, 5)) * 30.0
        kw = dict(state_in=S0, dstate_out=dS)
        ref = bw.attn_causal_backward(Q, K, V, W, b, 1.0, dout, **kw)[:3]
        scale = metrics.grad_error_scale(Q, K, V, W, b, 1.0, dout, True, **kw)
        real = favor.features
        monkeypatch.setattr(favor, "features", lambda *a, **k: (
            lambda f: f * (1 + delta * rng.uniform(-1, 1, size=f.shape)))(real(*a, **k)))
        pert = lambda x: x * (1 + delta * rng.uniform(-1, 1, size=x.shape))
        got = bw.attn_causal_backward(Q, K, pert(V), W, b, 1.0, pert(dout),
                                      state_in=pert(S0), dstate_out=pert(dS))[:3]
        monkeypatch.setattr(favor, "features", real)
        for g, r, a in zip(got, ref, scale):
            assert metrics.err_grad_rows(g, r, a) <= 4 * delta
