"""Pins for the oracle's feature map and FAVOR attention.

What fixes the values (the paper prints no numeric worked example):
  * Bochner / unbiasedness: E[phi(x)^T phi(y)] = exp(-||x - y||^2 / 2) and
    E[Q' K'^T] = exp(Q~ K~^T) (Sec. 2.3, Eqs. rfm and unbiased_attention_estimation)
  * the closed-form variance of the IID estimator (derived from Sec. 2.3)
  * the linear-order result equals the explicit L x L estimator (Sec. 2.5)
  * invariants: one-hot V, V = 1, Q = K = 0, causal first/last rows,
    linearity and permutations, feature rescaling, state carry-over
  * exact softmax attention against torch's scaled_dot_product_attention
  * convergence to softmax attention as M grows (Theorem 1)
"""
import numpy as np
import pytest
import torch

from oracle import favor

D = 16


def _inputs(seed, B, H, L, d, scale_qk=True):
    rng = np.random.default_rng(seed)
    s = d ** -0.25 if scale_qk else 1.0
    Q = rng.standard_normal((B, H, L, d)) * s
    K = rng.standard_normal((B, H, L, d)) * s
    V = rng.standard_normal((B, H, L, d))
    return Q, K, V


# ---------------------------------------------------------------- kernel identities
def test_bochner_gaussian_kernel_iid():
    """Large-M IID features reproduce the Gaussian kernel (no D factors)."""
    d, M = 4, 1 << 16
    W, b = favor.orf_draw(1, 1, M, d, favor.RF_IID)
    rng = np.random.default_rng(2)
    x = rng.standard_normal((6, d)) * 0.6
    y = rng.standard_normal((6, d)) * 0.6
    # strip D_X by using unit scale on the feature map of x and then dividing it out
    fx = favor.feature_map(x, W, b, 1.0) / np.exp(0.5 * np.sum(x * x, 1))[:, None]
    fy = favor.feature_map(y, W, b, 1.0) / np.exp(0.5 * np.sum(y * y, 1))[:, None]
    est = fx @ fy.T
    exact = np.exp(-0.5 * np.sum((x[:, None, :] - y[None, :, :]) ** 2, -1))
    assert np.max(np.abs(est - exact)) < 6.0 / np.sqrt(M)


def test_unbiased_attention_matrix_orf():
    """mean over seeds of Q' K'^T -> exp(Q~ K~^T), entrywise within 5 sd / sqrt(S)."""
    L, d, M, S = 6, D, 32, 400
    Q, K, _ = _inputs(3, 1, 1, L, d)
    Q, K = Q[0, 0], K[0, 0]
    s = d ** -0.25
    A = np.exp((s * Q) @ (s * K).T)
    ests = []
    for seed in range(1000, 1000 + S):
        W, b = favor.orf_draw(seed, 1, M, d, favor.RF_ORTHO_CHI)
        ests.append(favor.feature_map(Q, W, b, s) @ favor.feature_map(K, W, b, s).T)
    ests = np.array(ests)
    mean, sd = ests.mean(0), ests.std(0)
    assert np.all(np.abs(mean - A) <= 5 * sd / np.sqrt(S) + 1e-12)


def test_biased_variants_would_fail_the_unbiasedness_pin():
    """The same check rejects a feature map with a dropped D factor."""
    L, d, M, S = 6, D, 32, 200
    Q, K, _ = _inputs(3, 1, 1, L, d)
    Q, K = Q[0, 0], K[0, 0]
    s = d ** -0.25
    A = np.exp((s * Q) @ (s * K).T)
    ests = []
    for seed in range(2000, 2000 + S):
        W, b = favor.orf_draw(seed, 1, M, d, favor.RF_ORTHO_CHI)
        fq = favor.feature_map(Q, W, b, s) / np.exp(0.5 * s * s * np.sum(Q * Q, 1))[:, None]
        ests.append(fq @ favor.feature_map(K, W, b, s).T)
    ests = np.array(ests)
    mean, sd = ests.mean(0), ests.std(0)
    assert not np.all(np.abs(mean - A) <= 5 * sd / np.sqrt(S))


def test_iid_variance_closed_form():
    """Var[B-hat_ij] = (1 - e^{-|z|^2} + e^{-2|z|^2} / 2) / M for IID features,
    z = x~ - y~ (derived from the single-cos features of Sec. 2.3)."""
    d, M, S = 8, 16, 3000
    rng = np.random.default_rng(4)
    x = rng.standard_normal(d) * 0.35
    y = rng.standard_normal(d) * 0.35
    vals = []
    for seed in range(S):
        W, b = favor.orf_draw(seed, 1, M, d, favor.RF_IID)
        fx = favor.feature_map(x[None], W, b, 1.0)[0] / np.exp(0.5 * x @ x)
        fy = favor.feature_map(y[None], W, b, 1.0)[0] / np.exp(0.5 * y @ y)
        vals.append(fx @ fy)
    z2 = np.sum((x - y) ** 2)
    pred = (1 - np.exp(-z2) + 0.5 * np.exp(-2 * z2)) / M
    var = np.var(vals, ddof=1)
    assert abs(var / pred - 1) < 5 * np.sqrt(2.0 / S)
    assert abs(np.mean(vals) - np.exp(-0.5 * z2)) < 5 * np.sqrt(pred / S)


def test_orf_variance_not_above_iid():
    """Sec. 2.4 / Sec. 4.2: orthogonal features do not increase the error."""
    d, M, L, S = 16, 64, 32, 60
    Q, K, _ = _inputs(5, 1, 1, L, d)
    Q, K = Q[0, 0], K[0, 0]
    s = d ** -0.25
    A = np.exp((s * Q) @ (s * K).T)
    def mse(kind):
        e = []
        for seed in range(S):
            W, b = favor.orf_draw(seed, 1, M, d, kind)
            e.append(np.mean((favor.feature_map(Q, W, b, s) @ favor.feature_map(K, W, b, s).T - A) ** 2))
        return np.mean(e)
    assert mse(favor.RF_ORTHO_CHI) < mse(favor.RF_IID)


# ---------------------------------------------------------------- Algorithm 1 vs explicit
@pytest.mark.parametrize("L,M", [(1, 16), (37, 32), (128, 64), (256, 48)])
def test_bidir_equals_explicit(L, M):
    Q, K, V = _inputs(L, 2, 3, L, D)
    W, b = favor.orf_draw(L + 1, 3, M, D)
    s = D ** -0.25
    out = favor.attn_bidir(Q, K, V, W, b, s)
    ref = favor.attn_explicit(Q, K, V, W, b, s, causal=False)
    assert np.max(np.abs(out - ref)) <= 1e-12 * np.max(np.abs(ref))


@pytest.mark.parametrize("L,M", [(1, 16), (37, 32), (128, 64), (256, 48)])
def test_causal_equals_explicit(L, M):
    Q, K, V = _inputs(L + 7, 2, 3, L, D)
    W, b = favor.orf_draw(L + 2, 3, M, D)
    s = D ** -0.25
    out, _ = favor.attn_causal(Q, K, V, W, b, s)
    ref = favor.attn_explicit(Q, K, V, W, b, s, causal=True)
    assert np.max(np.abs(out - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_one_hot_values_extract_attention_matrix():
    """Running FAVOR on V = I_L returns D-hat^-1 A-hat itself (App. C.4 trick)."""
    L, M = 24, 32
    Q, K, _ = _inputs(6, 1, 1, L, D)
    W, b = favor.orf_draw(6, 1, M, D)
    s = D ** -0.25
    I = np.eye(L)[None, None]
    Qp = favor.feature_map(Q, W, b, s)
    Kp = favor.feature_map(K, W, b, s)
    Ahat = Qp[0, 0] @ Kp[0, 0].T
    bi = favor.attn_bidir(Q, K, I, W, b, s)[0, 0]
    assert np.allclose(bi, Ahat / Ahat.sum(1, keepdims=True), rtol=1e-10, atol=1e-12)
    ca, _ = favor.attn_causal(Q, K, I, W, b, s)
    T = np.tril(Ahat)
    assert np.allclose(ca[0, 0], T / T.sum(1, keepdims=True), rtol=1e-10, atol=1e-12)
    assert np.all(np.triu(ca[0, 0], 1) == 0)


def test_constant_values_give_ones():
    Q, K, _ = _inputs(7, 1, 2, 50, D)
    W, b = favor.orf_draw(7, 2, 32, D)
    V = np.ones((1, 2, 50, D))
    s = D ** -0.25
    assert np.allclose(favor.attn_bidir(Q, K, V, W, b, s), 1.0, rtol=1e-12)
    assert np.allclose(favor.attn_causal(Q, K, V, W, b, s)[0], 1.0, rtol=1e-12)


def test_causal_first_and_last_rows():
    Q, K, V = _inputs(8, 2, 2, 40, D)
    W, b = favor.orf_draw(8, 2, 32, D)
    s = D ** -0.25
    ca, _ = favor.attn_causal(Q, K, V, W, b, s)
    bi = favor.attn_bidir(Q, K, V, W, b, s)
    assert np.allclose(ca[..., 0, :], V[..., 0, :], rtol=1e-12)
    assert np.allclose(ca[..., -1, :], bi[..., -1, :], rtol=1e-10)


def test_zero_queries_and_keys_average_values():
    """Q = K = 0: every feature is sqrt(2/M) cos(b_m), so A-hat is a constant
    matrix; bidir returns the column mean of V, causal the running mean."""
    L = 30
    rng = np.random.default_rng(9)
    V = rng.standard_normal((1, 1, L, D))
    Z = np.zeros((1, 1, L, D))
    W, b = favor.orf_draw(9, 1, 32, D)
    bi = favor.attn_bidir(Z, Z, V, W, b, 0.5)
    assert np.allclose(bi, V.mean(axis=2, keepdims=True), rtol=1e-12)
    ca, _ = favor.attn_causal(Z, Z, V, W, b, 0.5)
    run = np.cumsum(V, axis=2) / np.arange(1, L + 1)[None, None, :, None]
    assert np.allclose(ca, run, rtol=1e-11)


def test_linearity_and_permutations():
    L = 33
    Q, K, V = _inputs(10, 1, 1, L, D)
    _, _, V2 = _inputs(11, 1, 1, L, D)
    W, b = favor.orf_draw(10, 1, 32, D)
    s = D ** -0.25
    f = lambda q, k, v: favor.attn_bidir(q, k, v, W, b, s)
    assert np.allclose(f(Q, K, 2 * V - 3 * V2), 2 * f(Q, K, V) - 3 * f(Q, K, V2), atol=1e-11)
    p = np.random.default_rng(0).permutation(L)
    assert np.allclose(f(Q, K[:, :, p], V[:, :, p]), f(Q, K, V), atol=1e-12)
    assert np.allclose(f(Q[:, :, p], K, V), f(Q, K, V)[:, :, p], atol=1e-12)


def test_feature_rescaling_invariance():
    L, M = 40, 32
    Q, K, V = _inputs(12, 1, 2, L, D)
    W, b = favor.orf_draw(12, 2, M, D)
    s = D ** -0.25
    Qp = favor.feature_map(Q, W, b, s)
    Kp = favor.feature_map(K, W, b, s)
    c = np.random.default_rng(1).uniform(0.5, 2.0, size=(1, 2, L, 1))
    ref = favor.attn_bidir_features(Qp, Kp, V)
    assert np.allclose(favor.attn_bidir_features(c * Qp, Kp, V), ref, rtol=1e-10)
    assert np.allclose(favor.attn_bidir_features(Qp, 3.7 * Kp, V), ref, rtol=1e-10)
    ref_c, _ = favor.attn_causal_features(Qp, Kp, V)
    out_c, _ = favor.attn_causal_features(c * Qp, Kp, V)
    assert np.allclose(out_c, ref_c, rtol=1e-10)


def test_causal_state_carry_over():
    """One call over L equals two calls over halves with the state handed on;
    the final state is the bidirectional Buf1 = K'^T [V 1]."""
    L, M = 64, 32
    Q, K, V = _inputs(13, 2, 2, L, D)
    W, b = favor.orf_draw(13, 2, M, D)
    s = D ** -0.25
    full, S = favor.attn_causal(Q, K, V, W, b, s)
    h = 27
    o1, S1 = favor.attn_causal(Q[..., :h, :], K[..., :h, :], V[..., :h, :], W, b, s)
    o2, S2 = favor.attn_causal(Q[..., h:, :], K[..., h:, :], V[..., h:, :], W, b, s, state_in=S1)
    assert np.allclose(np.concatenate([o1, o2], axis=2), full, rtol=1e-11, atol=1e-12)
    assert np.allclose(S2, S, rtol=1e-12)
    Kp = favor.feature_map(K, W, b, s)
    C = np.concatenate([V, np.ones(V.shape[:-1] + (1,))], -1)
    assert np.allclose(S, np.swapaxes(Kp, -1, -2) @ C, rtol=1e-11)


def test_denominator_stabiliser_placement():
    """denom_eps is added to D-hat: with V = 1 the output is buf4 / (buf4 + eps)."""
    L, M = 20, 32
    Q, K, _ = _inputs(14, 1, 1, L, D)
    W, b = favor.orf_draw(14, 1, M, D)
    s = D ** -0.25
    V = np.ones((1, 1, L, D))
    Qp = favor.feature_map(Q, W, b, s)
    Kp = favor.feature_map(K, W, b, s)
    dhat = (Qp @ (np.swapaxes(Kp, -1, -2) @ np.ones((1, 1, L, 1))))[..., 0]
    out = favor.attn_bidir(Q, K, V, W, b, s, denom_eps=0.25)
    assert np.allclose(out, (dhat / (dhat + 0.25))[..., None], rtol=1e-12)


# ---------------------------------------------------------------- exact attention
@pytest.mark.parametrize("causal", [False, True])
def test_softmax_matches_torch_sdpa(causal):
    Q, K, V = _inputs(15, 2, 3, 70, D)
    s = D ** -0.25
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q), torch.from_numpy(K), torch.from_numpy(V),
        is_causal=causal, scale=s * s).numpy()
    out = favor.softmax_attn(Q, K, V, s, causal)
    assert np.allclose(out, ref, rtol=1e-10, atol=1e-12)


def test_converges_to_softmax_as_m_grows():
    """Error vs exact attention shrinks roughly as M^-1/2 (Theorem 1, Sec. 4.2)."""
    L, d = 128, D
    Q, K, V = _inputs(16, 1, 1, L, d)
    s = d ** -0.25
    ex = favor.softmax_attn(Q, K, V, s, False)
    def err(M):
        e = []
        for seed in range(12):
            W, b = favor.orf_draw(100 + seed, 1, M, d)
            o = favor.attn_bidir(Q, K, V, W, b, s)
            e.append(np.linalg.norm(o - ex) / np.linalg.norm(ex))
        return np.mean(e)
    e1, e2, e3 = err(64), err(256), err(1024)
    assert e1 > e2 > e3
    assert 0.3 < e2 / e1 < 0.7 and 0.3 < e3 / e2 < 0.7


# ---------------------------------------------------------------- generalized attention, f = ReLU
def _arccos1(x, y):
    """First-order arc-cosine kernel (Cho and Saul, NeurIPS 2009): for omega ~ N(0, I),
    E[ReLU(omega . x) ReLU(omega . y)] = |x| |y| (sin t + (pi - t) cos t) / (2 pi)."""
    nx, ny = np.linalg.norm(x, axis=-1), np.linalg.norm(y, axis=-1)
    t = np.arccos(np.clip(np.sum(x * y, -1) / (nx * ny), -1.0, 1.0))
    return nx * ny * (np.sin(t) + (np.pi - t) * np.cos(t)) / (2 * np.pi)


def test_relu_features_reproduce_the_arccosine_kernel():
    """Large-M IID ReLU features: phi(x)^T phi(y) -> the arc-cosine kernel of x~, y~
    (pins f = ReLU, the 1/sqrt(M) scale, the input scale and the absence of D factors)."""
    d, M, s = 8, 1 << 16, 0.7
    W, b = favor.orf_draw(5, 1, M, d, favor.RF_IID)
    rng = np.random.default_rng(6)
    x = rng.standard_normal((8, d))
    y = rng.standard_normal((8, d))
    y[0] = x[0]                      # theta = 0: E = |x~|^2 / 2
    y[1] = -x[1]                     # theta = pi: E = 0
    fx = favor.feature_map_relu(x, W, s, kernel_eps=0.0)
    fy = favor.feature_map_relu(y, W, s, kernel_eps=0.0)
    est = np.sum(fx * fy, -1)
    want = _arccos1(s * x, s * y)
    # per-feature products have sample sd sd_m; the mean of M of them has sd sd_m / sqrt(M)
    prod = fx * fy * M
    se = np.std(prod, -1) / np.sqrt(M)
    assert np.all(np.abs(est - want) <= 5 * se + 1e-12)
    assert abs(want[1]) < 1e-12 and abs(est[1]) == 0.0
    np.testing.assert_allclose(want[0], 0.5 * s * s * np.sum(x[0] ** 2), rtol=1e-12)


def test_relu_feature_stabiliser_placement():
    """kernel_eps is added to every feature after the ReLU and the scaling: a zero
    projection gives exactly eps, a negative one too, and features never go below it."""
    d, M, eps = 16, 64, 1e-3
    W, b = favor.orf_draw(7, 1, M, d, favor.RF_ORTHO_CHI)
    X = np.random.default_rng(8).standard_normal((40, d))
    f0 = favor.feature_map_relu(X, np.zeros_like(W), 1.0, eps)
    assert np.all(f0 == eps)
    f = favor.feature_map_relu(X, W, 0.5, eps)
    proj = 0.5 * X @ W[0].T
    assert np.all(f >= eps)
    assert np.all(f[proj < 0] == eps)
    np.testing.assert_allclose(f[proj > 0], proj[proj > 0] / np.sqrt(M) + eps, rtol=1e-14)


@pytest.mark.parametrize("renormalize", [True, False])
@pytest.mark.parametrize("L,M", [(1, 16), (37, 32), (128, 64)])
def test_relu_attention_equals_explicit(L, M, renormalize):
    """Algorithm 1 (bidirectional and prefix-sum) with ReLU features equals the explicit
    L x L generalized-attention estimator, with and without the final renormalisation."""
    Q, K, V = _inputs(9 + L, 2, 3, L, D)
    W, b = favor.orf_draw(10 + L, 3, M, D)
    kw = dict(kernel=favor.KERNEL_RELU, kernel_eps=1e-3, renormalize=renormalize)
    ob = favor.attn_bidir(Q, K, V, W, b, 1.0, **kw)
    oc, _ = favor.attn_causal(Q, K, V, W, b, 1.0, **kw)
    np.testing.assert_allclose(ob, favor.attn_explicit(Q, K, V, W, b, 1.0, False, **kw),
                               rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(oc, favor.attn_explicit(Q, K, V, W, b, 1.0, True, **kw),
                               rtol=1e-11, atol=1e-11)


def test_relu_denominator_positive_and_constant_values():
    """Non-negative features plus eps make D-hat > 0; V = 1 returns 1 (renormalised)
    and D-hat itself (not renormalised)."""
    Q, K, V = _inputs(11, 1, 2, 200, D, scale_qk=False)
    W, b = favor.orf_draw(12, 2, 64, D)
    kw = dict(kernel=favor.KERNEL_RELU, kernel_eps=1e-3)
    ones = np.ones_like(V)
    np.testing.assert_allclose(favor.attn_bidir(Q, K, ones, W, b, 1.0, **kw), 1.0, rtol=1e-12)
    Qp = favor.feature_map_relu(Q, W, 1.0)
    Kp = favor.feature_map_relu(K, W, 1.0)
    Dhat = Qp @ np.swapaxes(Kp, -1, -2).sum(-1, keepdims=True)
    assert np.all(Dhat > 0)
    off = favor.attn_bidir(Q, K, ones, W, b, 1.0, renormalize=False, **kw)
    np.testing.assert_allclose(off, np.broadcast_to(Dhat, off.shape), rtol=1e-12)
