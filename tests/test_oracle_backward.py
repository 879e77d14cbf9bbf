"""Pins of the oracle's backward pass (oracle.backward), CPU only.

The gradients are hand-derived; they are pinned by two things that do not share
that derivation: central finite differences of the (separately pinned) forward
oracle, and PyTorch autograd through the explicit L x L estimator written here
with torch operations. Plus the exact invariants the method has.
"""
import numpy as np
import pytest
import torch

from oracle import backward as bw
from oracle import favor

D = 4


def _setup(seed, B, H, L, M, d=D, scale=1.0):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((B, H, L, d)) * scale
    K = rng.standard_normal((B, H, L, d)) * scale
    V = rng.standard_normal((B, H, L, d))
    W, b = favor.orf_draw(seed + 1, H, M, d)
    dout = rng.standard_normal((B, H, L, d))
    return Q, K, V, W, b, dout


def _loss_bidir(Q, K, V, W, b, s, dout, **kw):
    return float(np.sum(dout * favor.attn_bidir(Q, K, V, W, b, s, **kw)))


def _loss_causal(Q, K, V, W, b, s, dout, state_in=None, dstate_out=None, **kw):
    out, st = favor.attn_causal(Q, K, V, W, b, s, state_in=state_in, **kw)
    val = float(np.sum(dout * out))
    if dstate_out is not None:
        val += float(np.sum(dstate_out * st))
    return val


def _fd(f, x, direction, h=1e-6):
    return (f(x + h * direction) - f(x - h * direction)) / (2 * h)


KINDS = [
    dict(kernel=favor.KERNEL_SOFTMAX),
    dict(kernel=favor.KERNEL_SOFTMAX, denom_eps=0.3),
    dict(kernel=favor.KERNEL_SOFTMAX, renormalize=False),
    dict(kernel=favor.KERNEL_RELU),
    dict(kernel=favor.KERNEL_RELU, renormalize=False, kernel_eps=0.01),
]


@pytest.mark.parametrize("kw", KINDS)
def test_bidir_backward_matches_finite_differences(kw):
    s = 0.7
    Q, K, V, W, b, dout = _setup(3, 1, 2, 9, 8)
    dQ, dK, dV = bw.attn_bidir_backward(Q, K, V, W, b, s, dout, **kw)
    rng = np.random.default_rng(4)
    for name, x, g in (("Q", Q, dQ), ("K", K, dK), ("V", V, dV)):
        E = rng.standard_normal(x.shape)

        def f(xx, name=name):
            args = {"Q": Q, "K": K, "V": V}
            args[name] = xx
            return _loss_bidir(args["Q"], args["K"], args["V"], W, b, s, dout, **kw)

        fd = _fd(f, x, E)
        an = float(np.sum(g * E))
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)


@pytest.mark.parametrize("kw", KINDS)
def test_causal_backward_matches_finite_differences(kw):
    s = 0.7
    Q, K, V, W, b, dout = _setup(5, 1, 2, 9, 8)
    rng = np.random.default_rng(6)
    M = W.shape[1]
    S0 = rng.standard_normal((1, 2, M, D + 1)) * 0.5
    S0[..., D] = np.abs(S0[..., D]) + 1.0
    if kw.get("kernel") == favor.KERNEL_SOFTMAX and kw.get("renormalize", True):
        S0 = None   # a signed state_in can cancel the softmax denominators; tested below
    dS = rng.standard_normal((1, 2, M, D + 1))
    dQ, dK, dV, dS0 = bw.attn_causal_backward(Q, K, V, W, b, s, dout, state_in=S0,
                                              dstate_out=dS, **kw)
    args0 = {"Q": Q, "K": K, "V": V, "S": S0}
    items = [("Q", dQ), ("K", dK), ("V", dV)] + ([("S", dS0)] if S0 is not None else [])
    for name, g in items:
        x = args0[name]
        E = rng.standard_normal(x.shape)

        def f(xx, name=name):
            a = dict(args0)
            a[name] = xx
            return _loss_causal(a["Q"], a["K"], a["V"], W, b, s, dout, a["S"], dS, **kw)

        fd = _fd(f, x, E)
        an = float(np.sum(g * E))
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)


def test_causal_backward_state_in_gradient_softmax():
    """dstate_in for softmax features with a positive state (denominators stay away from 0)."""
    s = 0.5
    Q, K, V, W, b, dout = _setup(7, 1, 1, 7, 8)
    M = W.shape[1]
    rng = np.random.default_rng(8)
    S0 = np.abs(rng.standard_normal((1, 1, M, D + 1))) + 0.5
    _, _, _, dS0 = bw.attn_causal_backward(Q, K, V, W, b, s, dout, state_in=S0)
    E = rng.standard_normal(S0.shape)
    fd = _fd(lambda x: _loss_causal(Q, K, V, W, b, s, dout, x), S0, E)
    assert abs(fd - float(np.sum(dS0 * E))) <= 1e-6 * max(1.0, abs(fd))


def _torch_features(X, W, b, s, kernel, keps):
    Xs = s * X
    proj = Xs @ W.transpose(-1, -2)
    M = W.shape[-2]
    if kernel == favor.KERNEL_RELU:
        return torch.relu(proj) / M ** 0.5 + keps
    D = torch.exp(0.5 * (Xs * Xs).sum(-1, keepdim=True))
    return D * (2.0 / M) ** 0.5 * torch.cos(proj + b[..., None, :])


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("kw", KINDS)
def test_backward_matches_autograd_of_explicit_estimator(causal, kw):
    """Autograd through A-hat = Q' K'^T (tril when causal), D-hat^-1 A-hat V."""
    s = 0.6
    Q, K, V, W, b, dout = _setup(9, 2, 2, 11, 12)
    kernel = kw.get("kernel", favor.KERNEL_SOFTMAX)
    keps = kw.get("kernel_eps", 1e-3)
    eps = kw.get("denom_eps", 0.0)
    renorm = kw.get("renormalize", True)
    t = lambda a: torch.tensor(a, dtype=torch.float64, requires_grad=True)
    tQ, tK, tV = t(Q), t(K), t(V)
    tW = torch.tensor(W, dtype=torch.float64)
    tb = torch.tensor(b, dtype=torch.float64)
    Qp = _torch_features(tQ, tW, tb, s, kernel, keps)
    Kp = _torch_features(tK, tW, tb, s, kernel, keps)
    A = Qp @ Kp.transpose(-1, -2)
    if causal:
        A = torch.tril(A)
    out = A @ tV
    if renorm:
        out = out / (A.sum(-1, keepdim=True) + eps)
    (out * torch.tensor(dout)).sum().backward()
    if causal:
        dQ, dK, dV, _ = bw.attn_causal_backward(Q, K, V, W, b, s, dout, **kw)
    else:
        dQ, dK, dV = bw.attn_bidir_backward(Q, K, V, W, b, s, dout, **kw)
    for got, ref in ((dQ, tQ.grad), (dK, tK.grad), (dV, tV.grad)):
        ref = ref.numpy()
        assert np.max(np.abs(got - ref)) <= 1e-10 * max(1.0, np.max(np.abs(ref)))


def test_feature_vjps_match_finite_differences():
    s = 0.8
    rng = np.random.default_rng(10)
    X = rng.standard_normal((2, 3, 5, D))
    W, b = favor.orf_draw(11, 3, 12, D)
    dXp = rng.standard_normal((2, 3, 5, 12))
    E = rng.standard_normal(X.shape)
    for kernel in (favor.KERNEL_SOFTMAX, favor.KERNEL_RELU):
        g = bw.features_vjp(X, W, b, s, dXp, kernel)
        f = lambda x: float(np.sum(dXp * favor.features(x, W, b, s, kernel)))
        fd = _fd(f, X, E)
        assert abs(fd - float(np.sum(g * E))) <= 1e-7 * max(1.0, abs(fd))


@pytest.mark.parametrize("kernel", [favor.KERNEL_SOFTMAX, favor.KERNEL_RELU])
def test_value_gradient_sums_to_output_gradient(kernel):
    """Renormalised rows are affine in V with weights summing to 1: shifting every
    value by c shifts every output by c, so sum_j dV_j = sum_i dout_i."""
    Q, K, V, W, b, dout = _setup(12, 1, 2, 10, 16)
    _, _, dVb = bw.attn_bidir_backward(Q, K, V, W, b, 0.5, dout, kernel=kernel)
    _, _, dVc, _ = bw.attn_causal_backward(Q, K, V, W, b, 0.5, dout, kernel=kernel)
    ref = dout.sum(axis=-2)
    assert np.allclose(dVb.sum(axis=-2), ref, atol=1e-10)
    assert np.allclose(dVc.sum(axis=-2), ref, atol=1e-10)


def test_renormalised_output_ignores_the_radial_direction_of_queries():
    """With eps = 0 the output is invariant to rescaling a query's features; for
    softmax features D_Q carries the norm of q, so the query gradient of the
    renormalised bidirectional output has no component along the feature scale.
    Checked via the ReLU case, where Q' is positively homogeneous in q up to
    kernel_eps: with kernel_eps = 0, dQ_i . q_i = 0."""
    Q, K, V, W, b, dout = _setup(13, 1, 1, 8, 16)
    dQ, _, _ = bw.attn_bidir_backward(Q, K, V, W, b, 1.0, dout, kernel=favor.KERNEL_RELU,
                                      kernel_eps=0.0)
    assert np.max(np.abs(np.sum(dQ * Q, axis=-1))) <= 1e-10


def test_causal_backward_in_pieces_equals_one_call():
    """The state hand-off: the backward of two pieces, with the second piece's
    dstate_in passed as the first piece's dstate_out, equals one backward."""
    Q, K, V, W, b, dout = _setup(14, 1, 2, 12, 8)
    kw = dict(kernel=favor.KERNEL_RELU)
    dQ, dK, dV, _ = bw.attn_causal_backward(Q, K, V, W, b, 0.5, dout, **kw)
    c = 5
    _, s1 = favor.attn_causal(Q[..., :c, :], K[..., :c, :], V[..., :c, :], W, b, 0.5, **kw)
    dQ2, dK2, dV2, dS1 = bw.attn_causal_backward(Q[..., c:, :], K[..., c:, :], V[..., c:, :],
                                                 W, b, 0.5, dout[..., c:, :], state_in=s1, **kw)
    dQ1, dK1, dV1, _ = bw.attn_causal_backward(Q[..., :c, :], K[..., :c, :], V[..., :c, :],
                                               W, b, 0.5, dout[..., :c, :], dstate_out=dS1, **kw)
    for whole, a, z in ((dQ, dQ1, dQ2), (dK, dK1, dK2), (dV, dV1, dV2)):
        assert np.allclose(np.concatenate([a, z], axis=-2), whole, atol=1e-12)
