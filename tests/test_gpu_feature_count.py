"""GPU parity for numbers of random features M other than the kernels' 64, 128
and 256 rows (any multiple of 16 up to 256): the library pads W'' with zero
rows whose features vanish, and every array the caller sees keeps M. Each
case is checked against the fp64 oracle run with exactly M features, and the
arrays are checked for writes past their M-sized extent (a sentinel tail).

Tolerances as everywhere: 1e-4 for fp32 inputs, 2e-2 for bf16 inputs.
"""
import numpy as np
import pytest

import workloads as wl
from helpers import TOL, parity, to_dev, to_host
from oracle import favor
from test_gpu_backward import _check_all, _host_grads, _oracle_grads, _oracle_w

pytestmark = pytest.mark.gpu

S64 = 64 ** -0.25
RELU = favor.KERNEL_RELU
SOFTMAX = favor.KERNEL_SOFTMAX
SENTINEL = 12345.0


def _fv():
    import paper_2006_03555_amd as fv
    return fv


def _qkv(B, H, L, dtype, seed):
    return wl.make_qkv(wl.Workload("t", "bidir", B, H, L, 64, 64, dtype, seed))


def _features(seed, H, M):
    W, b = favor.orf_draw(seed, H, M, 64)
    return W.astype(np.float32), b.astype(np.float32)


def _with_tail(shape, dtype):
    """A tensor of `shape` at the start of a buffer whose 64-element tail holds a
    sentinel; returns (view, buffer)."""
    import torch
    n = int(np.prod(shape))
    buf = torch.full((n + 64,), SENTINEL, dtype=dtype, device="cuda")
    return buf[:n].view(shape), buf


def _tail_intact(buf, n):
    import torch
    ref = torch.tensor(SENTINEL, dtype=buf.dtype, device=buf.device)
    return bool(torch.all(buf[n:] == ref).item())


@pytest.mark.parametrize("din,dout", [("f32", "f32"), ("bf16", "bf16")])
@pytest.mark.parametrize("M", [16, 48, 144, 208])
@pytest.mark.parametrize("kernel", [SOFTMAX, RELU])
def test_feature_map_any_m(din, dout, M, kernel):
    import torch
    fv = _fv()
    B, H, L = 2, 3, 150
    Q, _, _ = _qkv(B, H, L, din, seed=M + 1)
    W, b = _features(M, H, M)
    tdt = torch.bfloat16 if dout == "bf16" else torch.float32
    out, buf = _with_tail((B, H, L, M), tdt)
    fv.feature_map(to_dev(Q, din), to_dev(W), to_dev(b), S64, out=out, kernel=kernel)
    torch.cuda.synchronize()
    ref = favor.features(Q.astype(np.float64), W, b, S64, kernel, 1e-3)
    got = to_host(out)
    scale = np.max(np.abs(ref), axis=-1, keepdims=True)
    assert np.max(np.abs(got - ref) / scale) <= TOL[din if din == dout else "bf16"]
    assert _tail_intact(buf, B * H * L * M)


BIDIR_CASES = [
    # B, H, L, M, dtype, kernel, renormalize, denom_eps
    (1, 2, 300, 16, "f32", SOFTMAX, True, 0.0),
    (2, 2, 517, 48, "bf16", SOFTMAX, True, 0.0),
    (1, 3, 200, 80, "f32", RELU, True, 0.0),
    (1, 2, 1000, 208, "bf16", SOFTMAX, True, 0.3),
    (1, 2, 333, 240, "bf16", RELU, False, 0.0),
    (1, 1, 129, 112, "f32", SOFTMAX, False, 0.0),
]


@pytest.mark.parametrize("B,H,L,M,dtype,kernel,renorm,eps", BIDIR_CASES)
def test_bidir_any_m(B, H, L, M, dtype, kernel, renorm, eps):
    import torch
    fv = _fv()
    Q, K, V = _qkv(B, H, L, dtype, seed=L + M)
    W, b = _features(L + 2 * M, H, M)
    out = fv.attn_bidir(to_dev(Q, dtype), to_dev(K, dtype), to_dev(V, dtype), to_dev(W),
                        to_dev(b), S64, denom_eps=eps, kernel=kernel, renormalize=renorm)
    torch.cuda.synchronize()
    parity(to_host(out), Q, K, V, W, b, S64, False, dtype, eps=eps, kernel=kernel,
           renormalize=renorm)


CAUSAL_CASES = [
    # B, H, L, M, dtype, kernel
    (1, 2, 400, 48, "f32", SOFTMAX),
    (1, 2, 300, 112, "f32", RELU),
    (2, 2, 1100, 208, "bf16", SOFTMAX),
    (1, 3, 700, 16, "bf16", RELU),
    (1, 2, 250, 176, "bf16", SOFTMAX),
]


@pytest.mark.parametrize("B,H,L,M,dtype,kernel", CAUSAL_CASES)
def test_causal_any_m_with_states(B, H, L, M, dtype, kernel):
    """A carried state_in [.., M, d+1] and state_out against the oracle's, and no
    write past state_out's M rows."""
    import torch
    fv = _fv()
    Q, K, V = _qkv(B, H, L, dtype, seed=3 * L + M)
    W, b = _features(L + M, H, M)
    Qe, Ke, Ve = _qkv(B, H, 150, dtype, seed=M)
    _, S0 = favor.attn_causal(Qe, Ke, Ve, W, b, S64, kernel=kernel)
    S0 = S0.astype(np.float32)
    st_out, buf = _with_tail((B, H, M, 65), torch.float32)
    out = fv.attn_causal(to_dev(Q, dtype), to_dev(K, dtype), to_dev(V, dtype), to_dev(W),
                         to_dev(b), S64, state_in=to_dev(S0), state_out=st_out, kernel=kernel)
    torch.cuda.synchronize()
    parity(to_host(out), Q, K, V, W, b, S64, True, dtype, state_in=S0, kernel=kernel)
    _, ref_state = favor.attn_causal(Q, K, V, W, b, S64, state_in=S0, kernel=kernel)
    got = to_host(st_out)
    assert np.max(np.abs(got - ref_state)) <= TOL[dtype] * np.max(np.abs(ref_state))
    assert _tail_intact(buf, B * H * M * 65)


@pytest.mark.parametrize("M,dtype", [(80, "bf16"), (32, "f32")])
def test_both_any_m(M, dtype):
    import torch
    fv = _fv()
    B, H, L = 1, 2, 900
    Q, K, V = _qkv(B, H, L, dtype, seed=M)
    W, b = _features(M + 5, H, M)
    ob, oc = fv.attn_both(to_dev(Q, dtype), to_dev(K, dtype), to_dev(V, dtype), to_dev(W),
                          to_dev(b), S64)
    torch.cuda.synchronize()
    parity(to_host(ob), Q, K, V, W, b, S64, False, dtype)
    parity(to_host(oc), Q, K, V, W, b, S64, True, dtype)


def _bwd_inputs(B, H, L, M, dtype, seed):
    Q, K, V = _qkv(B, H, L, dtype, seed)
    dout = np.random.default_rng(seed + 7).standard_normal((B, H, L, 64)).astype(np.float32)
    if dtype == "bf16":
        import torch
        dout = torch.from_numpy(dout).to(torch.bfloat16).float().numpy()
    W, b = _features(seed + 3, H, M)
    return Q, K, V, dout, W, b


# With few cosine features the estimated denominator D-hat of some rows comes
# close to 0 (at M = 16 about one row in a thousand falls below 1% of
# sum |q'| |k'|), and the gradient of such a row amplifies the rounding of its
# features by that ratio; the gate is in units of the oracle's error scale,
# which grows with that ratio, so any inputs serve (the last two cases).
BACKWARD_CASES = [
    # B, H, L, M, dtype, kernel, causal, seed
    (1, 2, 300, 48, "f32", SOFTMAX, False, 348),
    (1, 2, 300, 48, "f32", SOFTMAX, True, 348),
    (1, 2, 700, 80, "bf16", RELU, False, 780),
    (1, 2, 700, 80, "bf16", RELU, True, 780),
    (2, 2, 1000, 208, "bf16", SOFTMAX, True, 1208),
    (1, 3, 333, 16, "f32", SOFTMAX, False, 430),
    (1, 3, 333, 16, "bf16", SOFTMAX, False, 17),
    (1, 3, 333, 32, "bf16", SOFTMAX, True, 18),
]


@pytest.mark.parametrize("B,H,L,M,dtype,kernel,causal,seed", BACKWARD_CASES)
def test_backward_any_m(B, H, L, M, dtype, kernel, causal, seed):
    """Gradients at M features, the causal ones with a carried state and a state
    gradient of M rows (no write past dstate_in's M rows)."""
    import torch
    fv = _fv()
    Q, K, V, dout, W, b = _bwd_inputs(B, H, L, M, dtype, seed=seed)
    args = [to_dev(x, dtype) for x in (Q, K, V)] + [to_dev(W), to_dev(b), S64,
                                                    to_dev(dout, dtype)]
    Wo = _oracle_w(W, M, dtype, kernel)
    if not causal:
        got = fv.attn_bidir_backward(*args, kernel=kernel)
        torch.cuda.synchronize()
        ref, scale, _ = _oracle_grads(Q, K, V, Wo, b, dout, False, kernel=kernel)
    else:
        Qe, Ke, Ve = _qkv(B, H, 150, dtype, seed=M + 2)
        _, S0 = favor.attn_causal(Qe, Ke, Ve, W, b, S64, kernel=kernel)
        S0 = S0.astype(np.float32)
        dS = np.random.default_rng(9).standard_normal(S0.shape).astype(np.float32) * 0.01
        ds_in, buf = _with_tail((B, H, M, 65), torch.float32)
        got = fv.attn_causal_backward(*args, state_in=to_dev(S0), dstate_out=to_dev(dS),
                                      dstate_in=ds_in, return_state_grad=True,
                                      kernel=kernel)
        torch.cuda.synchronize()
        ref, scale, rS = _oracle_grads(Q, K, V, Wo, b, dout, True, state_in=S0, dstate_out=dS,
                                       kernel=kernel)
        gS = to_host(got[3])
        assert np.max(np.abs(gS - rS)) <= TOL[dtype] * np.max(np.abs(rS))
        assert _tail_intact(buf, B * H * M * 65)
    _check_all(_host_grads(got), ref, dtype, scale)


# fp32 inputs at M > 128: the causal scan runs as two passes over the feature
# halves (the first stores each row's raw numerators and denominator)
FP32_CAUSAL_CASES = [
    # B, H, L, M, kernel, renormalize, denom_eps, causal segment rows
    (1, 2, 700, 256, SOFTMAX, True, 0.0, 0),
    (2, 1, 1100, 208, RELU, True, 0.0, 256),
    (1, 2, 333, 256, SOFTMAX, False, 0.0, 0),
    (1, 1, 513, 144, SOFTMAX, True, 0.4, 128),
]


@pytest.mark.parametrize("B,H,L,M,kernel,renorm,eps,segment", FP32_CAUSAL_CASES)
def test_fp32_causal_feature_halves(B, H, L, M, kernel, renorm, eps, segment):
    import torch
    fv = _fv()
    Q, K, V = _qkv(B, H, L, "f32", seed=L + M)
    W, b = _features(M + 11, H, M)
    Qe, Ke, Ve = _qkv(B, H, 90, "f32", seed=M + 3)
    _, S0 = favor.attn_causal(Qe, Ke, Ve, W, b, S64, kernel=kernel)
    S0 = S0.astype(np.float32)
    kw = dict(denom_eps=eps, kernel=kernel, renormalize=renorm, segment=segment)
    out, st = fv.attn_causal(to_dev(Q), to_dev(K), to_dev(V), to_dev(W), to_dev(b), S64,
                             state_in=to_dev(S0), return_state=True, **kw)
    torch.cuda.synchronize()
    parity(to_host(out), Q, K, V, W, b, S64, True, "f32", eps=eps, state_in=S0, kernel=kernel,
           renormalize=renorm)
    _, ref_state = favor.attn_causal(Q, K, V, W, b, S64, state_in=S0, kernel=kernel)
    assert np.max(np.abs(to_host(st) - ref_state)) <= 1e-4 * np.max(np.abs(ref_state))


def test_fp32_both_directions_feature_halves_and_saved_scales():
    """attn_both at fp32 M = 256: both outputs against the oracle, and the
    causal row scales written by the second pass equal the oracle's."""
    import torch
    from test_gpu_backward import _expected_row_scale
    fv = _fv()
    B, H, L, M = 1, 2, 900, 256
    Q, K, V = _qkv(B, H, L, "f32", seed=77)
    W, b = _features(78, H, M)
    rb = torch.empty((B, H, L), device="cuda")
    rc = torch.empty((B, H, L), device="cuda")
    ob, oc = fv.attn_both(to_dev(Q), to_dev(K), to_dev(V), to_dev(W), to_dev(b), S64,
                          row_scale_bidir=rb, row_scale_causal=rc)
    torch.cuda.synchronize()
    parity(to_host(ob), Q, K, V, W, b, S64, False, "f32")
    parity(to_host(oc), Q, K, V, W, b, S64, True, "f32")
    for causal, r in ((False, rb), (True, rc)):
        want = _expected_row_scale(Q, K, W, b, M, SOFTMAX, 0.0, causal)
        assert np.max(np.abs(to_host(r) - want) / np.abs(want)) <= 1e-4


# fp32 gradients beyond the kernels' LDS tables (128 features bidirectional, 64
# causal): feature slices whose parts add into dQ, dK, dV
FP32_BWD_CASES = [
    # B, H, L, M, kernel, causal, renormalize
    (1, 2, 300, 256, SOFTMAX, False, True),
    (1, 2, 333, 144, RELU, False, True),
    (1, 2, 300, 128, SOFTMAX, True, True),
    (1, 2, 400, 256, RELU, True, True),
    (1, 1, 257, 208, SOFTMAX, True, False),
]


@pytest.mark.parametrize("B,H,L,M,kernel,causal,renorm", FP32_BWD_CASES)
def test_fp32_backward_feature_slices(B, H, L, M, kernel, causal, renorm):
    import torch
    fv = _fv()
    Q, K, V, dout, W, b = _bwd_inputs(B, H, L, M, "f32", seed=L + M + 1)
    args = [to_dev(x) for x in (Q, K, V)] + [to_dev(W), to_dev(b), S64, to_dev(dout)]
    kw = dict(kernel=kernel, renormalize=renorm)
    names = ("dQ", "dK", "dV")
    if not causal:
        got = fv.attn_bidir_backward(*args, **kw)
        torch.cuda.synchronize()
        ref, scale, _ = _oracle_grads(Q, K, V, W, b, dout, False, **kw)
    else:
        Qe, Ke, Ve = _qkv(B, H, 120, "f32", seed=M + 4)
        _, S0 = favor.attn_causal(Qe, Ke, Ve, W, b, S64, **kw)
        S0 = S0.astype(np.float32)
        dS = np.random.default_rng(5).standard_normal(S0.shape).astype(np.float32) * 0.01
        got = fv.attn_causal_backward(*args, state_in=to_dev(S0), dstate_out=to_dev(dS),
                                      return_state_grad=True, **kw)
        torch.cuda.synchronize()
        ref, scale, rS = _oracle_grads(Q, K, V, W, b, dout, True, state_in=S0, dstate_out=dS,
                                       **kw)
        assert np.max(np.abs(to_host(got[3]) - rS)) <= 1e-4 * np.max(np.abs(rS))
    _check_all(_host_grads(got), ref, "f32", scale)


def test_fp32_backward_slices_with_saved_statistics():
    """attn_both at fp32 M = 256 saving the row scales, then both backward calls
    from the saved outputs: the gradients of the calls that recompute them."""
    import torch
    fv = _fv()
    B, H, L, M = 1, 2, 500, 256
    Q, K, V, dout, W, b = _bwd_inputs(B, H, L, M, "f32", seed=91)
    q, k, v, do = (to_dev(x) for x in (Q, K, V, dout))
    Wd, bd = to_dev(W), to_dev(b)
    rb = torch.empty((B, H, L), device="cuda")
    rc = torch.empty((B, H, L), device="cuda")
    ob, oc = fv.attn_both(q, k, v, Wd, bd, S64, row_scale_bidir=rb, row_scale_causal=rc)
    for f, o, r in ((fv.attn_bidir_backward, ob, rb), (fv.attn_causal_backward, oc, rc)):
        plain = f(q, k, v, Wd, bd, S64, do)[:3]
        saved = f(q, k, v, Wd, bd, S64, do, out=o, row_scale=r)[:3]
        torch.cuda.synchronize()
        _, scale, _ = _oracle_grads(Q, K, V, W, b, dout, f is fv.attn_causal_backward)
        _check_all(_host_grads(saved), _host_grads(plain), "f32", scale)
