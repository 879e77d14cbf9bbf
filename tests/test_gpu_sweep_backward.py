"""A seeded sweep of random configurations through the backward entry points
(favor_attn_bidir_backward, favor_attn_causal_backward, favor_attn_both_backward),
each against the fp64 oracle's gradients: B, H, ragged L, M (a multiple of 16;
cos features from 64, see test_gpu_sweep), dtype, feature kind, normalisation,
stabiliser, carried state with a state gradient, and saved or recomputed
forward statistics.
Gate as in test_gpu_backward (per tensor and row, in units of the oracle's
first-order error scale of that row).
"""
import numpy as np
import pytest

import workloads as wl
from helpers import TOL, to_dev, to_host
from oracle import favor
from test_gpu_backward import _check_all, _host_grads, _oracle_grads, _oracle_w

pytestmark = pytest.mark.gpu

S64 = 64 ** -0.25


def _configs(n=16, seed=31337):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        dtype = "f32" if rng.random() < 0.4 else "bf16"
        kernel = favor.KERNEL_RELU if rng.random() < 0.4 else favor.KERNEL_SOFTMAX
        renorm = bool(rng.random() < 0.8)
        out.append(dict(
            case=i, B=int(rng.integers(1, 3)), H=int(rng.integers(1, 3)),
            L=int(rng.choice([1, 40, 64, 129, 300, 700])),
            M=int(16 * rng.integers(1 if kernel == favor.KERNEL_RELU else 4, 17)),
            dtype=dtype, kernel=kernel, renorm=renorm,
            eps=float(rng.choice([0.0, 0.0, 0.3])) if renorm else 0.0,
            causal=bool(rng.random() < 0.5), state=bool(rng.random() < 0.5),
            saved=bool(renorm and rng.random() < 0.5)))
    return out


CONFIGS = _configs()


@pytest.mark.parametrize("cfg", CONFIGS, ids=[f"case{c['case']}" for c in CONFIGS])
def test_random_backward_configuration(cfg):
    import torch
    fv = __import__("paper_2006_03555_amd")
    print(f"\n{cfg}", flush=True)
    B, H, L, M, dtype = cfg["B"], cfg["H"], cfg["L"], cfg["M"], cfg["dtype"]
    Q, K, V = wl.make_qkv(wl.Workload("t", "bidir", B, H, L, 64, 64, dtype, 3000 + cfg["case"]))
    dout = np.random.default_rng(cfg["case"]).standard_normal((B, H, L, 64)).astype(np.float32)
    if dtype == "bf16":
        dout = torch.from_numpy(dout).to(torch.bfloat16).float().numpy()
    W, b = favor.orf_draw(4000 + cfg["case"], H, M, 64)
    W, b = W.astype(np.float32), b.astype(np.float32)
    kw = dict(kernel=cfg["kernel"], renormalize=cfg["renorm"], denom_eps=cfg["eps"])
    q, k, v, do = (to_dev(x, dtype) for x in (Q, K, V, dout))
    Wd, bd = to_dev(W), to_dev(b)
    Wo = _oracle_w(W, M, dtype, cfg["kernel"])
    names = ("dQ", "dK", "dV")
    if not cfg["causal"]:
        extra = {}
        if cfg["saved"]:
            r = torch.empty((B, H, L), device="cuda")
            o = fv.attn_bidir(q, k, v, Wd, bd, S64, row_scale=r, **kw)
            extra = dict(out=o, row_scale=r)
        got = fv.attn_bidir_backward(q, k, v, Wd, bd, S64, do, **kw, **extra)
        torch.cuda.synchronize()
        ref, scale, _ = _oracle_grads(Q, K, V, Wo, b, dout, False, **kw)
    else:
        S0 = dS = None
        if cfg["state"]:
            Qe, Ke, Ve = wl.make_qkv(wl.Workload("t", "bidir", B, H, 90, 64, 64, dtype, 11))
            _, S0 = favor.attn_causal(Qe, Ke, Ve, W, b, S64, kernel=cfg["kernel"])
            S0 = S0.astype(np.float32)
            dS = np.random.default_rng(3).standard_normal(S0.shape).astype(np.float32) * 0.01
        dev = lambda x: None if x is None else to_dev(x)
        extra = {}
        if cfg["saved"]:
            r = torch.empty((B, H, L), device="cuda")
            o = fv.attn_causal(q, k, v, Wd, bd, S64, state_in=dev(S0), row_scale=r, **kw)
            extra = dict(out=o, row_scale=r)
        got = fv.attn_causal_backward(q, k, v, Wd, bd, S64, do, state_in=dev(S0),
                                      dstate_out=dev(dS), return_state_grad=True, **kw, **extra)
        torch.cuda.synchronize()
        ref, scale, rS = _oracle_grads(Q, K, V, Wo, b, dout, True, state_in=S0, dstate_out=dS,
                                       **kw)
        assert np.max(np.abs(to_host(got[3]) - rS)) <= TOL[dtype] * max(np.max(np.abs(rS)), 1e-30)
    _check_all(_host_grads(got), ref, dtype, scale)


BOTH_CONFIGS = _configs(n=8, seed=4711)


@pytest.mark.parametrize("cfg", BOTH_CONFIGS, ids=[f"both{c['case']}" for c in BOTH_CONFIGS])
def test_random_both_backward_configuration(cfg):
    """favor_attn_both_backward on the same kind of random configuration (the
    causal flag unused): the sum of the oracle's bidirectional and causal
    gradients, gated by the sum of their error scales, and the causal state
    gradient."""
    import torch
    fv = __import__("paper_2006_03555_amd")
    print(f"\n{cfg}", flush=True)
    B, H, L, M, dtype = cfg["B"], cfg["H"], cfg["L"], cfg["M"], cfg["dtype"]
    Q, K, V = wl.make_qkv(wl.Workload("t", "bidir", B, H, L, 64, 64, dtype, 5000 + cfg["case"]))
    rng = np.random.default_rng(100 + cfg["case"])
    douts = [rng.standard_normal((B, H, L, 64)).astype(np.float32) for _ in range(2)]
    if dtype == "bf16":
        douts = [torch.from_numpy(x).to(torch.bfloat16).float().numpy() for x in douts]
    W, b = favor.orf_draw(6000 + cfg["case"], H, M, 64)
    W, b = W.astype(np.float32), b.astype(np.float32)
    kw = dict(kernel=cfg["kernel"], renormalize=cfg["renorm"], denom_eps=cfg["eps"])
    q, k, v, db, dc = (to_dev(x, dtype) for x in (Q, K, V, *douts))
    Wd, bd = to_dev(W), to_dev(b)
    Wo = _oracle_w(W, M, dtype, cfg["kernel"])
    S0 = dS = None
    if cfg["state"]:
        Qe, Ke, Ve = wl.make_qkv(wl.Workload("t", "bidir", B, H, 90, 64, 64, dtype, 12))
        _, S0 = favor.attn_causal(Qe, Ke, Ve, W, b, S64, kernel=cfg["kernel"])
        S0 = S0.astype(np.float32)
        dS = np.random.default_rng(4).standard_normal(S0.shape).astype(np.float32) * 0.01
    dev = lambda x: None if x is None else to_dev(x)
    extra = {}
    if cfg["saved"]:
        rb = torch.empty((B, H, L), device="cuda")
        rc = torch.empty((B, H, L), device="cuda")
        ob, oc = fv.attn_both(q, k, v, Wd, bd, S64, state_in=dev(S0), row_scale_bidir=rb,
                              row_scale_causal=rc, **kw)
        extra = dict(out_bidir=ob, row_scale_bidir=rb, out_causal=oc, row_scale_causal=rc)
    got = fv.attn_both_backward(q, k, v, Wd, bd, S64, db, dc, state_in=dev(S0),
                                dstate_out=dev(dS), return_state_grad=True, **kw, **extra)
    torch.cuda.synchronize()
    rb_, sb, _ = _oracle_grads(Q, K, V, Wo, b, douts[0], False, **kw)
    rc_, sc, rS = _oracle_grads(Q, K, V, Wo, b, douts[1], True, state_in=S0, dstate_out=dS,
                                **kw)
    assert np.max(np.abs(to_host(got[3]) - rS)) <= TOL[dtype] * max(np.max(np.abs(rS)), 1e-30)
    _check_all(_host_grads(got), {n: rb_[n] + rc_[n] for n in rb_}, dtype,
               {n: sb[n] + sc[n] for n in sb})
