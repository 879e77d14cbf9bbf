"""A seeded sweep of random call configurations through every forward entry
point (favor_feature_map, favor_attn_bidir, favor_attn_causal, favor_attn_both),
each against the fp64 oracle on the same inputs and features: B, H, ragged L,
any M that is a multiple of 16, in/out dtypes, feature kind, renormalisation,
stabiliser, causal segment length, the scan's chunk length (bf16 cases cycle
through 32, 64 and the default) and a carried state (cos features from M 64,
ReLU features from M 16; a second list takes cos features at M 16 to 48 and
gates them by E_cond alone, as are the unnormalised outputs, whose rows
cancel). The configurations are drawn once from a fixed seed, so a failure
names a reproducible case.

Tolerances as everywhere: 1e-4 for fp32 inputs, 2e-2 for bf16 inputs.
"""
import numpy as np
import pytest

import workloads as wl
from helpers import TOL, parity, to_dev, to_host
from oracle import favor

pytestmark = pytest.mark.gpu

S64 = 64 ** -0.25


def _configs(n=24, seed=20261202):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        dtype = "f32" if rng.random() < 0.4 else "bf16"
        kernel = favor.KERNEL_RELU if rng.random() < 0.4 else favor.KERNEL_SOFTMAX
        out.append(dict(
            case=i,
            B=int(rng.integers(1, 3)), H=int(rng.integers(1, 4)),
            L=int(rng.choice([1, 17, 63, 64, 65, 200, 511, 777, 1300])),
            # cos features at M < 64 can leave a row's D-hat near 0 (E_row has no
            # conditioning term): small M is swept with ReLU features
            M=int(16 * rng.integers(1 if kernel == favor.KERNEL_RELU else 4, 17)),
            dtype=dtype,
            out_dtype="f32" if dtype == "bf16" and rng.random() < 0.3 else dtype,
            kernel=kernel,
            renorm=bool(rng.random() < 0.8),
            eps=float(rng.choice([0.0, 0.0, 0.25])),
            segment=int(rng.choice([0, 0, 64, 192, 512])),
            state=bool(rng.random() < 0.5),
            kind=int(rng.choice([favor.RF_ORTHO_CHI, favor.RF_IID, favor.RF_HADAMARD])),
        ))
    return out


CONFIGS = _configs()


def _small_m_configs(n=8, seed=777):
    """Cosine features at M 16 to 48: D-hat can nearly cancel on some rows, so
    these are gated by E_cond alone (E_row is printed)."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        dtype = "f32" if rng.random() < 0.5 else "bf16"
        out.append(dict(
            case=100 + i,
            B=int(rng.integers(1, 3)), H=int(rng.integers(1, 4)),
            L=int(rng.choice([1, 63, 65, 200, 777, 1300])),
            M=int(16 * rng.integers(1, 4)),
            dtype=dtype, out_dtype=dtype, kernel=favor.KERNEL_SOFTMAX,
            renorm=bool(rng.random() < 0.8),
            eps=0.0,
            segment=int(rng.choice([0, 64, 192])),
            state=bool(rng.random() < 0.5),
            kind=int(rng.choice([favor.RF_ORTHO_CHI, favor.RF_IID, favor.RF_HADAMARD])),
            gate="cond",
        ))
    return out


CONFIGS_SMALL_M = _small_m_configs()


def _check(got, ref, tol):
    scale = np.max(np.abs(ref), axis=-1, keepdims=True)
    assert np.max(np.abs(got - ref) / np.maximum(scale, 1e-30)) <= tol


@pytest.mark.parametrize("cfg", CONFIGS + CONFIGS_SMALL_M,
                         ids=[f"case{c['case']}" for c in CONFIGS + CONFIGS_SMALL_M])
def test_random_configuration(cfg):
    import torch
    fv = __import__("paper_2006_03555_amd")
    B, H, L, M, dtype = cfg["B"], cfg["H"], cfg["L"], cfg["M"], cfg["dtype"]
    # bf16 cases cycle through 32-token chunks, 64-token chunks and the library
    # default (32 for M <= 128, else 64); fp32 inputs take 64
    chunk = (0, 32, 64)[cfg["case"] % 3] if dtype == "bf16" else 0
    eff = chunk or (32 if dtype == "bf16" and M <= 128 else 64)
    print(f"\n{cfg} chunk {eff}", flush=True)
    Q, K, V = wl.make_qkv(wl.Workload("t", "bidir", B, H, L, 64, 64, dtype,
                                      1000 + cfg["case"]))
    W, b = favor.orf_draw(2000 + cfg["case"], H, M, 64, cfg["kind"])
    W, b = W.astype(np.float32), b.astype(np.float32)
    kw = dict(kernel=cfg["kernel"], renormalize=cfg["renorm"])
    odt = torch.float32 if cfg["out_dtype"] == "f32" else torch.bfloat16
    tol = TOL[dtype]
    q, k, v, Wd, bd = to_dev(Q, dtype), to_dev(K, dtype), to_dev(V, dtype), to_dev(W), to_dev(b)
    S0 = None
    if cfg["state"]:
        Qe, Ke, Ve = wl.make_qkv(wl.Workload("t", "bidir", B, H, 100, 64, 64, dtype, 7))
        _, S0 = favor.attn_causal(Qe, Ke, Ve, W, b, S64, **kw)
        S0 = S0.astype(np.float32)

    Xp = fv.feature_map(q, Wd, bd, S64, out_dtype=odt, kernel=cfg["kernel"])
    ob = fv.attn_bidir(q, k, v, Wd, bd, S64, denom_eps=cfg["eps"], out_dtype=odt, **kw)
    oc, st = fv.attn_causal(q, k, v, Wd, bd, S64, denom_eps=cfg["eps"], segment=cfg["segment"],
                            state_in=None if S0 is None else to_dev(S0), return_state=True,
                            out_dtype=odt, chunk=chunk, **kw)
    ob2, oc2 = fv.attn_both(q, k, v, Wd, bd, S64, denom_eps=cfg["eps"], segment=cfg["segment"],
                            state_in=None if S0 is None else to_dev(S0), out_dtype=odt,
                            chunk=chunk, **kw)
    torch.cuda.synchronize()

    ref_f = favor.features(Q.astype(np.float64), W, b, S64, cfg["kernel"], 1e-3)
    _check(to_host(Xp), ref_f, tol if cfg["out_dtype"] == dtype else TOL["bf16"])
    ptol = tol if cfg["out_dtype"] == dtype else TOL["bf16"]
    # an unnormalised output is the numerator Q'(S + K'^T V) itself: its rows
    # cancel (cos weights of both signs; any weights against values of both
    # signs, with no denominator whose rounding follows the numerator's), and
    # E_row, with no conditioning term, bounds nothing there; E_cond, scaled by
    # the absolute-value sums, is the gate
    gate = cfg.get("gate", "both" if cfg["renorm"] else "cond")
    for out in (ob, ob2):
        e = parity(to_host(out), Q, K, V, W, b, S64, False, dtype, eps=cfg["eps"], tol=ptol,
                   kernel=cfg["kernel"], renormalize=cfg["renorm"], gate=gate)
        print(f"bidir E_row {e[0]:.2e} E_cond {e[1]:.2e}", flush=True)
    for out in (oc, oc2):
        e = parity(to_host(out), Q, K, V, W, b, S64, True, dtype, eps=cfg["eps"], tol=ptol,
                   state_in=S0, kernel=cfg["kernel"], renormalize=cfg["renorm"], gate=gate)
        print(f"causal E_row {e[0]:.2e} E_cond {e[1]:.2e}", flush=True)
    _, ref_state = favor.attn_causal(Q, K, V, W, b, S64, state_in=S0, **kw)
    assert np.max(np.abs(to_host(st) - ref_state)) <= tol * np.max(np.abs(ref_state))
