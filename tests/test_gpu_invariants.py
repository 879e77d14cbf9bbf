"""GPU checks of the method's exact invariants, special cases and numerical edge
cases, through the C ABI, against what the paper's formulas fix:

  * input_scale = 1 (the workloads' d^-1/4-scaled tensors taken as the
    logits themselves; Sec. 2.1 evaluated literally): D-hat cancels on many
    rows, so the gate is the conditioning-aware E_cond alone; E_row and the
    distribution of kappa = S_d / |D-hat| are printed.
  * V = 1 gives 1 (Algorithm 1 divides Buf3 by buf4, which is Buf3 for V = 1).
  * Causal row 1 is V_1 (Eq. cumsum with one key); the last causal row is the
    last bidirectional row (the prefix at i = L is the whole sum).
  * Q = K = 0: every feature is sqrt(2/M) cos(b_m) (Sec. 2.3), so every pair
    of rows has the same weight and the output is the mean of V (bidirectional)
    or the running mean of V_1..V_i (causal).
  * A zero denominator (Algorithm 1 divides by buf4): with ReLU features,
    kernel_eps = 0 and Q = K = 0 every feature is exactly 0 in any precision,
    so out = 0/0 = NaN on every row, as in the oracle; a stabiliser turns it
    into 0, and so does switching renormalisation off. (Cosine features cannot
    be made exactly 0: pi/2 is not representable, so cos(b) only nearly
    vanishes and the ratio stays the mean of V.)
  * A NaN key: every bidirectional row of its head is NaN; causal rows of
    earlier 64-token chunks are untouched, bit for bit. Rows of the key's own
    chunk before it may also turn NaN (the masked block product multiplies the
    zeroed weights by the NaN values) and are not checked.
"""
import numpy as np
import pytest

import workloads as wl
from helpers import TOL, parity, to_dev, to_host
from oracle import favor, metrics

pytestmark = pytest.mark.gpu

S64 = 64 ** -0.25
SOFTMAX = favor.KERNEL_SOFTMAX
RELU = favor.KERNEL_RELU


def _fv():
    import paper_2006_03555_amd as fv
    return fv


def _qkv(B, H, L, dtype, seed):
    return wl.make_qkv(wl.Workload("t", "bidir", B, H, L, 64, 64, dtype, seed))


def _features(seed, H, M, kind=favor.RF_ORTHO_CHI):
    W, b = favor.orf_draw(seed, H, M, 64, kind)
    return W.astype(np.float32), b.astype(np.float32)


# ------------------------------------------------------------ input_scale = 1
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("direction", ["bidir", "causal", "both"])
def test_input_scale_one_stress_mode(dtype, direction):
    import torch
    fv = _fv()
    B, H, L, M = 1, 2, 1000, 256
    Q, K, V = _qkv(B, H, L, dtype, seed=303)
    W, b = _features(404, H, M)
    q, k, v = (to_dev(x, dtype) for x in (Q, K, V))
    Wd, bd = to_dev(W), to_dev(b)
    outs = []
    if direction in ("bidir", "both"):
        outs.append((False, fv.attn_bidir(q, k, v, Wd, bd, 1.0)))
    if direction in ("causal", "both"):
        outs.append((True, fv.attn_causal(q, k, v, Wd, bd, 1.0)))
    if direction == "both":
        ob, oc = fv.attn_both(q, k, v, Wd, bd, 1.0)
        outs += [(False, ob), (True, oc)]
    torch.cuda.synchronize()
    for causal, out in outs:
        st = {}
        e_row, e_cond = parity(to_host(out), Q, K, V, W, b, 1.0, causal, dtype, gate="cond",
                               stats=st)
        kap = st["kappa"]
        print(f"\ns=1 {dtype} {'causal' if causal else 'bidir'}: E_cond {e_cond:.2e} "
              f"E_row {e_row:.2e} kappa median {np.median(kap):.1f} p90 "
              f"{np.quantile(kap, 0.9):.1f} max {kap.max():.3g}", flush=True)


# ------------------------------------------------------------ V = 1
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kernel", [SOFTMAX, RELU])
def test_values_one_give_one(dtype, kernel):
    import torch
    fv = _fv()
    Q, K, _ = _qkv(2, 2, 777, dtype, seed=17)
    V = np.ones_like(Q)
    W, b = _features(18, 2, 256)
    q, k, v = (to_dev(x, dtype) for x in (Q, K, V))
    ob = fv.attn_bidir(q, k, v, to_dev(W), to_dev(b), S64, kernel=kernel)
    oc = fv.attn_causal(q, k, v, to_dev(W), to_dev(b), S64, kernel=kernel)
    ob2, oc2 = fv.attn_both(q, k, v, to_dev(W), to_dev(b), S64, kernel=kernel)
    torch.cuda.synchronize()
    # fp32: the same sums over the same features in numerator and denominator;
    # bf16: one rounding of the output (spacing 2^-8 below 1, 2^-7 above)
    bound = 1e-5 if dtype == "f32" else 2.0 ** -7
    for o in (ob, oc, ob2, oc2):
        err = float(np.max(np.abs(to_host(o) - 1.0)))
        print(f"\nV=1 {dtype} kernel {kernel}: max |out - 1| = {err:.2e}", flush=True)
        assert err <= bound


# ------------------------------------------------------------ causal ends
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("L", [1, 64, 1000])
def test_causal_first_row_is_v1_and_last_row_is_bidirectional(dtype, L):
    import torch
    fv = _fv()
    Q, K, V = _qkv(2, 3, L, dtype, seed=27 + L)
    W, b = _features(28, 3, 256)
    q, k, v = (to_dev(x, dtype) for x in (Q, K, V))
    oc = to_host(fv.attn_causal(q, k, v, to_dev(W), to_dev(b), S64))
    ob = to_host(fv.attn_bidir(q, k, v, to_dev(W), to_dev(b), S64))
    torch.cuda.synchronize()
    first = metrics.err_row(oc[..., 0, :], V[..., 0, :])
    last = metrics.err_row(oc[..., -1, :], ob[..., -1, :])
    print(f"\n{dtype} L {L}: row 1 vs V_1 {first:.2e}; last causal vs bidir {last:.2e}",
          flush=True)
    assert first <= (1e-5 if dtype == "f32" else 1e-2)
    assert last <= TOL[dtype]


# ------------------------------------------------------------ Q = K = 0
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kernel", [SOFTMAX, RELU])
@pytest.mark.parametrize("M", [64, 256])
def test_zero_queries_and_keys_give_means(dtype, kernel, M):
    import torch
    fv = _fv()
    B, H, L = 1, 2, 700
    _, _, V = _qkv(B, H, L, dtype, seed=37)
    Z = np.zeros_like(V)
    W, b = _features(38, H, M)
    z, v = to_dev(Z, dtype), to_dev(V, dtype)
    ob = to_host(fv.attn_bidir(z, z, v, to_dev(W), to_dev(b), S64, kernel=kernel))
    oc = to_host(fv.attn_causal(z, z, v, to_dev(W), to_dev(b), S64, kernel=kernel))
    ob2, oc2 = map(to_host, fv.attn_both(z, z, v, to_dev(W), to_dev(b), S64, kernel=kernel))
    torch.cuda.synchronize()
    Vd = V.astype(np.float64)
    mean = np.broadcast_to(Vd.mean(axis=-2, keepdims=True), Vd.shape)
    run = np.cumsum(Vd, axis=-2) / np.arange(1, L + 1)[:, None]
    tol = 1e-5 if dtype == "f32" else TOL[dtype]
    for got, want in ((ob, mean), (ob2, mean), (oc, run), (oc2, run)):
        # the ratio of equal weights is the plain mean; all weights share one
        # sign (kappa = 1), so the row-relative error is the right gate
        e = metrics.err_row(got, want)
        print(f"\nQ=K=0 {dtype} kernel {kernel} M {M}: E_row {e:.2e}", flush=True)
        assert e <= tol


# ------------------------------------------------------------ D-hat = 0
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_zero_denominator_gives_nan_rows_like_the_oracle(dtype):
    import torch
    fv = _fv()
    B, H, L, M = 1, 2, 300, 128
    _, _, V = _qkv(B, H, L, dtype, seed=47)
    Z = np.zeros_like(V)
    W, b = _features(48, H, M)
    z, v, Wd, bd = to_dev(Z, dtype), to_dev(V, dtype), to_dev(W), to_dev(b)
    kw = dict(kernel=RELU, kernel_eps=0.0)
    with np.errstate(invalid="ignore", divide="ignore"):
        refb = favor.attn_bidir(Z, Z, V, W, b, S64, **kw)
        refc, _ = favor.attn_causal(Z, Z, V, W, b, S64, **kw)
    assert np.all(np.isnan(refb)) and np.all(np.isnan(refc))
    ob = fv.attn_bidir(z, z, v, Wd, bd, S64, **kw)
    oc = fv.attn_causal(z, z, v, Wd, bd, S64, **kw)
    ob2, oc2 = fv.attn_both(z, z, v, Wd, bd, S64, **kw)
    # a stabiliser makes the row 0 / eps = 0; no renormalisation returns Buf3 = 0
    eb = fv.attn_bidir(z, z, v, Wd, bd, S64, denom_eps=0.5, **kw)
    ec = fv.attn_causal(z, z, v, Wd, bd, S64, denom_eps=0.5, **kw)
    nb = fv.attn_bidir(z, z, v, Wd, bd, S64, renormalize=False, **kw)
    nc = fv.attn_causal(z, z, v, Wd, bd, S64, renormalize=False, **kw)
    torch.cuda.synchronize()
    for o in (ob, oc, ob2, oc2):
        assert torch.isnan(o).all()
    for o in (eb, ec, nb, nc):
        assert torch.count_nonzero(o) == 0


# ------------------------------------------------------------ NaN inputs
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_nan_key_reaches_only_its_head_and_later_chunks(dtype):
    import torch
    fv = _fv()
    B, H, L, M, j = 2, 2, 1000, 256, 700
    Q, K, V = _qkv(B, H, L, dtype, seed=57)
    W, b = _features(58, H, M)
    q, k, v, Wd, bd = tuple(to_dev(x, dtype) for x in (Q, K, V)) + (to_dev(W), to_dev(b))
    for segment in (0, 128):
        kb = k.clone()
        kb[1, 0, j, 5] = float("nan")
        cb = fv.attn_bidir(q, k, v, Wd, bd, S64)
        cc = fv.attn_causal(q, k, v, Wd, bd, S64, segment=segment)
        ob = fv.attn_bidir(q, kb, v, Wd, bd, S64)
        oc = fv.attn_causal(q, kb, v, Wd, bd, S64, segment=segment)
        torch.cuda.synchronize()
        assert torch.isnan(ob[1, 0]).all()
        assert torch.isnan(oc[1, 0, j:]).all()
        start = 64 * (j // 64)
        assert torch.equal(oc[1, 0, :start], cc[1, 0, :start])
        for bi, hi in ((0, 0), (0, 1), (1, 1)):
            assert torch.equal(ob[bi, hi], cb[bi, hi])
            assert torch.equal(oc[bi, hi], cc[bi, hi])


# ------------------------------------------------------------ caller's stream
def test_side_stream_without_workspace_is_not_raced():
    """A call on a side stream without a workspace: the binding allocates the
    outputs and the temporary workspace on that stream, so memory the current
    stream allocates and overwrites meanwhile cannot be the workspace the
    delayed side-stream kernels still use."""
    import torch
    fv = _fv()
    dtype = "bf16"
    B, H, L, M = 2, 4, 3000, 256
    Q, K, V = _qkv(B, H, L, dtype, seed=67)
    W, b = _features(68, H, M)
    q, k, v, Wd, bd = tuple(to_dev(x, dtype) for x in (Q, K, V)) + (to_dev(W), to_dev(b))
    refb, refc = fv.attn_both(q, k, v, Wd, bd, S64)
    refc1 = fv.attn_causal(q, k, v, Wd, bd, S64)
    torch.cuda.synchronize()
    g = fv.make_desc(B, H, L, 64, M, fv.BF16, fv.BF16, S64)
    sizes = [fv.workspace_size(g, c) for c in (0, 1, 2)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        torch.cuda._sleep(20_000_000)        # hold the side stream back
    ob, oc = fv.attn_both(q, k, v, Wd, bd, S64, stream=side)
    oc1 = fv.attn_causal(q, k, v, Wd, bd, S64, stream=side)
    junk = [torch.full((n // 4 + 1,), float("nan"), device="cuda") for n in sizes * 3]
    torch.cuda.synchronize()
    del junk
    assert torch.equal(ob, refb) and torch.equal(oc, refc) and torch.equal(oc1, refc1)


# ------------------------------------------------------------ concurrent calls
def test_concurrent_calls_on_two_streams_match_serial_calls():
    """The library holds no state between calls (beyond the no-allocation
    entry point's documented scratch): two calls running at the same time on
    two streams, each with its own workspace, give bitwise the results of the
    same calls made one after the other."""
    import torch
    fv = _fv()
    B, H, L, M = 2, 4, 2000, 256
    Q, K, V = _qkv(B, H, L, "bf16", seed=71)
    W, b = _features(72, H, M)
    a = tuple(to_dev(x, "bf16") for x in (Q, K, V)) + (to_dev(W), to_dev(b))
    Q2, K2, V2 = _qkv(B, H, L, "bf16", seed=73)
    a2 = tuple(to_dev(x, "bf16") for x in (Q2, K2, V2)) + (to_dev(W), to_dev(b))
    refb, refc = fv.attn_both(*a, S64)
    ref2 = fv.attn_causal(*a2, S64, chunk=32)
    refx = fv.attn_bidir(*a2, S64)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for s in (s1, s2):
        s.wait_stream(torch.cuda.current_stream())
    for _ in range(3):
        ob, oc = fv.attn_both(*a, S64, stream=s1)
        o2 = fv.attn_causal(*a2, S64, chunk=32, stream=s2)
        ox = fv.attn_bidir(*a2, S64, stream=s2)
        torch.cuda.synchronize()
        assert torch.equal(ob, refb) and torch.equal(oc, refc)
        assert torch.equal(o2, ref2) and torch.equal(ox, refx)
