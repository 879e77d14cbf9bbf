"""The causal scan with 32-token chunks (favor_desc.chunk = 32, bf16 inputs)
against the fp64 oracle.

The chunk length only changes how the scan groups the tokens of a segment
(Eq. cumsum is the same sum, taken 32 instead of 64 tokens per step), so the
outputs meet the bounds the 64-token scan meets: 2e-2 (E_row and E_cond) for
bf16 inputs. The final state is formed from the segment aggregates, not by the
scan, so with equal segments it is bitwise the state of the 64-token scan.
Cases: every M class the kernels take (64, 128, 256 rows, with padding),
lengths around the chunk and segment boundaries, both feature kinds,
renormalisation off, the stabiliser, a carried state, fp32 outputs, saved row
scales, both directions in one call, the no-allocation entry point, and
full-size workloads on sampled heads (M = 256, and M = 128 where 32-token
chunks are the default).
"""
import numpy as np
import pytest

import workloads as wl
from helpers import TOL, parity, to_dev, to_host
from oracle import favor

pytestmark = pytest.mark.gpu

S64 = 64 ** -0.25
SOFTMAX, RELU = favor.KERNEL_SOFTMAX, favor.KERNEL_RELU


def _fv():
    import paper_2006_03555_amd as fv
    return fv


def _features(seed, H, M):
    W, b = favor.orf_draw(seed, H, M, 64, favor.RF_ORTHO_CHI)
    return W.astype(np.float32), b.astype(np.float32)


def _qkv(B, H, L, seed):
    return wl.make_qkv(wl.Workload("t", "causal", B, H, L, 64, 64, "bf16", seed))


CASES = [
    # B, H, L, M, segment rows, kernel, renormalize, eps, carried state, out dtype
    (1, 1, 1, 256, 0, SOFTMAX, True, 0.0, False, "bf16"),
    (1, 2, 31, 256, 0, SOFTMAX, True, 0.0, False, "bf16"),
    (1, 2, 32, 128, 0, SOFTMAX, True, 0.0, False, "bf16"),
    (2, 1, 33, 64, 0, SOFTMAX, True, 0.0, False, "bf16"),
    (2, 2, 1000, 256, 0, SOFTMAX, True, 0.0, False, "bf16"),
    (1, 2, 1000, 256, 64, SOFTMAX, True, 0.0, True, "bf16"),    # two chunks per segment
    (1, 3, 777, 128, 128, SOFTMAX, True, 0.5, False, "bf16"),
    (2, 2, 300, 48, 0, SOFTMAX, True, 0.0, True, "bf16"),       # 48 features in 64 rows
    (1, 2, 517, 208, 0, SOFTMAX, True, 0.0, False, "f32"),      # 208 features in 256 rows
    (1, 2, 650, 256, 192, RELU, True, 0.0, True, "bf16"),
    (1, 1, 400, 16, 0, RELU, True, 0.0, False, "bf16"),
    (2, 1, 300, 256, 0, SOFTMAX, False, 0.0, False, "f32"),
    (1, 2, 300, 128, 64, RELU, False, 0.0, True, "bf16"),
]


@pytest.mark.parametrize("B,H,L,M,segment,kernel,renorm,eps,state,odt", CASES)
def test_chunk32_causal_parity(B, H, L, M, segment, kernel, renorm, eps, state, odt):
    import torch
    fv = _fv()
    Q, K, V = _qkv(B, H, L, seed=300 + L + M)
    W, b = _features(301 + L, H, M)
    kw = dict(kernel=kernel, renormalize=renorm)
    S0 = None
    if state:
        Qe, Ke, Ve = _qkv(B, H, 90, seed=7)
        _, S0 = favor.attn_causal(Qe, Ke, Ve, W, b, S64, **kw)
        S0 = S0.astype(np.float32)
    q, k, v = (to_dev(x, "bf16") for x in (Q, K, V))
    out_dtype = torch.float32 if odt == "f32" else torch.bfloat16
    args = (q, k, v, to_dev(W), to_dev(b), S64)
    common = dict(denom_eps=eps, segment=segment, out_dtype=out_dtype, return_state=True,
                  state_in=None if S0 is None else to_dev(S0), **kw)
    o32, s32 = fv.attn_causal(*args, chunk=32, **common)
    o64, s64 = fv.attn_causal(*args, chunk=64, **common)
    torch.cuda.synchronize()
    print(f"\nB{B} H{H} L{L} M{M} segment {segment} kernel {kernel} renorm {renorm} eps {eps}",
          flush=True)
    # cos features below 64 rows can nearly cancel a row's D-hat: E_cond alone there
    gate = "cond" if kernel == SOFTMAX and M < 64 else "both"
    e = parity(to_host(o32), Q, K, V, W, b, S64, True, "bf16", eps=eps, state_in=S0,
               kernel=kernel, renormalize=renorm, gate=gate)
    print(f"chunk 32: E_row {e[0]:.2e} E_cond {e[1]:.2e}", flush=True)
    e = parity(to_host(o64), Q, K, V, W, b, S64, True, "bf16", eps=eps, state_in=S0,
               kernel=kernel, renormalize=renorm, gate=gate)
    print(f"chunk 64: E_row {e[0]:.2e} E_cond {e[1]:.2e}", flush=True)
    assert torch.equal(s32, s64)
    if gate == "both":
        a, c = to_host(o32), to_host(o64)
        assert np.max(np.abs(a - c)) <= 2 * TOL["bf16"] * np.max(np.abs(c))


def test_chunk32_both_directions_and_row_scales():
    """attn_both with 32-token chunks: the bidirectional half is the one of the
    64-token call (the scan length does not enter it), the causal half is the
    one attn_causal gives with the same chunks, and the saved row scales equal
    the oracle's 1 / D-hat in units of the unscaled features."""
    import torch
    fv = _fv()
    from test_gpu_backward import _expected_row_scale
    B, H, L, M = 2, 2, 1000, 256
    Q, K, V = _qkv(B, H, L, seed=411)
    W, b = _features(412, H, M)
    args = tuple(to_dev(x, "bf16") for x in (Q, K, V)) + (to_dev(W), to_dev(b), S64)
    rb = torch.full((B, H, L), float("nan"), device="cuda")
    rc = torch.full((B, H, L), float("nan"), device="cuda")
    ob, oc = fv.attn_both(*args, chunk=32, row_scale_bidir=rb, row_scale_causal=rc)
    ob64, _ = fv.attn_both(*args, chunk=64)
    oc1 = fv.attn_causal(*args, chunk=32)
    torch.cuda.synchronize()
    assert torch.equal(ob, ob64)
    assert torch.equal(oc, oc1)
    parity(to_host(oc), Q, K, V, W, b, S64, True, "bf16")
    want = _expected_row_scale(Q, K, W, b, M, SOFTMAX, 0.0, True)
    got = to_host(rc).astype(np.float64)
    assert np.all(np.isfinite(got))
    assert np.max(np.abs(got - want) / np.abs(want)) <= TOL["bf16"]


def test_chunk32_no_alloc_entry_point():
    import torch
    fv = _fv()
    B, H, L, M = 1, 4, 1500, 256
    Q, K, V = _qkv(B, H, L, seed=421)
    W, b = _features(422, H, M)
    args = tuple(to_dev(x, "bf16") for x in (Q, K, V)) + (to_dev(W), to_dev(b), S64)
    ob, oc = fv.attn_both(*args, chunk=32)
    nb, nc = fv.attn_both_noalloc(*args, chunk=32)
    torch.cuda.synchronize()
    assert torch.equal(ob, nb) and torch.equal(oc, nc)


def test_chunk32_full_size_causal_b8h8():
    """The configuration the chunk sweep is measured on (B8 H8 L8192 M256), with
    the library's segments, checked on two heads."""
    import torch
    fv = _fv()
    w = wl.WORKLOADS["causal_b8h8"]
    Q, K, V = wl.make_qkv(w)
    W, b = _features(431, w.H, w.M)
    out = fv.attn_causal(*(to_dev(x, "bf16") for x in (Q, K, V)), to_dev(W), to_dev(b),
                         w.input_scale, chunk=32)
    torch.cuda.synchronize()
    heads = [(0, 3), (7, 6)]
    e = parity(to_host(out), Q, K, V, W, b, w.input_scale, True, "bf16", heads=heads)
    print(f"\ncausal_b8h8, chunk 32, heads {heads}: E_row {e[0]:.2e} E_cond {e[1]:.2e}",
          flush=True)


def test_default_chunk_full_size_m128():
    """B8 H8 L8192 at M = 128, where chunk = 0 scans 32-token chunks at two
    workgroups per CU (512 segments of 1024 tokens), checked on two heads; the
    explicit 64-token call meets the same bound."""
    import torch
    fv = _fv()
    w = wl.WORKLOADS["causal_b8h8"]
    Q, K, V = wl.make_qkv(w)
    W, b = _features(451, w.H, 128)
    args = tuple(to_dev(x, "bf16") for x in (Q, K, V)) + (to_dev(W), to_dev(b), w.input_scale)
    out = fv.attn_causal(*args)
    o64 = fv.attn_causal(*args, chunk=64)
    torch.cuda.synchronize()
    heads = [(1, 2), (6, 7)]
    for name, o in (("default (32)", out), ("64", o64)):
        e = parity(to_host(o), Q, K, V, W, b, w.input_scale, True, "bf16", heads=heads)
        print(f"\nM 128, chunk {name}, heads {heads}: E_row {e[0]:.2e} E_cond {e[1]:.2e}",
              flush=True)


def test_chunk32_backward_recomputes_with_its_chunks():
    """The causal backward call without saved statistics recomputes the forward
    outputs and row scales with the descriptor's chunks: its gradients are those
    of the 64-token call within the gradient gate of the backward tests, and,
    given the outputs and row scales a 32-token forward call saved, the same
    bits as recomputing them."""
    import torch
    fv = _fv()
    from test_gpu_backward import _check_all, _host_grads, _oracle_grads
    B, H, L, M = 1, 2, 700, 128
    Q, K, V = _qkv(B, H, L, seed=441)
    dout = np.random.default_rng(442).standard_normal(Q.shape).astype(np.float32)
    W, b = _features(443, H, M)
    q, k, v, do = (to_dev(x, "bf16") for x in (Q, K, V, dout))
    Wd, bd = to_dev(W), to_dev(b)
    g32 = fv.attn_causal_backward(q, k, v, Wd, bd, S64, do, chunk=32)[:3]
    rs = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
    o32 = fv.attn_causal(q, k, v, Wd, bd, S64, chunk=32, row_scale=rs)
    s32 = fv.attn_causal_backward(q, k, v, Wd, bd, S64, do, out=o32, row_scale=rs)[:3]
    torch.cuda.synchronize()
    for a, c in zip(g32, s32):
        assert torch.equal(a, c)
    Qb, Kb, Vb, dob = (np.asarray(to_host(x), dtype=np.float64) for x in (q, k, v, do))
    ref, scale, _ = _oracle_grads(Qb, Kb, Vb, W, b, dob, True)
    _check_all(_host_grads(g32), ref, "bf16", scale)
