"""GPU parity of favor_attn_both_backward: the gradients of a loss of both
outputs of favor_attn_both (Algorithm 1 and Eq. cumsum in reverse), against the
fp64 oracle's bidirectional plus causal gradients on the same seeded inputs.

The gradient of a sum is the sum of the gradients, so the reference is the
oracle's bidirectional gradient plus its causal one, and the per-row gate of the
backward tests uses the sum of the two error scales (the error of a sum is at
most the sum of the errors); 1e-4 for fp32 inputs, 2e-2 for bf16 inputs. The
causal state gradient is the causal direction's alone: the bidirectional output
does not depend on state_in. Reading the forward call's workspace gives bitwise
the gradients of recomputing what it holds.
"""
import numpy as np
import pytest

from helpers import TOL, to_dev, to_host
from oracle import favor
from test_gpu_backward import S64, RELU, SOFTMAX, _check_all, _host_grads, _inputs, \
    _oracle_grads, _oracle_w

pytestmark = pytest.mark.gpu


def _fv():
    import paper_2006_03555_amd as fv
    return fv


def _douts(Q, dtype, seed):
    d2 = np.random.default_rng(seed).standard_normal(Q.shape).astype(np.float32)
    if dtype == "bf16":
        import torch
        d2 = torch.from_numpy(d2).to(torch.bfloat16).float().numpy()
    return d2


CASES = [
    # B, H, L, M, dtype, kernel, renormalize, denom_eps, with states
    (1, 2, 300, 64, "f32", SOFTMAX, True, 0.0, False),
    (2, 2, 1000, 256, "bf16", SOFTMAX, True, 0.0, False),
    (1, 3, 65, 128, "bf16", SOFTMAX, True, 0.0, True),
    (1, 1, 1, 64, "f32", SOFTMAX, True, 0.0, False),
    (1, 2, 300, 128, "bf16", SOFTMAX, True, 0.5, False),
    (1, 1, 190, 64, "f32", SOFTMAX, False, 0.0, True),
    (1, 2, 257, 64, "f32", RELU, True, 0.0, True),
    (1, 2, 777, 256, "bf16", RELU, True, 0.0, False),
    (1, 2, 1500, 128, "bf16", SOFTMAX, True, 0.0, True),
]


@pytest.mark.parametrize("B,H,L,M,dtype,kernel,renorm,eps,states", CASES)
def test_both_backward_parity(B, H, L, M, dtype, kernel, renorm, eps, states):
    import torch
    fv = _fv()
    Q, K, V, dout_b, W, b = _inputs(B, H, L, M, dtype, seed=81 + L + M)
    dout_c = _douts(Q, dtype, seed=83 + L)
    kw = dict(kernel=kernel, renormalize=renorm)
    S0 = dS = None
    if states:
        Qe, Ke, Ve, _, _, _ = _inputs(B, H, 200, M, dtype, seed=5)
        _, S0 = favor.attn_causal(Qe, Ke, Ve, W, b, S64, **kw, kernel_eps=1e-3)
        S0 = S0.astype(np.float32)
        dS = np.random.default_rng(9).standard_normal(S0.shape).astype(np.float32) * 0.01
    dev = lambda x: None if x is None else to_dev(x)
    dQ, dK, dV, dS0 = fv.attn_both_backward(
        to_dev(Q, dtype), to_dev(K, dtype), to_dev(V, dtype), to_dev(W), to_dev(b), S64,
        to_dev(dout_b, dtype), to_dev(dout_c, dtype), denom_eps=eps, state_in=dev(S0),
        dstate_out=dev(dS), return_state_grad=True, **kw)
    torch.cuda.synchronize()
    Wo = _oracle_w(W, M, dtype, kernel)
    rb, sb, _ = _oracle_grads(Q, K, V, Wo, b, dout_b, False, denom_eps=eps, **kw)
    rc, sc, rS = _oracle_grads(Q, K, V, Wo, b, dout_c, True, denom_eps=eps, state_in=S0,
                               dstate_out=dS, **kw)
    ref = {n: rb[n] + rc[n] for n in rb}
    scale = {n: sb[n] + sc[n] for n in sb}
    _check_all(_host_grads((dQ, dK, dV)), ref, dtype, scale)
    got = to_host(dS0)
    assert np.max(np.abs(got - rS)) <= TOL[dtype] * np.max(np.abs(rS))


@pytest.mark.parametrize("dtype,M,chunk", [("bf16", 256, 0), ("bf16", 256, 32), ("bf16", 128, 0),
                                           ("bf16", 64, 0), ("f32", 64, 0)])
def test_both_backward_reads_saved_forward_quantities(dtype, M, chunk):
    """Given the workspace of the attn_both call (W'', b'', Buf1 and the segment
    prefixes; 32-token chunks at M <= 128 in bf16, and when asked for at
    M = 256, the segment plan of two workgroups per CU), the gradients are
    bitwise those of recomputing them; given also
    its outputs and row scales, within the gate of recomputing them. The causal
    state gradient is bitwise that of attn_causal_backward."""
    import torch
    fv = _fv()
    B, H, L = 1, 2, 700
    Q, K, V, dout_b, W, b = _inputs(B, H, L, M, dtype, seed=91)
    dout_c = _douts(Q, dtype, seed=92)
    q, k, v, db, dc = (to_dev(x, dtype) for x in (Q, K, V, dout_b, dout_c))
    Wd, bd = to_dev(W), to_dev(b)
    dS = torch.randn((B, H, M, 65), device="cuda") * 0.01
    g = fv.make_desc(B, H, L, 64, M, fv.BF16 if dtype == "bf16" else fv.F32,
                     fv.BF16 if dtype == "bf16" else fv.F32, S64, chunk=chunk)
    ws = torch.empty(fv.workspace_size(g, 2), dtype=torch.uint8, device="cuda")
    rb = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
    rc = torch.empty_like(rb)
    ob, oc = fv.attn_both(q, k, v, Wd, bd, S64, workspace=ws, row_scale_bidir=rb,
                          row_scale_causal=rc, chunk=chunk)
    kw = dict(dstate_out=dS, return_state_grad=True, chunk=chunk)
    fresh = fv.attn_both_backward(q, k, v, Wd, bd, S64, db, dc, **kw)
    reuse = fv.attn_both_backward(q, k, v, Wd, bd, S64, db, dc, forward_workspace=ws,
                                  forward_call="both", **kw)
    saved = fv.attn_both_backward(q, k, v, Wd, bd, S64, db, dc, out_bidir=ob,
                                  row_scale_bidir=rb, out_causal=oc, row_scale_causal=rc,
                                  forward_workspace=ws, forward_call="both", **kw)
    causal = fv.attn_causal_backward(q, k, v, Wd, bd, S64, dc, **kw)
    torch.cuda.synchronize()
    for a, c in zip(reuse, fresh):
        assert torch.equal(a, c)
    assert torch.equal(fresh[3], causal[3])
    assert torch.equal(saved[3], causal[3])
    _, sb, _ = _oracle_grads(Q, K, V, W, b, dout_b, False)
    _, sc, _ = _oracle_grads(Q, K, V, W, b, dout_c, True)
    _check_all(_host_grads(saved), _host_grads(fresh), dtype,
               {n: sb[n] + sc[n] for n in sb})


def test_both_backward_empty_sequence_passes_state_gradient():
    import torch
    fv = _fv()
    Q = torch.zeros((1, 2, 0, 64), dtype=torch.bfloat16, device="cuda")
    W, b = _inputs(1, 2, 1, 128, "bf16", 3)[4:]
    dS = torch.randn((1, 2, 128, 65), device="cuda")
    _, _, _, dS0 = fv.attn_both_backward(Q, Q, Q, to_dev(W), to_dev(b), S64, Q, Q,
                                         dstate_out=dS, return_state_grad=True)
    torch.cuda.synchronize()
    assert torch.equal(dS0, dS)
