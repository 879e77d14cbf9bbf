"""HIP graph capture of the library's calls. Every entry point launches kernels
only (no allocation, fill, copy or synchronisation on the stream), so a whole
step can be captured once and replayed: the ORF draw (Sec. 2.4), both
directions of FAVOR (Algorithm 1 and Eq. cumsum) with a carried state, and the
backward pass of both. Each replay is checked bitwise against eager calls on
the same inputs, with the program's own eager work, a synchronisation and new
input contents between the replays (a replay reads whatever its buffers hold).
"""
import numpy as np
import pytest

import workloads as wl
from helpers import to_dev

pytestmark = pytest.mark.gpu

S64 = 64 ** -0.25
SEED = 4242


def _fv():
    import paper_2006_03555_amd as fv
    return fv


def _data(B, H, L, M, k):
    """Seeded inputs of data set k (bf16 values), an upstream gradient per
    output, and a carried state and its gradient."""
    Q, K, V = wl.make_qkv(wl.Workload("t", "both", B, H, L, 64, M, "bf16", 700 + k))
    rng = np.random.default_rng(900 + k)
    d1, d2 = (rng.standard_normal((B, H, L, 64)).astype(np.float32) for _ in range(2))
    S0 = np.abs(rng.standard_normal((B, H, M, 65))).astype(np.float32) * 0.01
    dS = rng.standard_normal((B, H, M, 65)).astype(np.float32) * 0.01
    return ([to_dev(x, "bf16") for x in (Q, K, V, d1, d2)], to_dev(S0), to_dev(dS))


def _same_bits(a, b):
    """Bit-for-bit equality (NaNs included)."""
    import torch
    it = {torch.bfloat16: torch.int16, torch.float32: torch.int32}[a.dtype]
    return a.dtype == b.dtype and torch.equal(a.view(it), b.view(it))


def _capture(step):
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # one eager run on a side stream before capture
        step()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    return graph


@pytest.mark.parametrize("M", [256, 128])
def test_captured_training_step_replays_bitwise(M):
    """Draw, attn_both with row scales and a carried state, and
    attn_both_backward reading the saved outputs and the forward workspace, as
    one graph; M = 128 runs the 32-token causal chunks."""
    import torch
    fv = _fv()
    B, H, L = 2, 3, 1500
    (q, k, v, d1, d2), s0, ds = _data(B, H, L, M, 0)
    g = fv.make_desc(B, H, L, 64, M, fv.BF16, fv.BF16, S64)

    def buffers():
        f32 = dict(dtype=torch.float32, device="cuda")
        return dict(
            W=torch.empty((H, M, 64), **f32), b=torch.empty((H, M), **f32),
            ob=torch.empty_like(q), oc=torch.empty_like(q), so=torch.empty((B, H, M, 65), **f32),
            rb=torch.empty((B, H, L), **f32), rc=torch.empty((B, H, L), **f32),
            ws=torch.empty(fv.workspace_size(g, 2), dtype=torch.uint8, device="cuda"),
            wsb=torch.empty(fv.backward_workspace_size(g, 2), dtype=torch.uint8, device="cuda"),
            dQ=torch.empty_like(q), dK=torch.empty_like(q), dV=torch.empty_like(q),
            dS0=torch.empty((B, H, M, 65), **f32))

    def step(x):
        fv.orf_draw(SEED, H, M, 64, W=x["W"], b=x["b"])
        fv.attn_both(q, k, v, x["W"], x["b"], S64, state_in=s0, return_state=True,
                     out_bidir=x["ob"], out_causal=x["oc"], state_out=x["so"],
                     workspace=x["ws"], row_scale_bidir=x["rb"], row_scale_causal=x["rc"])
        fv.attn_both_backward(q, k, v, x["W"], x["b"], S64, d1, d2, state_in=s0,
                              dstate_out=ds, return_state_grad=True, dQ=x["dQ"], dK=x["dK"],
                              dV=x["dV"], dstate_in=x["dS0"], workspace=x["wsb"],
                              out_bidir=x["ob"], row_scale_bidir=x["rb"], out_causal=x["oc"],
                              row_scale_causal=x["rc"], forward_workspace=x["ws"],
                              forward_call="both")

    cap, ref = buffers(), buffers()
    graph = _capture(lambda: step(cap))
    for rep in range(3):
        (nq, nk, nv, n1, n2), ns0, nds = _data(B, H, L, M, rep + 1)
        for dst, src in ((q, nq), (k, nk), (v, nv), (d1, n1), (d2, n2), (s0, ns0), (ds, nds)):
            dst.copy_(src)
        for t in cap.values():   # no stale contents may reach a replay's results
            t.fill_(0)
        step(ref)                # eager, on the same inputs
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name in ("W", "b", "ob", "oc", "so", "rb", "rc", "dQ", "dK", "dV", "dS0"):
            assert _same_bits(cap[name], ref[name]), (rep, name)
        assert torch.isfinite(cap["dQ"].float()).all()


def test_captured_noalloc_step_matches_eager_attn_both():
    """favor_attn_both_noalloc (the library's static scratch) captured with the
    draw; every replay equals eager attn_both with a caller workspace."""
    import torch
    fv = _fv()
    B, H, L, M = 1, 4, 2100, 256
    (q, k, v, _, _), s0, _ = _data(B, H, L, M, 5)
    f32 = dict(dtype=torch.float32, device="cuda")
    W, b = torch.empty((H, M, 64), **f32), torch.empty((H, M), **f32)
    ob, oc = torch.empty_like(q), torch.empty_like(q)
    so = torch.empty((B, H, M, 65), **f32)

    def step():
        fv.orf_draw(SEED + 1, H, M, 64, W=W, b=b)
        fv.attn_both_noalloc(q, k, v, W, b, S64, state_in=s0, out_bidir=ob, out_causal=oc,
                             state_out=so)

    step()   # eagerly first: the library takes the scratch array's address at set-up
    graph = _capture(step)
    for rep in range(3):
        (nq, nk, nv, _, _), ns0, _ = _data(B, H, L, M, 10 + rep)
        for dst, src in ((q, nq), (k, nk), (v, nv), (s0, ns0)):
            dst.copy_(src)
        Wr, br = fv.orf_draw(SEED + 1, H, M, 64)
        rb, rc, rs = fv.attn_both(q, k, v, Wr, br, S64, state_in=s0, return_state=True)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert _same_bits(W, Wr) and _same_bits(b, br), rep
        assert _same_bits(ob, rb) and _same_bits(oc, rc) and _same_bits(so, rs), rep
