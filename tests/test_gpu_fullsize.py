"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark uses (library defaults: segment length, workgroup counts).

The whole output is computed on the GPU; the fp64 oracle recomputes sampled
(batch, head) pairs exactly, and properties that hold at any size are checked
on the whole output (finite values, equal token ids giving equal rows for the
protein-shaped workload, the last causal row equal to the bidirectional one).
"""
import numpy as np
import pytest

import workloads as wl
from helpers import parity, to_dev, to_host
from oracle import favor

pytestmark = pytest.mark.gpu


def _fv():
    import paper_2006_03555_amd as fv
    return fv


def _run(w, seed_w, heads, gpu_draw=False):
    import torch
    fv = _fv()
    Q, K, V = wl.make_qkv(w)
    dt = w.dtype
    dQ, dK, dV = (to_dev(x, dt) for x in (Q, K, V))
    if gpu_draw:
        Wd, bd = fv.orf_draw(seed_w, w.H, w.M)
        Wr, br = favor.orf_draw(seed_w, w.H, w.M, w.d)
    else:
        Wr, br = favor.orf_draw(seed_w, w.H, w.M, w.d)
        Wr, br = Wr.astype(np.float32), br.astype(np.float32)
        Wd, bd = to_dev(Wr), to_dev(br)
    out = {}
    if w.direction == "both":      # one key pass for both directions, as the benchmark runs it
        out["bidir"], out["causal"] = fv.attn_both(dQ, dK, dV, Wd, bd, w.input_scale)
    elif w.direction == "bidir":
        out["bidir"] = fv.attn_bidir(dQ, dK, dV, Wd, bd, w.input_scale)
    else:
        out["causal"] = fv.attn_causal(dQ, dK, dV, Wd, bd, w.input_scale)
    torch.cuda.synchronize()
    out = {k: to_host(v) for k, v in out.items()}
    for k, v in out.items():
        assert np.all(np.isfinite(v)), k
        parity(v, Q, K, V, Wr, br, w.input_scale, k == "causal", dt, heads=heads)
    return Q, out


def test_bidir_b8h8_full():
    w = wl.WORKLOADS["bidir_b8h8"]
    _run(w, 2, heads=[(0, 0), (7, 5)])


def test_causal_b8h8_full():
    w = wl.WORKLOADS["causal_b8h8"]
    _run(w, 3, heads=[(0, 3), (6, 7)])


def test_protein_b4h8_full_both_directions():
    w = wl.WORKLOADS["protein_b4h8"]
    Q, out = _run(w, 4, heads=[(1, 2)], gpu_draw=True)
    ids = wl.protein_ids(w)
    # bidirectional rows depend only on the query row: equal token ids (so equal
    # Q rows within a head) give bitwise equal outputs
    bi = out["bidir"]
    for b in range(w.B):
        first = {}
        for l, tok in enumerate(ids[b]):
            first.setdefault(int(tok), l)
        for h in range(w.H):
            ref_rows = {tok: bi[b, h, l] for tok, l in first.items()}
            for l in range(0, w.L, 97):
                assert np.array_equal(bi[b, h, l], ref_rows[int(ids[b, l])])
    # the causal output's last row attends to every key, like the bidirectional one
    ca = out["causal"]
    np.testing.assert_allclose(ca[:, :, -1, :], bi[:, :, -1, :], rtol=0, atol=2e-2 * np.max(np.abs(bi)))


def test_causal_long_full_with_gpu_draw():
    w = wl.WORKLOADS["causal_long"]
    _run(w, 5, heads=[(0, 11)], gpu_draw=True)


def test_protein_b4h8_full_backward():
    """Both backward passes at the protein workload's full size (B4 H8 L8192 M256
    bf16), and the backward of both directions in one call (the same upstream
    gradient for each output), sampled heads against the oracle's gradients; the
    gate of test_gpu_backward (per row, in units of the oracle's error scale;
    for the sum of the two directions, the sum of their scales)."""
    import torch
    fv = _fv()
    from test_gpu_backward import _check_all, _host_grads, _oracle_grads
    w = wl.WORKLOADS["protein_b4h8"]
    Q, K, V = wl.make_qkv(w)
    dout = np.random.default_rng(123).standard_normal(Q.shape).astype(np.float32)
    dout = torch.from_numpy(dout).to(torch.bfloat16).float().numpy()
    Wr, br = favor.orf_draw(8, w.H, w.M, w.d)
    Wr, br = Wr.astype(np.float32), br.astype(np.float32)
    args = [to_dev(x, "bf16") for x in (Q, K, V)] + [to_dev(Wr), to_dev(br), w.input_scale,
                                                      to_dev(dout, "bf16")]
    gb = fv.attn_bidir_backward(*args)
    gc = fv.attn_causal_backward(*args)
    gx = fv.attn_both_backward(*args, args[-1])
    torch.cuda.synchronize()
    gb = [to_host(t) for t in gb]
    gc = [to_host(t) for t in gc]
    gx = [to_host(t) for t in gx]
    for t in gb + gc + gx:
        assert np.all(np.isfinite(t))
    for (bi, hi) in [(0, 0), (3, 6)]:
        sl = lambda a: a[bi:bi + 1, hi:hi + 1]
        Wh, bh = Wr[hi:hi + 1], br[hi:hi + 1]
        refs = []
        for causal, got in ((False, gb), (True, gc)):
            ref, scale, _ = _oracle_grads(sl(Q), sl(K), sl(V), Wh, bh, sl(dout), causal)
            _check_all(_host_grads([sl(g) for g in got]), ref, "bf16", scale)
            refs.append((ref, scale))
        (rb, sb), (rc, sc) = refs
        _check_all(_host_grads([sl(g) for g in gx]), {n: rb[n] + rc[n] for n in rb}, "bf16",
                   {n: sb[n] + sc[n] for n in sb})
