"""favor_attn_both_noalloc (the entry point for callers that cannot allocate
device memory) against favor_attn_both on the same inputs: two calls in a row,
the second smaller, each bit-identical to favor_attn_both (same kernels, same
plan) and within the parity tolerance of the oracle; the static scratch is
reused across the calls without clearing. (The rejection of a workspace beyond
the scratch is host logic, tested in test_abi.)"""
import numpy as np
import pytest

import workloads as wl
from helpers import parity, to_dev, to_host
from oracle import favor

pytestmark = pytest.mark.gpu

S64 = 64 ** -0.25


def _case(B, H, L, M, seed):
    Q, K, V = wl.make_qkv(wl.Workload("t", "both", B, H, L, 64, M, "bf16", seed))
    W, b = favor.orf_draw(seed + 1, H, M, 64)
    return Q, K, V, W.astype(np.float32), b.astype(np.float32)


def test_noalloc_matches_attn_both_on_two_calls():
    import torch
    import paper_2006_03555_amd as fv
    torch.cuda.set_device(0)
    for (B, H, L, M, seed) in ((2, 4, 3000, 256, 5), (1, 2, 500, 128, 6)):
        print(f"\nnoalloc case B{B} H{H} L{L} M{M}", flush=True)
        Q, K, V, W, b = _case(B, H, L, M, seed)
        q, k, v = (to_dev(x, "bf16") for x in (Q, K, V))
        Wd, bd = to_dev(W), to_dev(b)
        g = fv.make_desc(B, H, L, 64, M, fv.BF16, fv.BF16, S64)
        assert 0 < fv.workspace_size(g, 2) <= fv.noalloc_scratch_bytes()
        ob = torch.empty_like(q)
        oc = torch.empty_like(q)
        st = torch.empty((B, H, M, 65), dtype=torch.float32, device="cuda")
        rb = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
        rc = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        before = torch.cuda.memory_allocated()
        fv.attn_both_noalloc(q, k, v, Wd, bd, S64, out_bidir=ob, out_causal=oc, state_out=st,
                             row_scale_bidir=rb, row_scale_causal=rc)
        torch.cuda.synchronize()
        assert torch.cuda.memory_allocated() == before
        eb, ec, est = fv.attn_both(q, k, v, Wd, bd, S64, return_state=True)
        erb = torch.empty_like(rb)
        erc = torch.empty_like(rc)
        fv.attn_both(q, k, v, Wd, bd, S64, row_scale_bidir=erb, row_scale_causal=erc)
        torch.cuda.synchronize()
        assert torch.equal(ob, eb) and torch.equal(oc, ec) and torch.equal(st, est)
        assert torch.equal(rb, erb) and torch.equal(rc, erc)
        parity(to_host(ob), Q, K, V, W, b, S64, False, "bf16")
        parity(to_host(oc), Q, K, V, W, b, S64, True, "bf16")

