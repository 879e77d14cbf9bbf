"""The largest number of heads the calls take (B * H = 65535, the grid's second
dimension), against the fp64 oracle on sampled heads: the random-feature draw
for every head, the materialised feature map, both attention directions in one
call and the causal backward, over a ragged length; and the shortest sequence
(L = 1) at the same head count.

The inputs (Q, K ~ N(0, 1) d^-1/4, V ~ N(0, 1), rounded to bf16) are drawn on
the device by a seeded generator; the oracle takes the sampled heads' values
back from the device, so both sides see the same inputs. Tolerances as
everywhere: 2e-2 (E_row and E_cond) for bf16 inputs; the draw within 1e-4 of
the oracle relative to the row norm; gradients by the per-row gate of the
backward tests.
"""
import numpy as np
import pytest

from helpers import TOL, parity, to_host
from oracle import favor

pytestmark = pytest.mark.gpu

S64 = 64 ** -0.25
B, H = 5, 13107          # B * H = 65535
M = 64
HEADS = [(0, 0), (2, 6553), (4, 13106)]   # (batch, head) pairs checked


def _fv():
    import paper_2006_03555_amd as fv
    return fv


def _inputs(L, seed, n=3):
    import torch
    gen = torch.Generator(device="cuda").manual_seed(seed)
    shape = (B, H, L, 64)
    out = []
    for i in range(n):
        x = torch.randn(shape, generator=gen, device="cuda")
        out.append((x * S64 if i < 2 else x).to(torch.bfloat16).contiguous())
    return out


def _heads(t):
    """The sampled heads of a [B, H, ...] device tensor, [len(HEADS), 1, ...] fp64."""
    import torch
    return np.asarray(to_host(torch.stack([t[b, h] for b, h in HEADS])), np.float64)[:, None]


def _features_of_heads(Wd, bd):
    return (np.stack([to_host(Wd[h]) for _, h in HEADS])[:, None],
            np.stack([to_host(bd[h]) for _, h in HEADS])[:, None])


@pytest.mark.parametrize("L", [70, 1])
def test_most_heads(L):
    import torch
    fv = _fv()
    print(f"\nB{B} H{H} (B*H = {B * H}) L{L} M{M}", flush=True)
    q, k, v = _inputs(L, 551 + L)
    seed = 552
    Wd, bd = fv.orf_draw(seed, H, M, 64)
    Xp = fv.feature_map(q, Wd, bd, S64)
    ob, oc = fv.attn_both(q, k, v, Wd, bd, S64)
    torch.cuda.synchronize()
    # the draw of the sampled heads (each head is drawn from its own streams)
    hs = sorted({h for _, h in HEADS})
    Wo, bo = favor.orf_draw(seed, H, M, 64, heads=hs)
    for i, h in enumerate(hs):
        rho = np.linalg.norm(Wo[i], axis=-1, keepdims=True)
        assert np.max(np.abs(to_host(Wd[h]) - Wo[i]) / rho) <= 1e-4, h
        assert np.max(np.abs(to_host(bd[h]) - bo[i])) <= 1e-5, h
    Ws, bs = _features_of_heads(Wd, bd)
    Qs, Ks, Vs = _heads(q), _heads(k), _heads(v)
    ref_f = favor.features(Qs, Ws, bs, S64, favor.KERNEL_SOFTMAX, 1e-3)
    scale = np.max(np.abs(ref_f), axis=-1, keepdims=True)
    assert np.max(np.abs(_heads(Xp) - ref_f) / np.maximum(scale, 1e-30)) <= TOL["bf16"]
    eb = parity(_heads(ob), Qs, Ks, Vs, Ws, bs, S64, False, "bf16")
    ec = parity(_heads(oc), Qs, Ks, Vs, Ws, bs, S64, True, "bf16")
    print(f"bidir E_row {eb[0]:.2e}, causal E_row {ec[0]:.2e}", flush=True)


def test_most_heads_causal_backward():
    import torch
    fv = _fv()
    from test_gpu_backward import _check_all, _oracle_grads
    L = 70
    q, k, v, do = _inputs(L, 561, n=4)
    Wd, bd = fv.orf_draw(563, H, M, 64)
    grads = fv.attn_causal_backward(q, k, v, Wd, bd, S64, do)[:3]
    torch.cuda.synchronize()
    Ws, bs = _features_of_heads(Wd, bd)
    ref, scale, _ = _oracle_grads(_heads(q), _heads(k), _heads(v), Ws, bs, _heads(do), True)
    _check_all({n: _heads(g) for n, g in zip(("dQ", "dK", "dV"), grads)}, ref, "bf16", scale)
