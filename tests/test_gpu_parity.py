"""GPU parity: the HIP path (called through the C ABI) against the fp64 oracle
on the same seeded inputs and the same random features.

Tolerances (E_row and E_cond, see oracle.metrics): 1e-4 for fp32 inputs,
2e-2 for bf16 inputs with fp32 accumulation.
"""
import numpy as np
import pytest

import workloads as wl
from helpers import TOL, parity, to_dev, to_host
from oracle import favor

pytestmark = pytest.mark.gpu

S64 = 64 ** -0.25


def _fv():
    import paper_2006_03555_amd as fv
    return fv


def _features(seed, H, M, kind=favor.RF_ORTHO_CHI):
    W, b = favor.orf_draw(seed, H, M, 64, kind)
    return W.astype(np.float32), b.astype(np.float32)


def _qkv(B, H, L, dtype, seed):
    w = wl.Workload("t", "bidir", B, H, L, 64, 64, dtype, seed)
    return wl.make_qkv(w)


# ---------------------------------------------------------------- ORF draw
@pytest.mark.parametrize("kind", [favor.RF_ORTHO_CHI, favor.RF_ORTHO_FIXED, favor.RF_IID,
                                  favor.RF_HADAMARD, favor.RF_GIVENS])
@pytest.mark.parametrize("M,H", [(256, 8), (128, 1), (64, 3), (100, 2)])
def test_orf_draw_matches_oracle(kind, M, H):
    import torch
    fv = _fv()
    seed = 1234 + M + kind
    W, b = fv.orf_draw(seed, H, M, 64, kind)
    torch.cuda.synchronize()
    Wr, br = favor.orf_draw(seed, H, M, 64, kind)
    Wg, bg = to_host(W), to_host(b)
    rho = np.linalg.norm(Wr, axis=-1, keepdims=True)
    assert np.max(np.abs(Wg - Wr) / rho) <= 1e-4
    assert np.max(np.abs(bg - br)) <= 4e-6 * 2 * np.pi
    if kind != favor.RF_IID:
        for h in range(H):
            for k in range(-(-M // 64)):
                blk = Wg[h, 64 * k:64 * (k + 1)]
                G = blk @ blk.T
                nr = np.sqrt(np.diag(G))
                off = (G - np.diag(np.diag(G))) / np.outer(nr, nr)
                assert np.max(np.abs(off)) <= 1e-5


def test_orf_draw_zero_heads_is_noop():
    fv = _fv()
    W, b = fv.orf_draw(1, 0, 256, 64)
    assert W.numel() == 0


# ---------------------------------------------------------------- feature map
@pytest.mark.parametrize("din,dout", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")])
@pytest.mark.parametrize("M,L", [(256, 300), (128, 64), (64, 1)])
def test_feature_map_parity(din, dout, M, L):
    import torch
    fv = _fv()
    Q, _, _ = _qkv(2, 3, L, din, seed=L + M)
    W, b = _features(7, 3, M)
    Xp = fv.feature_map(to_dev(Q, din), to_dev(W), to_dev(b), S64,
                        out_dtype=torch.bfloat16 if dout == "bf16" else torch.float32)
    torch.cuda.synchronize()
    ref = favor.feature_map(Q.astype(np.float64), W.astype(np.float64), b.astype(np.float64), S64)
    got = to_host(Xp)
    scale = np.max(np.abs(ref), axis=-1, keepdims=True)
    err = np.max(np.abs(got - ref) / scale)
    tol = TOL["f32"] if din == "f32" and dout == "f32" else TOL["bf16"]
    assert err <= tol, err


# ---------------------------------------------------------------- bidirectional
BIDIR_CASES = [
    # B, H, L, M, dtype
    (1, 1, 1024, 128, "f32"),       # the small fp32 workload at full size
    (2, 2, 1000, 256, "bf16"),      # ragged, several tiles and splits
    (1, 3, 65, 64, "bf16"),
    (1, 2, 1, 128, "f32"),
    (2, 1, 63, 256, "f32"),
    (1, 1, 4096, 256, "bf16"),
]


@pytest.mark.parametrize("B,H,L,M,dtype", BIDIR_CASES)
def test_bidir_parity(B, H, L, M, dtype):
    import torch
    fv = _fv()
    Q, K, V = _qkv(B, H, L, dtype, seed=11 + L)
    W, b = _features(3 + L, H, M)
    out = fv.attn_bidir(to_dev(Q, dtype), to_dev(K, dtype), to_dev(V, dtype), to_dev(W),
                        to_dev(b), S64)
    torch.cuda.synchronize()
    parity(to_host(out), Q, K, V, W, b, S64, False, dtype)


def test_bidir_fp32_output_from_bf16_inputs():
    import torch
    fv = _fv()
    Q, K, V = _qkv(1, 2, 777, "bf16", seed=5)
    W, b = _features(5, 2, 256)
    out = fv.attn_bidir(to_dev(Q, "bf16"), to_dev(K, "bf16"), to_dev(V, "bf16"), to_dev(W),
                        to_dev(b), S64, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert out.dtype == torch.float32
    parity(to_host(out), Q, K, V, W, b, S64, False, "bf16")


def test_bidir_denominator_stabiliser():
    import torch
    fv = _fv()
    Q, K, V = _qkv(1, 2, 300, "f32", seed=6)
    W, b = _features(6, 2, 128)
    out = fv.attn_bidir(to_dev(Q), to_dev(K), to_dev(V), to_dev(W), to_dev(b), S64,
                        denom_eps=0.5)
    torch.cuda.synchronize()
    parity(to_host(out), Q, K, V, W, b, S64, False, "f32", eps=0.5)


# ---------------------------------------------------------------- causal
CAUSAL_CASES = [
    # B, H, L, M, dtype, causal segment rows
    (1, 1, 1024, 128, "f32", 0),
    (2, 2, 1000, 256, "bf16", 0),
    (1, 2, 1000, 256, "bf16", 64),     # one 64-token chunk per segment: most hand-offs
    (1, 3, 65, 64, "bf16", 0),
    (1, 1, 1, 128, "f32", 0),
    (2, 1, 200, 64, "f32", 128),
    (1, 1, 4096, 256, "bf16", 0),
    (1, 2, 777, 128, "bf16", 0),
    (2, 1, 300, 128, "bf16", 128),
]


@pytest.mark.parametrize("B,H,L,M,dtype,segment", CAUSAL_CASES)
def test_causal_parity(B, H, L, M, dtype, segment):
    import torch
    fv = _fv()
    Q, K, V = _qkv(B, H, L, dtype, seed=21 + L)
    W, b = _features(9 + L, H, M)
    out = fv.attn_causal(to_dev(Q, dtype), to_dev(K, dtype), to_dev(V, dtype), to_dev(W),
                         to_dev(b), S64, segment=segment)
    torch.cuda.synchronize()
    parity(to_host(out), Q, K, V, W, b, S64, True, dtype)


@pytest.mark.parametrize("M", [256, 64])
def test_causal_denominator_stabiliser_bf16(M):
    import torch
    fv = _fv()
    Q, K, V = _qkv(1, 2, 300, "bf16", seed=7)
    W, b = _features(7, 2, M)
    out = fv.attn_causal(to_dev(Q, "bf16"), to_dev(K, "bf16"), to_dev(V, "bf16"), to_dev(W),
                         to_dev(b), S64, denom_eps=0.5)
    torch.cuda.synchronize()
    parity(to_host(out), Q, K, V, W, b, S64, True, "bf16", eps=0.5)


def test_causal_state_carry_over():
    """Two calls with the state handed on equal one call; state_out is K'^T [V 1]."""
    import torch
    fv = _fv()
    B, H, L, M = 1, 2, 640, 256
    Q, K, V = _qkv(B, H, L, "bf16", seed=31)
    W, b = _features(31, H, M)
    dv = lambda x: to_dev(x, "bf16")
    h = 320
    o1, s1 = fv.attn_causal(dv(Q[:, :, :h]), dv(K[:, :, :h]), dv(V[:, :, :h]), to_dev(W),
                            to_dev(b), S64, return_state=True)
    o2, s2 = fv.attn_causal(dv(Q[:, :, h:]), dv(K[:, :, h:]), dv(V[:, :, h:]), to_dev(W),
                            to_dev(b), S64, state_in=s1, return_state=True)
    torch.cuda.synchronize()
    out = np.concatenate([to_host(o1), to_host(o2)], axis=2)
    parity(out, Q, K, V, W, b, S64, True, "bf16")
    Kp = favor.feature_map(K.astype(np.float64), W.astype(np.float64), b.astype(np.float64), S64)
    C = np.concatenate([V, np.ones(V.shape[:-1] + (1,))], -1).astype(np.float64)
    ref_state = np.swapaxes(Kp, -1, -2) @ C
    got = to_host(s2)
    assert np.max(np.abs(got - ref_state)) <= 2e-2 * np.max(np.abs(ref_state))


def test_causal_state_in_fp32():
    import torch
    fv = _fv()
    B, H, L, M = 1, 1, 200, 128
    Q, K, V = _qkv(B, H, L, "f32", seed=41)
    W, b = _features(41, H, M)
    rng = np.random.default_rng(0)
    S0 = np.abs(rng.standard_normal((B, H, M, 65))).astype(np.float32) * 5.0
    out, st = fv.attn_causal(to_dev(Q), to_dev(K), to_dev(V), to_dev(W), to_dev(b), S64,
                             state_in=to_dev(S0), return_state=True)
    torch.cuda.synchronize()
    parity(to_host(out), Q, K, V, W, b, S64, True, "f32", state_in=S0)


def test_causal_empty_sequence_passes_state_through():
    import torch
    fv = _fv()
    W, b = _features(1, 2, 64)
    S0 = np.random.default_rng(1).standard_normal((1, 2, 64, 65)).astype(np.float32)
    Z = torch.zeros((1, 2, 0, 64), device="cuda", dtype=torch.bfloat16)
    out, st = fv.attn_causal(Z, Z, Z, to_dev(W), to_dev(b), S64, state_in=to_dev(S0),
                             return_state=True)
    torch.cuda.synchronize()
    assert out.numel() == 0
    assert np.array_equal(to_host(st), S0.astype(np.float64))


# ---------------------------------------------------------------- invariants on the GPU
def test_one_hot_values_extract_attention_matrix():
    """V = I_L with L = d = 64: the output is D-hat^-1 A-hat itself."""
    import torch
    fv = _fv()
    L = 64
    Q, K, _ = _qkv(1, 1, L, "f32", seed=51)
    V = np.eye(L, dtype=np.float32)[None, None]
    W, b = _features(51, 1, 128)
    for causal in (False, True):
        f = fv.attn_causal if causal else fv.attn_bidir
        out = to_host(f(to_dev(Q), to_dev(K), to_dev(V), to_dev(W), to_dev(b), S64))
        torch.cuda.synchronize()
        Qp = favor.feature_map(Q.astype(np.float64), W.astype(np.float64), b.astype(np.float64), S64)
        Kp = favor.feature_map(K.astype(np.float64), W.astype(np.float64), b.astype(np.float64), S64)
        A = Qp[0, 0] @ Kp[0, 0].T
        if causal:
            A = np.tril(A)
        ref = A / A.sum(1, keepdims=True)
        assert np.max(np.abs(out[0, 0] - ref)) <= 1e-4 * np.max(np.abs(ref))
        if causal:
            assert np.all(np.triu(out[0, 0], 1) == 0.0)


def test_deterministic_bitwise():
    import torch
    fv = _fv()
    Q, K, V = _qkv(2, 2, 1500, "bf16", seed=61)
    W, b = _features(61, 2, 256)
    args = [to_dev(x, "bf16") for x in (Q, K, V)] + [to_dev(W), to_dev(b)]
    a1 = fv.attn_bidir(*args, S64)
    a2 = fv.attn_bidir(*args, S64)
    c1 = fv.attn_causal(*args, S64)
    c2 = fv.attn_causal(*args, S64)
    ob1, oc1 = fv.attn_both(*args, S64)
    ob2, oc2 = fv.attn_both(*args, S64)
    w1, b1 = fv.orf_draw(61, 2, 256)
    w2, b2 = fv.orf_draw(61, 2, 256)
    torch.cuda.synchronize()
    assert torch.equal(a1, a2) and torch.equal(c1, c2)
    assert torch.equal(ob1, ob2) and torch.equal(oc1, oc2)
    assert torch.equal(w1, w2) and torch.equal(b1, b2)


def test_empty_batch_is_noop():
    import torch
    fv = _fv()
    W, b = _features(1, 1, 64)
    Z = torch.zeros((0, 1, 128, 64), device="cuda", dtype=torch.bfloat16)
    assert fv.attn_bidir(Z, Z, Z, to_dev(W), to_dev(b), S64).numel() == 0
    assert fv.attn_causal(Z, Z, Z, to_dev(W), to_dev(b), S64).numel() == 0


def test_end_to_end_gpu_draw():
    """GPU-drawn features against oracle-drawn features (same seed)."""
    import torch
    fv = _fv()
    B, H, L, M = 1, 4, 2048, 256
    Q, K, V = _qkv(B, H, L, "bf16", seed=71)
    Wg, bg = fv.orf_draw(71, H, M)
    Wr, br = favor.orf_draw(71, H, M, 64)
    args = [to_dev(x, "bf16") for x in (Q, K, V)]
    ob = fv.attn_bidir(*args, Wg, bg, S64)
    oc = fv.attn_causal(*args, Wg, bg, S64)
    torch.cuda.synchronize()
    parity(to_host(ob), Q, K, V, Wr, br, S64, False, "bf16")
    parity(to_host(oc), Q, K, V, Wr, br, S64, True, "bf16")


# ---------------------------------------------------------------- both directions
@pytest.mark.parametrize("B,H,L,M,dtype,segment", [
    (2, 2, 1000, 256, "bf16", 0),
    (1, 3, 65, 64, "bf16", 64),
    (1, 2, 300, 128, "f32", 0),
])
def test_both_directions_one_pass(B, H, L, M, dtype, segment):
    import torch
    fv = _fv()
    Q, K, V = _qkv(B, H, L, dtype, seed=81 + L)
    W, b = _features(81 + L, H, M)
    args = [to_dev(x, dtype) for x in (Q, K, V)] + [to_dev(W), to_dev(b)]
    ob, oc = fv.attn_both(*args, S64, segment=segment)
    torch.cuda.synchronize()
    parity(to_host(ob), Q, K, V, W, b, S64, False, dtype)
    parity(to_host(oc), Q, K, V, W, b, S64, True, dtype)
    # the causal output is the one favor_attn_causal gives (same kernels, same order)
    oc2 = fv.attn_causal(*args, S64, segment=segment)
    torch.cuda.synchronize()
    assert torch.equal(oc, oc2)


def test_both_state_in_affects_causal_only():
    import torch
    fv = _fv()
    B, H, L, M = 1, 2, 200, 128
    Q, K, V = _qkv(B, H, L, "f32", seed=91)
    W, b = _features(91, H, M)
    S0 = np.abs(np.random.default_rng(2).standard_normal((B, H, M, 65))).astype(np.float32) * 3
    args = [to_dev(x) for x in (Q, K, V)] + [to_dev(W), to_dev(b)]
    ob, oc, st = fv.attn_both(*args, S64, state_in=to_dev(S0), return_state=True)
    oc2, st2 = fv.attn_causal(*args, S64, state_in=to_dev(S0), return_state=True)
    torch.cuda.synchronize()
    parity(to_host(ob), Q, K, V, W, b, S64, False, "f32")
    parity(to_host(oc), Q, K, V, W, b, S64, True, "f32", state_in=S0)
    assert torch.equal(oc, oc2) and torch.equal(st, st2)
