"""Pins for the oracle's orthogonal-random-feature draw (Sec. 2.4, R-ORFs).

Checked against: numpy's Householder QR (a library routine the oracle does not
use), exact orthogonality within each d x d block, the chi_d law of the row
norms, the N(0, 1) marginals ORFs are meant to keep, and the phase law.
"""
import numpy as np
import pytest
from scipy import stats

from oracle import favor, philox


def test_gram_schmidt_equals_sign_fixed_qr():
    rng = np.random.default_rng(0)
    for n in (4, 16, 64):
        G = rng.standard_normal((n, n))
        Qgs = favor.gram_schmidt_rows(G)
        # rows of G = L Qgs with L lower triangular, positive diagonal
        # <=> G^T = Qgs^T L^T is the QR factorisation of G^T with diag(R) > 0
        q, r = np.linalg.qr(G.T)
        sgn = np.sign(np.diag(r))
        assert np.allclose(Qgs, (q * sgn).T, atol=1e-10)


@pytest.mark.parametrize("M,d", [(256, 64), (128, 64), (40, 16), (48, 16)])
def test_blocks_orthogonal_with_chi_norms(M, d):
    W, b = favor.orf_draw(5, 3, M, d, favor.RF_ORTHO_CHI)
    assert W.shape == (3, M, d) and b.shape == (3, M)
    for h in range(3):
        for k in range(-(-M // d)):
            blk = W[h, k * d:(k + 1) * d]
            G = blk @ blk.T
            rho2 = np.sum(blk * blk, axis=1)
            off = G - np.diag(np.diag(G))
            assert np.max(np.abs(off) / np.sqrt(np.outer(rho2, rho2))) < 1e-12
    # different blocks are independent, not orthogonal to each other
    if M >= 2 * d:
        cross = W[0, :d] @ W[0, d:2 * d].T
        assert np.max(np.abs(cross)) > 1.0


def test_row_norms_are_chi_d():
    d = 64
    W, _ = favor.orf_draw(11, 16, 256, d, favor.RF_ORTHO_CHI)
    rho2 = np.sum(W * W, axis=-1).ravel()
    assert stats.kstest(rho2, stats.chi2(d).cdf).pvalue > 1e-3


def test_orf_entries_keep_gaussian_marginals():
    W, _ = favor.orf_draw(12, 16, 256, 64, favor.RF_ORTHO_CHI)
    # 262144 entries; each is marginally N(0,1) (the point of R-ORFs)
    x = W.ravel()[::7]
    assert stats.kstest(x, "norm").pvalue > 1e-3


def test_fixed_kind_norms():
    d = 32
    W, _ = favor.orf_draw(3, 2, 64, d, favor.RF_ORTHO_FIXED)
    assert np.allclose(np.sum(W * W, axis=-1), d, rtol=1e-12)


def test_iid_kind_is_unstructured_gaussian():
    d = 64
    W, _ = favor.orf_draw(4, 8, 256, d, favor.RF_IID)
    assert stats.kstest(W.ravel(), "norm").pvalue > 1e-3
    blk = W[0, :d]
    off = blk @ blk.T - np.diag(np.sum(blk * blk, axis=1))
    assert np.max(np.abs(off)) > 5.0     # not orthogonal


def test_phases_uniform_on_0_2pi():
    _, b = favor.orf_draw(8, 32, 256, 64)
    assert np.all(b > 0) and np.all(b < 2 * np.pi)
    assert stats.kstest(b.ravel() / (2 * np.pi), "uniform").pvalue > 1e-3


def test_draw_is_deterministic_and_seeded():
    W1, b1 = favor.orf_draw(9, 2, 128, 64)
    W2, b2 = favor.orf_draw(9, 2, 128, 64)
    W3, _ = favor.orf_draw(10, 2, 128, 64)
    assert np.array_equal(W1, W2) and np.array_equal(b1, b2)
    assert not np.allclose(W1, W3)


def test_head_h_uses_its_own_stream():
    W_all, b_all = favor.orf_draw(21, 3, 64, 16)
    # the Gaussian block of head 2 comes from (seed, head=2, purpose ORF)
    g = philox.gaussians(21, 2, philox.PURPOSE_ORF, 4 * 16 * 16).reshape(4, 16, 16)
    q0 = favor.gram_schmidt_rows(g[0])
    rho = np.linalg.norm(W_all[2, :16], axis=1)
    assert np.allclose(W_all[2, :16] / rho[:, None], q0, atol=1e-12)


# ---------------------------------------------------------------- structured ORFs
def test_hadamard_matrix_matches_scipy_sylvester_construction():
    import scipy.linalg
    for d in (2, 16, 64):
        np.testing.assert_array_equal(favor.hadamard(d) * np.sqrt(d), scipy.linalg.hadamard(d))


def test_hadamard_orf_block_is_the_hd_product_and_orthogonal():
    import scipy.linalg
    d = 64
    for blk in (0, 3):
        W = favor.hadamard_block(11, 2, blk, d)
        np.testing.assert_allclose(W @ W.T, d * np.eye(d), atol=1e-10)
        H = scipy.linalg.hadamard(d) / np.sqrt(d)
        D = favor.hadamard_signs(11, 2, blk, d)
        ref = np.sqrt(d) * H @ np.diag(D[2]) @ H @ np.diag(D[1]) @ H @ np.diag(D[0])
        np.testing.assert_allclose(W, ref, atol=1e-12)


def test_hadamard_signs_are_fair_and_block_local():
    D = np.concatenate([favor.hadamard_signs(5, h, blk, 64).ravel()
                        for h in range(4) for blk in range(8)])
    assert set(np.unique(D)) == {-1.0, 1.0}
    n = D.size
    assert abs(np.sum(D > 0) - n / 2) < 4 * np.sqrt(n / 4)
    # block 1 reads the stream after block 0: no overlap
    assert not np.array_equal(favor.hadamard_signs(5, 0, 0, 64), favor.hadamard_signs(5, 0, 1, 64))


def test_hadamard_orf_entries_are_nearly_gaussian():
    """Three HD factors: entries of sqrt(d) H D3 H D2 H D1 have mean 0, variance 1
    (rows of norm sqrt(d)) and a fourth moment near the Gaussian 3."""
    x = np.concatenate([favor.hadamard_block(7, h, 0, 64).ravel() for h in range(40)])
    assert abs(x.mean()) < 0.02
    np.testing.assert_allclose(np.mean(x * x), 1.0, atol=1e-12)
    assert 2.6 < np.mean(x ** 4) < 3.1


def test_givens_parameters_are_valid():
    i, j, th = favor.givens_params(3, 1, 2, 64, 5000)
    assert i.min() >= 0 and i.max() < 64 and j.min() >= 0 and j.max() < 64
    assert np.all(i != j)
    assert th.min() > 0 and th.max() < 2 * np.pi
    # pairs spread over all coordinates
    assert len(np.unique(i)) == 64 and len(np.unique(j)) == 64


def test_givens_block_is_the_rotation_product():
    d = 8
    for K in (1, 2, 3):
        W = favor.givens_block(9, 0, 1, d, K)
        i, j, th = favor.givens_params(9, 0, 1, d, K)
        ref = np.eye(d)
        for t in range(K):
            G = np.eye(d)
            c, s = np.cos(th[t]), np.sin(th[t])
            G[i[t], i[t]] = c
            G[j[t], j[t]] = c
            G[i[t], j[t]] = -s
            G[j[t], i[t]] = s
            ref = ref @ G
        np.testing.assert_allclose(W, np.sqrt(d) * ref, atol=1e-13)


def test_givens_orf_is_orthogonal_and_mixes():
    d = 64
    W = favor.givens_block(4, 0, 0, d)
    np.testing.assert_allclose(W @ W.T, d * np.eye(d), atol=1e-10)
    # 2 d log2 d rotations spread the mass: entries close to the N(0, 1) marginals
    # of a Haar-random orthogonal matrix (d log2 d alone leaves a fourth moment ~5.5)
    x = np.concatenate([favor.givens_block(4, h, 0, d).ravel() for h in range(30)])
    assert abs(x.mean()) < 0.03
    assert 2.7 < np.mean(x ** 4) < 3.3
    assert favor.givens_count(64) == 768


def test_orf_draw_structured_kinds_stack_blocks():
    W, b = favor.orf_draw(21, 2, 100, 64, favor.RF_HADAMARD)
    assert W.shape == (2, 100, 64)
    np.testing.assert_allclose(W[1, :64], favor.hadamard_block(21, 1, 0, 64), atol=0)
    np.testing.assert_allclose(W[1, 64:], favor.hadamard_block(21, 1, 1, 64)[:36], atol=0)
    W, _ = favor.orf_draw(21, 1, 64, 64, favor.RF_GIVENS)
    np.testing.assert_allclose(W[0], favor.givens_block(21, 0, 0, 64), atol=0)


def test_orf_draw_head_subset_equals_the_full_draw():
    """Drawing a subset of heads gives exactly those heads' rows of the full draw."""
    W, b = favor.orf_draw(5, 6, 100, 64)
    Ws, bs = favor.orf_draw(5, 6, 100, 64, heads=[4, 1])
    assert np.array_equal(Ws, W[[4, 1]]) and np.array_equal(bs, b[[4, 1]])
