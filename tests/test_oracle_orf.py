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
