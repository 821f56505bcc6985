"""Pins of the oracle's transform step (Sec. 3.1, Sec. 5.1, App. D)."""
import numpy as np
import pytest

from kvsynth import haar_orthogonal
from oracle import aatc


def _exact_cov_samples(rng, u, lam, n):
    """Samples whose uncentered sample covariance is exactly U diag(lam) U^T."""
    d = u.shape[0]
    z, _ = np.linalg.qr(rng.standard_normal((n, d)))      # orthonormal columns
    z *= np.sqrt(n)
    return (z * np.sqrt(lam)[None, :]) @ u.T


def test_pca_recovers_known_basis():
    rng = np.random.default_rng(0)
    d = 32
    u = haar_orthogonal(rng, d)
    lam = np.arange(1, d + 1, dtype=float) ** -1.5
    x = _exact_cov_samples(rng, u, lam, 512)
    p, ev = aatc.pca_basis(aatc.covariance(x))
    np.testing.assert_allclose(ev, lam, rtol=1e-10, atol=1e-14)
    # Same columns up to sign; the canonical sign makes the largest entry positive.
    for c in range(d):
        col = u[:, c] * np.sign(u[np.argmax(np.abs(u[:, c])), c])
        np.testing.assert_allclose(p[:, c], col, atol=1e-9)
        assert p[np.argmax(np.abs(p[:, c])), c] > 0


def test_transform_orthonormal_roundtrip_and_decorrelating():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((2048, 128)) @ rng.standard_normal((128, 128))
    cal = aatc.calibrate(x, 2.75)
    t = cal.T64
    np.testing.assert_allclose(t.T @ t, np.eye(128), atol=1e-12)
    np.testing.assert_allclose((x @ t) @ t.T, x, atol=1e-9 * np.abs(x).max())
    h = x @ t
    c = h.T @ h / h.shape[0]
    off = c - np.diag(np.diag(c))
    assert np.abs(off).max() <= 1e-10 * np.abs(np.diag(c)).max()
    # Channel variances are the eigenvalues, in storage order.
    np.testing.assert_allclose(np.diag(c), cal.sigma2[cal.perm], rtol=1e-9)


def test_paper_whitening_form_gives_same_allocation():
    """App. D: the whitening-based SVD and the PCA of K = X W give the same channels,
    and w_c * sigma_c^2 agrees, so both forms allocate the same bits."""
    rng = np.random.default_rng(2)
    n, dm, d = 4096, 48, 16
    x = rng.standard_normal((n, dm)) @ rng.standard_normal((dm, dm))
    w_k = rng.standard_normal((dm, d))
    queries = rng.standard_normal((300, d)) @ rng.standard_normal((d, d))
    # Paper form (Sec. 5.1): Sigma_X = L L^T, W~ = L^T W = U S P^T,
    # A = L^-T U sqrt(S), B = sqrt(S) P^T, H = X A, weights from B.
    sig_x = x.T @ x / n
    chol = np.linalg.cholesky(sig_x)
    uu, ss, pt = np.linalg.svd(chol.T @ w_k, full_matrices=False)
    a_mat = np.linalg.solve(chol.T, uu) * np.sqrt(ss)[None, :]
    b_mat = np.sqrt(ss)[:, None] * pt
    h = x @ a_mat
    var_h = (h ** 2).mean(axis=0)
    np.testing.assert_allclose(var_h, ss, rtol=1e-8)          # S = A^T Sigma_X A
    w_paper = ((queries @ b_mat.T) ** 2).mean(axis=0)
    wv_paper = w_paper * var_h
    # Oracle form: PCA of the keys, w from the eigenvectors.
    k = x @ w_k
    p, lam = aatc.pca_basis(aatc.covariance(k))
    wv_oracle = aatc.key_weights(p, queries, 1) * lam
    np.testing.assert_allclose(np.sort(wv_oracle), np.sort(wv_paper), rtol=1e-7)
    b1 = aatc.allocate_bits(np.sort(wv_oracle)[::-1], 40, 8)
    b2 = aatc.allocate_bits(np.sort(wv_paper)[::-1], 40, 8)
    np.testing.assert_array_equal(b1, b2)


def test_key_and_value_weights_special_cases():
    rng = np.random.default_rng(4)
    d = 8
    p = haar_orthogonal(rng, d)
    # Queries along one eigenvector load only that channel.
    q = np.outer(rng.standard_normal(50), p[:, 3])
    w = aatc.key_weights(p, q, 1)
    assert np.argmax(w) == 3 and np.allclose(np.delete(w, 3), 0, atol=1e-24)
    # GQA: two heads with the same queries give twice the single-head weight.
    q2 = np.concatenate([q, q])
    np.testing.assert_allclose(aatc.key_weights(p, q2, 2), 2 * w)
    # W_O = I gives unit value weights (orthonormal P).
    np.testing.assert_allclose(aatc.value_weights(p, np.eye(d)), np.ones(d), atol=1e-12)


def test_fixed_point_transform_identity_on_grid():
    """T = I and inputs with <= 14 significant bits below the token maximum: exact."""
    rng = np.random.default_rng(5)
    d = 16
    ints = rng.integers(-8191, 8192, size=(40, d))
    ints[:, 0] = 8191
    x = np.ldexp(ints.astype(np.float64), rng.integers(-20, 5, size=(40, 1))).astype(np.float32)
    h = aatc.fixed_point_transform(x, np.eye(d, dtype=np.float32))
    np.testing.assert_array_equal(h, x)


def test_fixed_point_transform_error_bound():
    """|h - T^T x| stays within the fixed-point resolution bound for real data."""
    rng = np.random.default_rng(6)
    x = (rng.standard_normal((500, 128)) * rng.lognormal(0, 2, size=(500, 1))).astype(np.float32)
    t = haar_orthogonal(rng, 128).astype(np.float32)
    h = aatc.fixed_point_transform(x, t).astype(np.float64)
    exact = x.astype(np.float64) @ t.astype(np.float64)
    xa = np.abs(x.astype(np.float64))
    m = xa.max(axis=1)
    e = np.frexp(m)[1] - 1
    x_res = np.ldexp(0.5, -(aatc.X_LEAD_BIT - e))               # half an x step
    bound = (xa.sum(axis=1) * 2.0 ** -(aatc.T_FRAC_BITS + 1)
             + x_res * np.abs(t).sum(axis=0).max() * (1 + 2.0 ** -14))[:, None]
    bound = bound + np.abs(exact) * 2.0 ** -24
    assert np.all(np.abs(h - exact) <= bound)
    assert np.all(np.abs(h - exact) <= 1e-3 * np.linalg.norm(x, axis=1, keepdims=True))


def test_fixed_point_transform_zero_token():
    x = np.zeros((3, 8), dtype=np.float32)
    x[1, 2] = 1.5
    h = aatc.fixed_point_transform(x, np.eye(8, dtype=np.float32))
    np.testing.assert_array_equal(h, x)
