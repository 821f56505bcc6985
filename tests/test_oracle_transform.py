"""Pins of the oracle's transform step (Sec. 3.1, Sec. 5.1, App. D)."""
from fractions import Fraction

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


def _rational_transform(x, t):
    """Every element by exact rational arithmetic: the definition with no fast path."""
    out = np.zeros((x.shape[0], t.shape[1]), dtype=np.float32)
    for i in range(x.shape[0]):
        for c in range(t.shape[1]):
            acc = Fraction(0)
            for j in range(x.shape[1]):
                acc += Fraction(float(x[i, j])) * Fraction(float(t[j, c]))
            out[i, c] = aatc.round_to_f32(acc)
    return out


def test_stored_transform_grid():
    """Entries are the nearest multiples of 2^-22, exactly representable in fp32."""
    rng = np.random.default_rng(7)
    t64 = haar_orthogonal(rng, 128)
    t = aatc.stored_transform(t64)
    assert t.dtype == np.float32
    q = np.ldexp(t.astype(np.float64), 22)
    np.testing.assert_array_equal(q, np.rint(q))
    assert np.abs(t.astype(np.float64) - t64).max() <= 2.0 ** -23
    np.testing.assert_array_equal(aatc.stored_transform(np.eye(16)), np.eye(16))


def test_round_to_f32_matches_ieee_cast():
    """round_to_f32 on rationals that are fp64 numbers equals the hardware fp64 -> fp32
    conversion (round to nearest, ties to even), including ties, subnormals and overflow."""
    rng = np.random.default_rng(8)
    vals = [1 + 2.0 ** -24, 1 + 3 * 2.0 ** -24, -(1 + 2.0 ** -24), 2.0 ** -149,
            2.0 ** -150, 3 * 2.0 ** -151, 2.0 ** -126 * (1 - 2.0 ** -25), 3.4028235677973366e38,
            2.0 ** 128 * (1 - 2.0 ** -25), 2.0 ** 128 * (1 - 2.0 ** -26), 0.1, -7.25e-40]
    vals += list(rng.standard_normal(2000) * np.exp2(rng.integers(-160, 130, 2000)))
    for v in vals:
        with np.errstate(over="ignore"):
            want = np.float64(v).astype(np.float32)
        got = aatc.round_to_f32(Fraction(v))
        assert got == want or (np.isinf(got) and np.isinf(want) and got == want), v


def test_int64_to_f32_cast_rounds_to_nearest_even():
    """The oracle's transform relies on numpy's int64 -> float32 conversion rounding once,
    to nearest with ties to even: checked against exact rational rounding on ties and on
    integers with many trailing zeros."""
    ties = [2 ** 24 + 1, 2 ** 24 + 3, -(2 ** 24 + 1), 2 ** 59 + 2 ** 35, 2 ** 59 + 2 ** 35 + 1,
            -(2 ** 40 + 2 ** 16), -(2 ** 40 + 2 ** 16 + 1), 2 ** 60 - 1]
    rng = np.random.default_rng(13)
    v = rng.integers(-2 ** 62, 2 ** 62, size=4000)
    v = (v >> rng.integers(0, 40, size=v.size)) << rng.integers(0, 20, size=v.size)
    vals = np.concatenate([np.array(ties, dtype=np.int64), v])
    got = vals.astype(np.float32)
    for a, g in zip(vals, got):
        assert aatc.round_to_f32(Fraction(int(a))) == g, int(a)


def test_transform_matches_rational_definition():
    """Random bf16-valued and fp32 tokens against exact rational sums, element by element."""
    from kvsynth.gen import bf16_bits_to_f32, f32_to_bf16_bits
    rng = np.random.default_rng(9)
    t = aatc.stored_transform(haar_orthogonal(rng, 128))[:, :12]
    xb = bf16_bits_to_f32(f32_to_bf16_bits(
        (rng.standard_normal((6, 128)) * rng.lognormal(0, 3, (6, 1))).astype(np.float32)))
    xf = (rng.standard_normal((6, 128)) * np.exp2(rng.integers(-30, 30, (6, 128)))).astype(np.float32)
    for x in (xb, xf):
        np.testing.assert_array_equal(aatc.transform(x, t), _rational_transform(x, t))


def test_transform_near_ties():
    """Sums within 2^-62 of an fp32 halfway point: summing in fp64 and then rounding to
    fp32 rounds twice and lands on the tie; the exact sum does not."""
    t = np.zeros((4, 1), dtype=np.float32)
    t[:, 0] = [1.0, 2.0 ** -22, 2.0 ** -22, 2.0 ** -22]
    cases = [
        # (x, exact result)
        ([1.0, 0.25, 2.0 ** -40, 0.0], 1 + 2.0 ** -23),      # just above the tie: up
        ([1.0, 0.25, -2.0 ** -40, 0.0], 1.0),                # just below the tie: down
        ([1.0, 0.25, 0.0, 0.0], 1.0),                        # the tie itself: to even
        ([1.0, 0.75, 0.0, 0.0], 1 + 2.0 ** -22),             # odd neighbour below: up
        ([-1.0, -0.25, -2.0 ** -40, 0.0], -(1 + 2.0 ** -23)),
        ([2.0 ** -100, 2.0 ** -100, 2.0 ** -60, -2.0 ** -60], 2.0 ** -100 + 2.0 ** -122),
    ]
    x = np.array([c[0] for c in cases], dtype=np.float32)
    want = np.array([[c[1]] for c in cases], dtype=np.float32)
    np.testing.assert_array_equal(aatc.transform(x, t), want)
    np.testing.assert_array_equal(_rational_transform(x, t), want)
    naive = (x.astype(np.float64) @ t.astype(np.float64)).astype(np.float32)
    assert naive[0, 0] != want[0, 0] and naive[4, 0] != want[4, 0]


def test_transform_identity_sign_and_scaling():
    """T = I gives h = x; h(-x) = -h(x); power-of-two scaling of x scales h exactly."""
    rng = np.random.default_rng(10)
    x = (rng.standard_normal((50, 128)) * np.exp2(rng.integers(-20, 20, (50, 1)))).astype(np.float32)
    np.testing.assert_array_equal(aatc.transform(x, np.eye(128, dtype=np.float32)), x)
    t = aatc.stored_transform(haar_orthogonal(rng, 128))
    h = aatc.transform(x, t)
    np.testing.assert_array_equal(aatc.transform(-x, t), -h)
    np.testing.assert_array_equal(aatc.transform(np.ldexp(x, 7), t), np.ldexp(h, 7))
    # and the zero token
    np.testing.assert_array_equal(aatc.transform(np.zeros((2, 128), np.float32), t), 0)


def test_transform_subnormal_results():
    """Sums below 2^-126 round to the fp32 subnormal grid (quantum 2^-149)."""
    t = np.zeros((2, 1), dtype=np.float32)
    t[:, 0] = [2.0 ** -22, 2.0 ** -22]
    x = np.array([[2.0 ** -120, 2.0 ** -126],            # 2^-142 + 2^-148: exact
                  [2.0 ** -126, 2.0 ** -127]], dtype=np.float32)   # 2^-148 + 2^-149: exact
    want = np.array([[2.0 ** -142 + 2.0 ** -148], [3 * 2.0 ** -149]], dtype=np.float32)
    np.testing.assert_array_equal(aatc.transform(x, t), want)
    x2 = np.array([[2.0 ** -127, 2.0 ** -149 * 3]], dtype=np.float32)  # 2^-149 + 1.5 2^-171
    np.testing.assert_array_equal(aatc.transform(x2, t), np.float32(2.0 ** -149))


# ---------------------------------------------------------------------------------------
# The paper's form of Step 1 (Sec. 5.1): whitened SVD from layer inputs and a projection
# ---------------------------------------------------------------------------------------
def test_whitened_svd_factorization_identities():
    """eq. AB-factorization: W = A B; A^T Sigma_X A = S (so H = X A has uncorrelated
    channels of variance S_c, in decreasing order); B = sqrt(S) P^T with orthonormal P."""
    from kvsynth import layer_inputs, projection
    x = layer_inputs(3, 1024, 64).astype(np.float64)
    w = projection(3, 64, 16).astype(np.float64)
    a_mat, b_mat, s, p = aatc.whitened_svd(x, w)
    np.testing.assert_allclose(a_mat @ b_mat, w, atol=1e-12 * np.abs(w).max())
    sig_x = x.T @ x / x.shape[0]
    np.testing.assert_allclose(a_mat.T @ sig_x @ a_mat, np.diag(s), atol=1e-10 * s[0])
    h = x @ a_mat
    np.testing.assert_allclose(h.T @ h / h.shape[0], np.diag(s), atol=1e-10 * s[0])
    assert np.all(np.diff(s) <= 0)
    np.testing.assert_allclose(p.T @ p, np.eye(16), atol=1e-12)
    np.testing.assert_allclose(b_mat @ b_mat.T, np.diag(s), atol=1e-12 * s[0])


def test_whitened_calibration_closed_form_on_whitened_inputs():
    """Sigma_X = I (inputs already white) and W = diag(2, 1, 1/2, 1/4): L = I, W~ = W, the
    singular values are (2, 1, 1/2, 1/4), P = I, and K's channel variances S^2 = (4, 1, 1/4,
    1/16) are the worked reverse water-filling example: 4 bits go (3, 1, 0, 0)."""
    n, d = 4096, 4
    q, _ = np.linalg.qr(np.random.default_rng(5).standard_normal((n, d)))
    x = q * np.sqrt(n)                                  # X^T X / n = I exactly (to rounding)
    w = np.diag([2.0, 1.0, 0.5, 0.25])
    a_mat, b_mat, s, p = aatc.whitened_svd(x, w)
    np.testing.assert_allclose(s, [2.0, 1.0, 0.5, 0.25], rtol=1e-12)
    np.testing.assert_allclose(np.abs(p), np.eye(4), atol=1e-12)
    cal = aatc.calibrate_whitened(x, w, avg_bits=1.0)
    np.testing.assert_allclose(cal.sigma2, [4.0, 1.0, 0.25, 0.0625], rtol=1e-12)
    # the variances come out of an SVD, so the exact ties of the worked example are broken
    # by the last bit; any of its three optima (objective 0.625) is the answer
    assert cal.bits_eig.tolist() in ([3, 1, 0, 0], [2, 2, 0, 0], [2, 1, 1, 0])
    assert aatc.allocation_objective([4.0, 1.0, 0.25, 0.0625], cal.bits_eig) == \
        pytest.approx(0.625, rel=1e-12)


@pytest.mark.parametrize("weights", ["var_only", "queries", "w_o"])
def test_whitened_calibration_equals_pca_of_the_keys(weights):
    """App. D: the whitened SVD of W and the PCA of K = X W give the same channels and the
    same products w_c sigma_c^2, so the same widths, stored transform and scales."""
    from kvsynth import layer_inputs, projection
    x = layer_inputs(7, 2048, 192)
    w = projection(7, 192, 128)
    k = x.astype(np.float64) @ w.astype(np.float64)
    rng = np.random.default_rng(8)
    kw = {}
    if weights == "queries":
        kw = dict(q_calib=rng.standard_normal((4 * 200, 128)), group=4)
    elif weights == "w_o":
        kw = dict(w_o=rng.standard_normal((128, 96)))
    c1 = aatc.calibrate_whitened(x, w, 2.75, **kw)
    c2 = aatc.calibrate(k, 2.75, **kw)
    np.testing.assert_array_equal(c1.bits, c2.bits)
    np.testing.assert_array_equal(c1.perm, c2.perm)
    np.testing.assert_allclose(c1.weight * c1.sigma2, c2.weight * c2.sigma2,
                               rtol=1e-8, atol=1e-12 * (c2.weight * c2.sigma2).max())
    np.testing.assert_allclose(c1.T64, c2.T64, atol=1e-10)
    np.testing.assert_array_equal(c1.s16, c2.s16)
