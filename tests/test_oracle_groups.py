"""Pins of the oracle's head-group reading (Sec. 5.1 remark on head groups; Sec. 5.2,
the token scale per head group; Sec. 6 setup, G = 2 groups for Llama and 1 for Qwen)."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import aatc, groups

D = 128


def _identity_group_calibration(gkv, bits=8):
    d = D * gkv
    b = np.full(d, bits, dtype=np.int64)
    budget = int(b.sum())
    return aatc.Calibration(d=d, budget=budget, record_bytes=4 * ((budget + 31) // 32),
                            d_active=d, bits=b, perm=np.arange(d), T64=np.eye(d),
                            T32=np.eye(d, dtype=np.float32),
                            s16=np.ones(d, dtype=np.float16), sigma2=np.ones(d),
                            weight=np.ones(d), bits_eig=b.copy())


def _grid_tokens(rng, n, gkv, hkv):
    """Tokens [n, hkv, 128] on the 8-bit grid of an identity calibration: every group's
    largest magnitude is exactly 1 (one element -1 per group), the rest k / 128."""
    codes = rng.integers(-127, 128, size=(n, hkv, D))
    for g in range(hkv // gkv):
        codes[:, g * gkv + rng.integers(0, gkv), 5] = -128
    return (codes / 128.0).astype(np.float32)


def test_group_tokens_concatenate_consecutive_heads():
    x = np.arange(3 * 8 * D).reshape(3, 8, D)
    xg = groups.group_tokens(x, 1, 4)
    assert xg.shape == (3, 4 * D)
    for kk in range(4):
        np.testing.assert_array_equal(xg[:, kk * D:(kk + 1) * D], x[:, 4 + kk])
    with pytest.raises(ValueError):
        groups.group_tokens(x, 2, 4)


def test_group_attention_lossless_on_grid_matches_per_head_softmax():
    """T = I over 2 x 256 group channels, 8 bits and grid tokens: the cache decodes
    exactly, so every query head must see exactly its own KV head's keys and values.  A
    wrong block, group or query-head mapping changes the result."""
    rng = np.random.default_rng(3)
    n, hkv, gkv, hq = 50, 4, 2, 12
    xk, xv = _grid_tokens(rng, n, gkv, hkv), _grid_tokens(rng, n, gkv, hkv)
    cal = _identity_group_calibration(gkv)
    krec, ka, vrec, va = [], [], [], []
    for g in range(hkv // gkv):
        r, a, _ = groups.encode_group(groups.group_tokens(xk, g, gkv), cal)
        np.testing.assert_array_equal(a.astype(np.float32), 1.0)
        krec.append(r), ka.append(a)
        r, a, _ = groups.encode_group(groups.group_tokens(xv, g, gkv), cal)
        vrec.append(r), va.append(a)
    q = rng.standard_normal((hq, D)).astype(np.float32)
    out = groups.group_attention(q, hkv, gkv, [cal] * 2, [cal] * 2, krec, ka, vrec, va, n)
    gq = hq // hkv
    for j in range(hq):
        k = j // gq
        ref = aatc.softmax_attention(q[j:j + 1], xk[:, k], xv[:, k], 1 / np.sqrt(D))
        np.testing.assert_allclose(out[j:j + 1], ref, rtol=1e-13, atol=1e-15)


def test_one_token_scale_per_group():
    """With T = I and s = 1 the group's alpha is the largest |x| over all of its heads:
    one scale per (token, group), not per head (Sec. 5.2)."""
    rng = np.random.default_rng(4)
    gkv = 4
    x = rng.standard_normal((20, gkv, D)).astype(np.float32)
    x[:, 2] *= 8.0                                    # one head dominates
    cal = _identity_group_calibration(gkv, bits=4)
    _, a16, code = groups.encode_group(groups.group_tokens(x, 0, gkv), cal)
    want = aatc.to_f16(np.abs(x).reshape(20, -1).max(axis=1))
    np.testing.assert_array_equal(a16, want)
    # the other heads' codes are coarse relative to their own range
    per_head_max = np.abs(code.reshape(20, gkv, D)).max(axis=2)
    assert np.all(per_head_max[:, 2] >= 7) and np.all(per_head_max[:, 0] <= 4)


def test_group_of_one_head_is_the_per_head_method():
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((300, 2, D)) * np.linspace(2, 0.1, D)).astype(np.float32)
    a = groups.calibrate_group(groups.group_tokens(x, 1, 1), 2.75)
    b = aatc.calibrate(x[:, 1], 2.75)
    np.testing.assert_array_equal(a.bits, b.bits)
    np.testing.assert_array_equal(a.T32, b.T32)
    np.testing.assert_array_equal(a.s16, b.s16)


def test_group_budget_and_widths():
    rng = np.random.default_rng(6)
    gkv = 4
    x = (rng.standard_normal((2000, gkv * D)) *
         np.repeat(np.linspace(3, 0.05, D)[None, :], gkv, axis=0).ravel()).astype(np.float32)
    cal = groups.calibrate_group(x, 2.75, b_max=16)
    assert cal.d == 512 and cal.budget == round(2.75 * 512) == int(cal.bits.sum())
    assert cal.record_bytes == 4 * ((1408 + 31) // 32) == 176
    assert np.all(np.diff(cal.bits) <= 0) and cal.bits.max() <= 16
    t = cal.T64
    np.testing.assert_allclose(t.T @ t, np.eye(512), atol=1e-10)


def test_block_diagonal_covariance_gives_block_supported_channels():
    """Independent heads with disjoint spectra: the group PCA's channels each live in one
    head's block (eigenvectors of a block-diagonal covariance), and the group's
    eigenvalues are the union of the heads' own."""
    rng = np.random.default_rng(7)
    gkv, n = 2, 20000
    lam0 = 4.0 ** -np.arange(D) * 10.0
    lam1 = lam0 * 3.0
    z = rng.standard_normal((n, 2 * D))
    u0 = np.linalg.qr(rng.standard_normal((D, D)))[0]
    u1 = np.linalg.qr(rng.standard_normal((D, D)))[0]
    x0 = (z[:, :D] * np.sqrt(lam0)) @ u0.T
    x1 = (z[:, D:] * np.sqrt(lam1)) @ u1.T
    xg = np.concatenate([x0, x1], axis=1)
    sigma = aatc.covariance(xg)
    sigma[:D, D:] = 0.0                         # exactly block-diagonal
    sigma[D:, :D] = 0.0
    p, lam = aatc.pca_basis(sigma)
    top = p[:, :16]
    in0 = np.abs(top[:D]).max(axis=0)
    in1 = np.abs(top[D:]).max(axis=0)
    assert np.all(np.minimum(in0, in1) < 1e-9)
    both = np.sort(np.concatenate([np.linalg.eigvalsh(sigma[:D, :D]),
                                   np.linalg.eigvalsh(sigma[D:, D:])]))[::-1]
    np.testing.assert_allclose(lam[:16], both[:16], rtol=1e-9)


def test_embedded_queries_sum_over_the_group_query_heads():
    """Key weights of a group: w_c = (1/T) sum over every query head of the group of
    (P_c^T q)^2, each query in its KV head's block; with P = I that is the per-element
    mean square of the queries of the block's head."""
    rng = np.random.default_rng(8)
    t, gkv, gq = 30, 2, 3
    q = rng.standard_normal((t, gkv, gq, D))
    qe = groups.embed_group_queries(q, gkv)
    w = aatc.key_weights(np.eye(gkv * D), qe, gkv * gq)
    for kk in range(gkv):
        want = (q[:, kk] ** 2).sum(axis=1).mean(axis=0)
        np.testing.assert_allclose(w[kk * D:(kk + 1) * D], want, rtol=1e-12)


def test_transform_of_512_elements_is_the_rational_definition():
    rng = np.random.default_rng(9)
    d = 512
    t = aatc.stored_transform(np.linalg.qr(rng.standard_normal((d, d)))[0])
    x = rng.standard_normal((3, d)).astype(np.float32)
    x[1, :7] *= 2.0 ** -30                      # a wide exponent range
    h = aatc.transform(x, t)
    for i in range(3):
        for c in (0, 1, 255, 511):
            acc = sum(Fraction(float(x[i, j])) * Fraction(float(t[j, c])) for j in range(d))
            assert h[i, c] == aatc.round_to_f32(acc)
