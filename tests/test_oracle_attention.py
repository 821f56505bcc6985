"""Pins of the oracle's decode attention (Def. 1; Alg. 1, online part)."""
import numpy as np
import pytest
import torch

from kvsynth import workload
from oracle import aatc


def test_softmax_attention_matches_torch_sdpa():
    rng = np.random.default_rng(0)
    q = rng.standard_normal((4, 64))
    k = rng.standard_normal((300, 64))
    v = rng.standard_normal((300, 64))
    ours = aatc.softmax_attention(q, k, v, 1 / 8)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, :, None], torch.from_numpy(k)[None, None].expand(1, 4, -1, -1),
        torch.from_numpy(v)[None, None].expand(1, 4, -1, -1), scale=1 / 8)[0, :, 0].numpy()
    np.testing.assert_allclose(ours, ref, rtol=1e-12, atol=1e-14)


def test_softmax_attention_brute_force_loops():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((2, 5))
    k = rng.standard_normal((7, 5))
    v = rng.standard_normal((7, 3))
    ours = aatc.softmax_attention(q, k, v, 0.3)
    for h in range(2):
        w = [np.exp(0.3 * sum(q[h, j] * k[i, j] for j in range(5))) for i in range(7)]
        z = sum(w)
        for c in range(3):
            assert ours[h, c] == pytest.approx(sum(w[i] * v[i, c] for i in range(7)) / z,
                                               rel=1e-12)


def _identity_calibration(d, bits, s):
    budget = int(np.sum(bits))
    return aatc.Calibration(d=d, budget=budget, record_bytes=4 * ((budget + 31) // 32),
                            d_active=int(np.count_nonzero(bits)), bits=np.array(bits),
                            perm=np.arange(d), T64=np.eye(d), T32=np.eye(d, dtype=np.float32),
                            s16=np.asarray(s, dtype=np.float64).astype(np.float16),
                            sigma2=np.ones(d), weight=np.ones(d), bits_eig=np.array(bits))


def test_lossless_special_case_on_grid():
    """T = I, 8 bits everywhere and tokens on the quantizer grid: the decoded cache is
    exact, so the attention equals plain softmax attention."""
    rng = np.random.default_rng(2)
    d, n = 8, 40
    codes = rng.integers(-128, 128, size=(n, d))
    codes[:, 0] = -128                  # alpha = 1 for every token
    x = (codes / 128.0).astype(np.float32)
    cal = _identity_calibration(d, [8] * d, [1.0] * d)
    rec, a16, _ = aatc.encode(x, cal)
    xh = aatc.decode_tokens(rec, a16, cal)
    np.testing.assert_array_equal(xh, x.astype(np.float64))
    q = rng.standard_normal((2, d)).astype(np.float32)
    out = aatc.decode_attention(q, [cal], [cal], [rec], [a16], [rec], [a16], n)
    np.testing.assert_allclose(out, aatc.softmax_attention(q, x, x, 1 / np.sqrt(d)),
                               rtol=1e-13)


def test_single_token_cache_returns_its_value():
    w = workload(1, n_tokens=1)
    cal_k = aatc.calibrate(w.calib(0, "k"), 2.75)
    cal_v = aatc.calibrate(w.calib(0, "v"), 2.75)
    k = w.as_f32(w.cache(0, 0, "k"))
    v = w.as_f32(w.cache(0, 0, "v"))
    kr, ka, _ = aatc.encode(k, cal_k)
    vr, va, _ = aatc.encode(v, cal_v)
    q = w.as_f32(w.queries(0))
    out = aatc.decode_attention(q, [cal_k], [cal_v], [kr], [ka], [vr], [va], 1)
    np.testing.assert_allclose(out[0], aatc.decode_tokens(vr, va, cal_v)[0], rtol=1e-12)


def test_attention_error_shrinks_with_bits():
    """Error goes to zero as the budget grows (Sec. 3.1; Theorem 1 with vanishing noise)."""
    w = workload(1, n_tokens=256)
    k = w.as_f32(w.cache(0, 0, "k"))
    v = w.as_f32(w.cache(0, 0, "v"))
    q = w.as_f32(w.queries(0))
    exact = aatc.softmax_attention(q, k, v, 1 / np.sqrt(128))
    errs = []
    for avg in (1.0, 2.0, 4.0, 6.0, 8.0):
        ck = aatc.calibrate(w.calib(0, "k"), avg)
        cv = aatc.calibrate(w.calib(0, "v"), avg)
        kr, ka, _ = aatc.encode(k, ck)
        vr, va, _ = aatc.encode(v, cv)
        out = aatc.decode_attention(q, [ck], [cv], [kr], [ka], [vr], [va], 256)
        errs.append(np.linalg.norm(out - exact) / np.linalg.norm(exact))
    assert all(a > b for a, b in zip(errs, errs[1:]))
    assert errs[-1] < 0.02


def test_gqa_heads_read_their_kv_head():
    w = workload(2, n_tokens=64)
    cals_k = [aatc.calibrate(w.calib(h, "k"), 2.75) for h in range(2)]
    cals_v = [aatc.calibrate(w.calib(h, "v"), 2.75) for h in range(2)]
    enc_k = [aatc.encode(w.as_f32(w.cache(0, h, "k")), cals_k[h]) for h in range(2)]
    enc_v = [aatc.encode(w.as_f32(w.cache(0, h, "v")), cals_v[h]) for h in range(2)]
    q = w.as_f32(w.queries(0))[:8]
    out = aatc.decode_attention(q, cals_k, cals_v, [e[0] for e in enc_k], [e[1] for e in enc_k],
                                [e[0] for e in enc_v], [e[1] for e in enc_v], 64)
    for h in range(2):
        kh = aatc.decode_tokens(enc_k[h][0], enc_k[h][1], cals_k[h])
        vh = aatc.decode_tokens(enc_v[h][0], enc_v[h][1], cals_v[h])
        np.testing.assert_allclose(out[4 * h:4 * h + 4],
                                   aatc.softmax_attention(q[4 * h:4 * h + 4], kh, vh,
                                                          1 / np.sqrt(128)), rtol=1e-12)


def test_midrise_grid_special_case():
    """T = I and b = 12 (beyond the printed 8-bit setting; App. E allows 16) with the
    midrise reading: each token's channel 0 is 1 (so alpha = 1, Delta = 2 / 2^b) and the
    others sit on the midrise levels (code + 1/2) Delta.  Those decode exactly; channel 0
    lands on the top level 1 - Delta / 2 (midrise has no level at alpha).  The attention
    equals plain softmax attention over exactly that cache."""
    rng = np.random.default_rng(3)
    d, n, b = 8, 40, 12
    half = 1 << (b - 1)
    codes = rng.integers(-half, half, size=(n, d))
    x = ((codes + 0.5) / half).astype(np.float32)
    x[:, 0] = 1.0
    cal = _identity_calibration(d, [b] * d, [1.0] * d)
    cal.quantizer = "midrise"
    rec, a16, code = aatc.encode(x, cal)
    assert np.all(a16.astype(np.float64) == 1.0)
    np.testing.assert_array_equal(code[:, 1:], codes[:, 1:])
    assert np.all(code[:, 0] == half - 1)
    expect = x.astype(np.float64)
    expect[:, 0] = 1.0 - 0.5 / half
    xh = aatc.decode_tokens(rec, a16, cal)
    np.testing.assert_array_equal(xh, expect)
    q = rng.standard_normal((2, d)).astype(np.float32)
    out = aatc.decode_attention(q, [cal], [cal], [rec], [a16], [rec], [a16], n)
    np.testing.assert_allclose(out, aatc.softmax_attention(q, expect, expect, 1 / np.sqrt(d)),
                               rtol=1e-13)
