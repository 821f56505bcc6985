"""Pins of the oracle's full-precision segment (Sec. 6 experimental setup; App. E "AATC":
the first s = 4 tokens and a recent window of w = 128 tokens at input precision, the oldest
16 window tokens quantized whenever the window is full)."""
import numpy as np
import pytest

import paper_2608_14191_amd as P
from oracle import aatc as ora


def _closed_form(n, s, w, step):
    m = max(n - s, 0)
    return 0 if m < w else step * ((m - w) // step + 1)


@pytest.mark.parametrize("s,w,step", [(4, 128, 16), (0, 8, 8), (2, 10, 3), (4, 32, 32), (1, 1, 1)])
def test_policy_matches_closed_form(s, w, step):
    """The token-by-token simulation against the closed form of the flush count, and the
    index sets it returns."""
    for n in range(0, 5 * w + 40):
        comp, seg = ora.segment_split(n, s, w, step)
        c = _closed_form(n, s, w, step)
        assert comp.size == c, (n, comp.size, c)
        np.testing.assert_array_equal(comp, np.arange(min(s, n), min(s, n) + c))
        np.testing.assert_array_equal(np.sort(np.concatenate([comp, seg])), np.arange(n))
        win = n - min(s, n) - c
        assert win < w and (c == 0 or win >= w - step)


def test_policy_paper_operating_point():
    """s = 4, w = 128, step 16: the first flush comes with token 132 (the window is full),
    leaving 112 window tokens; 16 tokens later the next."""
    assert ora.segment_split(131)[0].size == 0
    comp, seg = ora.segment_split(132)
    np.testing.assert_array_equal(comp, np.arange(4, 20))
    assert seg.size == 116 and seg[:4].tolist() == [0, 1, 2, 3] and seg[4] == 20
    assert ora.segment_split(147)[0].size == 16 and ora.segment_split(148)[0].size == 32


def test_host_policy_matches_oracle():
    for n in list(range(0, 400)) + [4096, 32768 + 7]:
        c, g = P.aatc_segment_counts(n)
        comp, seg = ora.segment_split(n)
        assert (c, g) == (comp.size, seg.size), n
    with pytest.raises(P.AatcError):
        P.aatc_segment_counts(10, 4, 16, 17)


def _cal_identity(d):
    bits = np.full(d, 8, dtype=np.int64)
    return ora.Calibration(d=d, budget=8 * d, record_bytes=d, d_active=d, bits=bits,
                           perm=np.arange(d), T64=np.eye(d), T32=np.eye(d, dtype=np.float32),
                           s16=np.ones(d, dtype=np.float16), sigma2=np.ones(d),
                           weight=np.ones(d), bits_eig=bits)


def test_attention_with_segment_special_cases():
    rng = np.random.default_rng(21)
    d, n = 16, 40
    cal = _cal_identity(d)
    k = rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    q = rng.standard_normal((2, d)).astype(np.float32)
    rk, ak, _ = ora.encode(k[:25].astype(np.float32), cal)
    rv, av, _ = ora.encode(v[:25].astype(np.float32), cal)
    # all tokens in the segment: plain softmax attention (and torch's, on the CPU)
    o_all = ora.attention_with_segment(q, [cal], [cal], [rk], [ak], [rv], [av], 0, [k], [v])
    np.testing.assert_allclose(o_all, ora.softmax_attention(q, k, v, d ** -0.5), rtol=1e-12)
    import torch
    ref = torch.nn.functional.scaled_dot_product_attention(         # (batch, heads, L, d)
        torch.from_numpy(q.astype(np.float64))[None, None], torch.from_numpy(k)[None, None],
        torch.from_numpy(v)[None, None])
    np.testing.assert_allclose(o_all, ref[0, 0].numpy(), rtol=1e-10)
    # an empty segment: the compressed-cache attention
    o_c = ora.attention_with_segment(q, [cal], [cal], [rk], [ak], [rv], [av], 25,
                                     [np.zeros((0, d))], [np.zeros((0, d))])
    np.testing.assert_allclose(o_c, ora.decode_attention(q, [cal], [cal], [rk], [ak], [rv], [av], 25),
                               rtol=1e-12)
    # the segment's order does not matter
    perm = rng.permutation(15)
    o1 = ora.attention_with_segment(q, [cal], [cal], [rk], [ak], [rv], [av], 25, [k[25:]], [v[25:]])
    o2 = ora.attention_with_segment(q, [cal], [cal], [rk], [ak], [rv], [av], 25,
                                    [k[25:][perm]], [v[25:][perm]])
    np.testing.assert_allclose(o1, o2, rtol=1e-12)
    # and it is the attention over the union of decoded and raw tokens
    kh = ora.decode_tokens(rk, ak, cal)
    vh = ora.decode_tokens(rv, av, cal)
    np.testing.assert_allclose(o1, ora.softmax_attention(q, np.concatenate([kh, k[25:]]),
                                                         np.concatenate([vh, v[25:]]), d ** -0.5),
                               rtol=1e-12)
