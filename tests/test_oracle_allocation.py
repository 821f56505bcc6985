"""Pins of the oracle's bit allocation (Sec. 3.1 eq. bit-allocation; Sec. 5.2; Alg. 1)."""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import aatc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_rwf_closed_form_worked_example():
    g = _golden("rwf_worked_example.json")
    lam, b = aatc.rwf_continuous(np.array(g["sigma2"]), g["avg_bits"])
    assert np.log2(lam) == pytest.approx(g["log2_water_level"], abs=1e-12)
    np.testing.assert_allclose(b, g["bits"], atol=1e-12)
    # Every retained coefficient sits at distortion lambda; dropped ones keep sigma^2.
    dist = np.array(g["sigma2"]) * 2.0 ** (-2 * b)
    np.testing.assert_allclose(dist, np.minimum(g["sigma2"], lam), rtol=1e-12)


@pytest.mark.parametrize("seed", range(5))
def test_rwf_continuous_properties(seed):
    rng = np.random.default_rng(seed)
    var = rng.lognormal(0, 2, size=16)
    avg = rng.uniform(0.5, 4)
    lam, b = aatc.rwf_continuous(var, avg)
    assert b.mean() == pytest.approx(avg, rel=1e-12)
    on = b > 0
    np.testing.assert_allclose(var[on] * 2.0 ** (-2 * b[on]), lam, rtol=1e-10)
    assert np.all(var[~on] <= lam * (1 + 1e-12))


def test_greedy_worked_example():
    g = _golden("rwf_worked_example.json")["integer"]
    w = np.array(_golden("rwf_worked_example.json")["sigma2"])
    b = aatc.allocate_bits(w, g["budget"], 8)
    assert b.tolist() == g["greedy_bits"]
    assert aatc.allocation_objective(w, b) == pytest.approx(g["optimum"], abs=1e-15)
    for other in g["other_optima"]:
        assert aatc.allocation_objective(w, np.array(other)) == pytest.approx(g["optimum"])


def _brute_force(w, budget, b_max):
    best = np.inf
    for bits in itertools.product(range(b_max + 1), repeat=w.size):
        if sum(bits) == budget:
            best = min(best, aatc.allocation_objective(w, np.array(bits)))
    return best


@pytest.mark.parametrize("seed", range(12))
def test_greedy_is_optimal_small(seed):
    rng = np.random.default_rng(100 + seed)
    d = int(rng.integers(2, 7))
    b_max = int(rng.integers(1, 5))
    budget = int(rng.integers(0, d * b_max + 1))
    w = rng.lognormal(0, 3, size=d)
    if seed % 3 == 0:          # exact ties
        w[1] = w[0]
    b = aatc.allocate_bits(w, budget, b_max)
    assert b.sum() == budget and b.min() >= 0 and b.max() <= b_max
    assert aatc.allocation_objective(w, b) == pytest.approx(_brute_force(w, budget, b_max),
                                                            rel=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_greedy_exchange_optimality(seed):
    """No single bit moved between two channels lowers the objective (d = 128)."""
    rng = np.random.default_rng(seed)
    w = rng.lognormal(0, 2, size=128)
    budget = 352
    b = aatc.allocate_bits(w, budget, 8)
    assert b.sum() == budget
    gain_add = np.where(b < 8, 0.75 * w * 4.0 ** (-b), -np.inf)       # best bit to add
    loss_del = np.where(b > 0, 3.0 * w * 4.0 ** (-b), np.inf)          # cost of removing one
    assert gain_add.max() <= loss_del.min() * (1 + 1e-12)


def test_budget_bounds():
    w = np.ones(4)
    assert aatc.allocate_bits(w, 32, 8).tolist() == [8, 8, 8, 8]
    with pytest.raises(ValueError):
        aatc.allocate_bits(w, 33, 8)
    assert aatc.allocate_bits(w, 0, 8).tolist() == [0, 0, 0, 0]


def test_integer_close_to_continuous():
    """Unclamped integer widths stay within one bit of the continuous optimum."""
    rng = np.random.default_rng(7)
    w = np.sort(rng.lognormal(0, 1.5, size=64))[::-1]
    avg = 2.75
    lam, bc = aatc.rwf_continuous(w, avg)
    bi = aatc.allocate_bits(w, int(round(avg * 64)), 16)
    assert np.all(np.abs(bi - bc) <= 1.0 + 1e-9)


def test_calibration_budget_and_storage_order():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2048, 128)) * (np.arange(1, 129) ** -0.75)
    cal = aatc.calibrate(x, 2.75)
    assert cal.bits.sum() == cal.budget == 352
    assert cal.record_bytes == 44
    assert np.all(np.diff(cal.bits) <= 0)                   # widest first
    assert sorted(cal.perm.tolist()) == list(range(128))
    np.testing.assert_array_equal(cal.bits, cal.bits_eig[cal.perm])
    assert np.all(cal.s16[cal.bits == 0] == 0)
    assert np.all(cal.s16[cal.bits > 0] > 0)


def test_channel_scale_is_99th_percentile_of_magnitude():
    """s_c = 99th percentile of |h_c| over calibration tokens (Sec. 5.2), with linear
    interpolation between order statistics, rounded to fp16.  Disjoint row blocks give
    an exactly diagonal covariance, so h_c is column c itself."""
    d, m = 4, 100
    x = np.zeros((d * m, d))
    for c in range(d):
        x[c * m:(c + 1) * m, c] = np.arange(1, m + 1) * 2.0 ** -c * (-1) ** np.arange(m)
    cal = aatc.calibrate(x, 4.0)
    assert cal.perm.tolist() == [0, 1, 2, 3] and np.all(cal.bits > 0)
    # sorted |h_c|: 300 zeros, then 1..100 (x 2^-c); position 0.99 * 399 = 395.01
    for c in range(d):
        assert float(cal.s16[c]) == float(np.float16(96.01 * 2.0 ** -c))


# ---- one budget over all layers (Sec. 5.2; App. E's normalization and protected layers)

def test_global_pool_is_optimal_brute_force():
    """Layers whose two channels have equal variance are normalized to (1, 1) whatever
    their scale, so the pool's objective is sum w_c 4^-b_c; the greedy over all layers
    reaches the minimum of every allocation of the budget (enumerated)."""
    import itertools
    s2 = np.array([[0.3, 0.3], [7.0, 7.0], [1e-3, 1e-3]])
    w = np.array([[5.0, 0.25], [1.0, 3.0], [0.5, 9.0]])
    b_max = 3
    for avg in (0.5, 1.0, 1.5, 2.0):
        got = aatc.allocate_global(s2, w, avg, b_max, n_protect=0)
        total = int(np.floor(avg * 6 + 0.5))
        assert got.sum() == total
        best = min(float(np.sum(w.ravel() * 4.0 ** -np.array(b)))
                   for b in itertools.product(range(b_max + 1), repeat=6) if sum(b) == total)
        assert np.sum(w * 4.0 ** -got) == pytest.approx(best, rel=1e-15)


def test_global_single_layer_is_the_per_head_allocation():
    """With one unprotected layer the per-layer scale is a common factor, which the
    greedy's decisions do not see: the widths are those of allocate_bits on w sigma2."""
    rng = np.random.default_rng(11)
    s2, w = rng.gamma(0.7, size=(1, 64)), rng.gamma(1.5, size=(1, 64))
    for norm in (False, True):
        got = aatc.allocate_global(s2, w, 2.75, 8, n_protect=0, normalize_weight=norm)
        np.testing.assert_array_equal(got[0], aatc.allocate_bits(w[0] * s2[0], 176, 8))


def test_global_layer_scale_is_removed():
    """Scaling one layer's variances (and, when normalized, its weights) by a power of
    two leaves every width unchanged; identical layers at different scales get
    identical widths."""
    rng = np.random.default_rng(5)
    s2, w = rng.gamma(0.5, size=(6, 32)), rng.gamma(1.0, size=(6, 32))
    base = aatc.allocate_global(s2, w, 2.0, 8, n_protect=2, protect_extra=1,
                               normalize_weight=True)
    k = np.ldexp(1.0, np.array([-12, 3, 0, 7, -2, 20]))[:, None]
    j = np.ldexp(1.0, np.array([4, -6, 1, 0, 9, -3]))[:, None]
    np.testing.assert_array_equal(
        aatc.allocate_global(s2 * k, w * j, 2.0, 8, n_protect=2, protect_extra=1,
                            normalize_weight=True), base)
    same = np.repeat(s2[:1], 4, axis=0) * np.ldexp(1.0, np.array([-10, 0, 5, -3]))[:, None]
    got = aatc.allocate_global(same, None, 2.5, 8, n_protect=0)
    assert np.all(got == got[0])


def test_global_budgets_and_protected_layers():
    rng = np.random.default_rng(8)
    s2, w = rng.gamma(0.5, size=(7, 40)), rng.gamma(1.0, size=(7, 40))
    avg, m, L = 2.75, 40, 7
    got = aatc.allocate_global(s2, w, avg, 8, n_protect=3, protect_extra=1, normalize_weight=True)
    assert got.min() >= 0 and got.max() <= 8
    assert got.sum() == int(np.floor(avg * m * L + 0.5))
    for layer in range(3):
        assert got[layer].sum() == int(np.floor((avg + 1) * m + 0.5))
        # a protected layer is allocated on its own channels
        np.testing.assert_array_equal(got[layer], aatc.allocate_bits(w[layer] * s2[layer],
                                                                    int(got[layer].sum()), 8))
    # all layers protected: the total plays no part
    allp = aatc.allocate_global(s2[:2], None, 2.0, 8, n_protect=3, protect_extra=1)
    assert list(allp.sum(axis=1)) == [120, 120]


def test_global_rejects_unmeetable_budgets():
    s2 = np.ones((4, 8))
    with pytest.raises(ValueError):     # protected layers take more than the total
        aatc.allocate_global(s2, None, 0.5, 8, n_protect=3, protect_extra=1)
    with pytest.raises(ValueError):     # the pool exceeds b_max per channel
        aatc.allocate_global(s2, None, 8.5, 8, n_protect=0)


def test_calibrate_with_given_bits_is_the_allocation():
    """The oracle's calibration with its own greedy widths passed in is the calibration
    itself; records padded to a larger size only add zero bytes."""
    rng = np.random.default_rng(41)
    x = rng.standard_normal((512, 128)) @ rng.standard_normal((128, 128))
    a = aatc.calibrate(x, 2.75)
    b = aatc.calibrate(x, 0.0, bits_eig=a.bits_eig)
    np.testing.assert_array_equal(a.bits, b.bits)
    np.testing.assert_array_equal(a.perm, b.perm)
    np.testing.assert_array_equal(a.s16, b.s16)
    assert (a.budget, a.record_bytes) == (b.budget, b.record_bytes) == (352, 44)
    c = aatc.calibrate(x, 0.0, bits_eig=a.bits_eig, record_bytes=64)
    xs = x[:20].astype(np.float32)
    ra, aa, _ = aatc.encode(xs, a)
    rc, ac, _ = aatc.encode(xs, c)
    assert rc.shape == (20, 64)
    np.testing.assert_array_equal(rc[:, :44], ra)
    assert not rc[:, 44:].any()
    np.testing.assert_array_equal(aa, ac)
