"""Pins of the oracle's quantizer and packing (Sec. 3.3 Def. 2; Sec. 5.2; App. B)."""
import json
import os

import numpy as np
import pytest

from oracle import aatc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _f16(v):
    return np.asarray(v, dtype=np.float64).astype(np.float16)


def test_quantizer_worked_example_two_bits():
    g = _golden("quantizer_worked_example.json")["two_bit"]
    h = np.array([g["h"]], dtype=np.float32)
    bits = np.array(g["bits"])
    c, a16 = aatc.quantize(h, bits, _f16(g["s"]))
    assert float(a16[0]) == g["alpha"]
    assert c[0].tolist() == g["codes"]
    assert (c[0] % 4).tolist() == g["stored"]
    rec = aatc.pack_records(c, bits)
    assert rec[0].tobytes().hex() == g["record_bytes_hex"]
    hh = aatc.dequantize(c, a16, bits, _f16(g["s"]))
    np.testing.assert_allclose(hh[0], g["h_hat"], atol=0)
    np.testing.assert_array_equal(aatc.unpack_records(rec, bits), c)


def test_quantizer_worked_example_one_bit():
    g = _golden("quantizer_worked_example.json")["one_bit"]
    h = np.array([g["h"]], dtype=np.float32)
    bits = np.array(g["bits"])
    c, a16 = aatc.quantize(h, bits, _f16(g["s"]))
    assert c[0].tolist() == g["codes"]
    rec = aatc.pack_records(c, bits)
    assert (np.unpackbits(rec[0], bitorder="little")[:2]).tolist() == g["stored"]
    hh = aatc.dequantize(c, a16, bits, _f16(g["s"]))
    np.testing.assert_allclose(hh[0], g["h_hat"], atol=1e-3)   # alpha is stored as fp16


def _random_case(seed, n=4000, d=24):
    rng = np.random.default_rng(seed)
    bits = np.sort(rng.integers(0, 9, size=d))[::-1]
    s16 = _f16(rng.lognormal(0, 1, size=d))
    s16[bits == 0] = 0
    h = (rng.standard_normal((n, d)) * s16.astype(np.float64) *
         rng.uniform(0.3, 1.2, size=(n, 1))).astype(np.float32)
    return h, bits, s16


@pytest.mark.parametrize("seed", range(4))
def test_quantizer_error_within_half_step(seed):
    """|h - h^| <= Delta/2 inside the clipping range (Def. 2); the top code absorbs
    the overload, so clamped elements stay within one step (plus the fp16 rounding of
    alpha)."""
    h, bits, s16 = _random_case(seed)
    c, a16 = aatc.quantize(h, bits, s16)
    hh = aatc.dequantize(c, a16, bits, s16)
    keep = bits > 0
    s = s16.astype(np.float64)
    a = a16.astype(np.float64)
    delta = 2 * a[:, None] * s[None, :] * 2.0 ** (-bits[None, :].astype(float))
    err = np.abs(h.astype(np.float64) - hh)
    top = c == (1 << np.maximum(bits - 1, 0))[None, :] - 1
    inner = keep[None, :] & ~top
    assert np.all(err[inner] <= delta[inner] * (0.5 + 1e-5))
    alpha = np.max(np.abs(h[:, keep].astype(np.float64) / s[keep]), axis=1)
    slack = np.abs(alpha - a)[:, None] * s[None, :]
    over = keep[None, :] & top
    assert np.all(err[over] <= (delta + slack)[over] * (1 + 1e-5))
    assert np.all(hh[:, ~keep] == 0)
    half = np.where(keep, 1 << np.maximum(bits - 1, 0), 0)[None, :]
    assert np.all((c >= -half) & (c < np.maximum(half, 1)))


def test_quantizer_is_round_half_up_of_the_fp32_ratio():
    """code = floor(x + 1/2) exactly, including the ties x = k + 1/2."""
    bits = np.array([4])
    s16 = _f16([1.0])
    # alpha = 1 (first token element), x = h * 8 exactly representable.
    vals = np.array([-8.0, -7.5, -2.5, -0.5, 0.0, 0.5, 1.5, 2.5, 7.49, 7.5, 8.0]) / 8.0
    h = np.stack([np.full_like(vals, 1.0), vals], axis=1).astype(np.float32)
    c, _ = aatc.quantize(h, np.array([4, 4]), _f16([1.0, 1.0]))
    codes = c[:, 1]
    assert codes.tolist() == [-8, -7, -2, 0, 0, 1, 2, 3, 7, 7, 7]


def test_noise_variance_closed_form_and_decay_with_bits():
    """Uniform inputs on [-alpha, alpha]: the Sec. 5.2 quantizer has MSE
    Delta^2/12 * (1 + 3 * 2^-b).  The extra term comes from the top cell
    [alpha - Delta/2, alpha], which the clamp maps one step down; integrating the
    squared error over the 2^b - 1 regular cells, the bottom half cell and that top
    cell gives the formula.  It tends to the Delta^2/12 of the noise model (App. B,
    eq. noise-model) and falls ~4x per bit (Sec. 3.1)."""
    rng = np.random.default_rng(9)
    n = 400000
    for b in range(1, 17):
        h = np.stack([np.ones(n), rng.uniform(-1, 1, n)], axis=1).astype(np.float32)
        bits = np.array([b, b])
        c, a16 = aatc.quantize(h, bits, _f16([1.0, 1.0]))
        hh = aatc.dequantize(c, a16, bits, _f16([1.0, 1.0]))
        mse = np.mean((h[:, 1].astype(np.float64) - hh[:, 1]) ** 2)
        delta = 2.0 ** (1 - b)
        assert mse == pytest.approx(delta ** 2 / 12 * (1 + 3 * 2.0 ** -b), rel=0.01)


def test_power_of_two_rescaling_invariance():
    """Scaling a channel and its scale by 2^k leaves every code unchanged (App. B:
    per-channel rescaling of the transform does not matter)."""
    h, bits, s16 = _random_case(11)
    k = np.random.default_rng(0).integers(-3, 4, size=bits.size)
    h2 = np.ldexp(h, k[None, :]).astype(np.float32)
    s2 = np.ldexp(s16.astype(np.float32), k).astype(np.float16)
    u1, a1 = aatc.quantize(h, bits, s16)
    u2, a2 = aatc.quantize(h2, bits, s2)
    np.testing.assert_array_equal(u1, u2)
    np.testing.assert_array_equal(a1, a2)


def test_zero_and_saturating_tokens():
    bits = np.array([3, 2, 0])
    s16 = _f16([1.0, 0.5, 0])
    h = np.array([[0, 0, 5], [1e6, -3e5, 0]], dtype=np.float32)
    c, a16 = aatc.quantize(h, bits, s16)
    assert c[0].tolist() == [0, 0, 0] and float(a16[0]) == 0.0
    assert float(a16[1]) == 65504.0
    hh = aatc.dequantize(c, a16, bits, s16)
    assert np.all(hh[0] == 0)


def test_record_roundtrip_and_padding():
    rng = np.random.default_rng(12)
    bits = np.sort(rng.integers(0, 9, size=128))[::-1]
    half = np.where(bits > 0, 1 << np.maximum(bits - 1, 0), 0)
    c = rng.integers(-128, 128, size=(70, 128))
    c = np.clip(c, -half[None, :], np.maximum(half - 1, 0)[None, :])
    rec = aatc.pack_records(c, bits)
    budget = int(bits.sum())
    assert rec.shape == (70, 4 * ((budget + 31) // 32))
    np.testing.assert_array_equal(aatc.unpack_records(rec, bits), c)
    pad = np.unpackbits(rec, axis=1, bitorder="little")[:, budget:]
    assert not pad.any()


def test_tile_layout_single_bit():
    """One set bit (token 64*1 + 37, record bit 13) lands at word (1, 13, 1), bit 10:
    t = 37 = 16*2 + 4*1 + 1, so W = 2 // 2 = 1 and p = 8*1 + 2*1 + 2 % 2 = 10."""
    rbytes = 8
    rec = np.zeros((128, rbytes), dtype=np.uint8)
    rec[64 + 37, 13 // 8] = 1 << (13 % 8)
    tiles = aatc.records_to_tiles(rec)
    assert tiles.shape == (2, 64 * rbytes)
    words = tiles.view("<u4").reshape(2, 8 * rbytes, 2)
    nz = np.argwhere(words)
    assert nz.tolist() == [[1, 13, 1]]
    assert words[1, 13, 1] == 1 << 10
    np.testing.assert_array_equal(aatc.tiles_to_records(tiles, rbytes), rec)


def test_tile_layout_is_a_permutation_of_tokens():
    """Each token of a tile owns exactly one bit position per record bit."""
    rbytes = 4
    for t in range(64):
        rec = np.zeros((64, rbytes), dtype=np.uint8)
        rec[t, 0] = 1
        words = aatc.records_to_tiles(rec).view("<u4").reshape(8 * rbytes, 2)
        assert np.count_nonzero(words) == 1 and bin(int(words.sum())).count("1") == 1


def test_tile_roundtrip_random():
    rng = np.random.default_rng(13)
    rec = rng.integers(0, 256, size=(192, 44)).astype(np.uint8)
    np.testing.assert_array_equal(aatc.tiles_to_records(aatc.records_to_tiles(rec), 44), rec)


def test_compression_arithmetic_matches_paper():
    """Sec. 6 / Table 2: 2.75 bits per element is the 5.82x point, and 1.07 GB of
    FP16 cache becomes ~184 MB (the packed payload; scales and the fp16 window are
    the rest)."""
    g = _golden("paper_compression.json")
    assert g["fp16_bits"] / g["avg_bits_main"] == pytest.approx(g["compression_main"], abs=5e-3)
    assert g["llama_fp16_bytes"] / g["compression_main"] == pytest.approx(
        g["llama_aatc_bytes"], rel=5e-3)
    per_token = g["llama_layers"] * g["llama_kv_heads"] * g["head_dim"] * 2 * 2
    assert g["llama_fp16_bytes"] / per_token == pytest.approx(8192, rel=0.02)


# ---------------------------------------------------------------------------------------
# The midrise reading (symmetric levels (code + 1/2) Delta; Sec. 4 remark, App. B noise
# model) and widths up to 16 bits (App. E).
# ---------------------------------------------------------------------------------------
def test_midrise_worked_example_two_bits():
    g = _golden("quantizer_midrise_example.json")["two_bit"]
    h = np.array([g["h"]], dtype=np.float32)
    bits = np.array(g["bits"])
    c, a16 = aatc.quantize(h, bits, _f16(g["s"]), "midrise")
    assert float(a16[0]) == g["alpha"]
    assert c[0].tolist() == g["codes"]
    c_mt, _ = aatc.quantize(h, bits, _f16(g["s"]), "midtread")
    assert c_mt[0].tolist() == g["codes_midtread"]
    rec = aatc.pack_records(c, bits)
    assert rec[0].tobytes().hex() == g["record_bytes_hex"]
    hh = aatc.dequantize(c, a16, bits, _f16(g["s"]), "midrise")
    np.testing.assert_allclose(hh[0], g["h_hat"], atol=0)


def test_midrise_worked_example_one_bit():
    g = _golden("quantizer_midrise_example.json")["one_bit"]
    h = np.array([g["h"]], dtype=np.float32)
    bits = np.array(g["bits"])
    c, a16 = aatc.quantize(h, bits, _f16(g["s"]), "midrise")
    assert c[0].tolist() == g["codes"]
    rec = aatc.pack_records(c, bits)
    assert (np.unpackbits(rec[0], bitorder="little")[:2]).tolist() == g["stored"]
    hh = aatc.dequantize(c, a16, bits, _f16(g["s"]), "midrise")
    np.testing.assert_allclose(hh[0], g["h_hat"], atol=0)


def _random_case16(seed, n=4000, d=24):
    rng = np.random.default_rng(seed)
    bits = np.sort(rng.integers(0, 17, size=d))[::-1]
    s16 = _f16(rng.lognormal(0, 1, size=d))
    s16[bits == 0] = 0
    h = (rng.standard_normal((n, d)) * s16.astype(np.float64) *
         rng.uniform(0.3, 1.2, size=(n, 1))).astype(np.float32)
    return h, bits, s16


@pytest.mark.parametrize("seed", range(4))
def test_midrise_error_within_half_step_everywhere(seed):
    """Midrise: |h - h^| <= Delta/2 for every element with |h / s| <= alpha16 (the top
    cell included: no overload, Sec. 4 remark); elements above alpha16 (the fp16 rounding
    of alpha) exceed it by at most that rounding.  Widths 0..16."""
    h, bits, s16 = _random_case16(seed)
    c, a16 = aatc.quantize(h, bits, s16, "midrise")
    hh = aatc.dequantize(c, a16, bits, s16, "midrise")
    keep = bits > 0
    s = s16.astype(np.float64)
    a = a16.astype(np.float64)
    delta = 2 * a[:, None] * s[None, :] * 2.0 ** (-bits[None, :].astype(float))
    err = np.abs(h.astype(np.float64) - hh)
    ratio = np.abs(h.astype(np.float64)) / np.where(s > 0, s, 1.0)[None, :]
    inside = keep[None, :] & (ratio <= a[:, None])
    # (the fp32 evaluation of r / alpha adds ~2^-23 relative to the position in the cell)
    tol = delta * 0.5 + a[:, None] * s[None, :] * 2.0 ** -20
    assert np.all(err[inside] <= tol[inside])
    over = keep[None, :] & ~inside
    slack = (ratio - a[:, None]) * s[None, :]
    assert np.all(err[over] <= (tol + slack)[over])
    assert np.all(hh[:, ~keep] == 0)
    half = np.where(keep, 1 << np.maximum(bits - 1, 0), 0)[None, :]
    assert np.all((c >= -half) & (c < np.maximum(half, 1)))


def test_midrise_levels_are_odd_and_b1_is_unbiased():
    """Midrise levels are symmetric: h -> -h maps the level to minus itself (floor(-x) =
    -floor(x) - 1 off the integers); at b = 1 the levels are +-alpha s / 2, so the mean
    error over symmetric inputs vanishes (the printed formula's {-alpha s, 0} does not)."""
    rng = np.random.default_rng(21)
    n = 200000
    for b in (1, 2, 3, 5, 8, 12, 16):
        v = rng.uniform(-1, 1, n)
        h = np.stack([np.ones(n), v, -v], axis=1).astype(np.float32)
        bits = np.array([b, b, b])
        s16 = _f16([1.0, 1.0, 1.0])
        c, a16 = aatc.quantize(h, bits, s16, "midrise")
        hh = aatc.dequantize(c, a16, bits, s16, "midrise")
        x = h[:, 1].astype(np.float64) * 2.0 ** (b - 1)
        off = x != np.floor(x)
        np.testing.assert_array_equal(hh[off, 1], -hh[off, 2])
    b = 1
    v = rng.uniform(-1, 1, n)
    h = np.stack([np.ones(n), v], axis=1).astype(np.float32)
    for kind, biased in (("midrise", False), ("midtread", True)):
        c, a16 = aatc.quantize(h, np.array([b, b]), _f16([1.0, 1.0]), kind)
        hh = aatc.dequantize(c, a16, np.array([b, b]), _f16([1.0, 1.0]), kind)
        mean_err = float(np.mean(hh[:, 1] - h[:, 1]))
        if biased:
            assert mean_err < -0.2               # levels {-1, 0}: mean error -1/2
        else:
            assert abs(mean_err) < 5e-3


def test_midrise_noise_variance_is_delta_squared_over_12():
    """Uniform inputs on [-alpha, alpha]: every midrise cell has width Delta and the level
    at its centre, so MSE = Delta^2 / 12 exactly in the limit (App. B eq. noise-model),
    for b = 1..16; it falls 4x per bit (Sec. 3.1)."""
    rng = np.random.default_rng(10)
    n = 400000
    prev = None
    for b in range(1, 17):
        h = np.stack([np.ones(n), rng.uniform(-1, 1, n)], axis=1).astype(np.float32)
        bits = np.array([b, b])
        c, a16 = aatc.quantize(h, bits, _f16([1.0, 1.0]), "midrise")
        hh = aatc.dequantize(c, a16, bits, _f16([1.0, 1.0]), "midrise")
        mse = np.mean((h[:, 1].astype(np.float64) - hh[:, 1]) ** 2)
        delta = 2.0 ** (1 - b)
        assert mse == pytest.approx(delta ** 2 / 12, rel=0.01)
        if prev is not None:
            assert mse / prev == pytest.approx(0.25, rel=0.03)
        prev = mse


def test_sixteen_bit_records_roundtrip():
    """Widths up to 16 (App. E): fields straddle words; the LSB-first bit string round
    trips and the two's complement pattern of each code is what is stored."""
    rng = np.random.default_rng(14)
    bits = np.sort(rng.integers(0, 17, size=128))[::-1]
    half = np.where(bits > 0, 1 << np.maximum(bits - 1, 0), 0)
    c = rng.integers(-32768, 32768, size=(50, 128))
    c = np.clip(c, -half[None, :], np.maximum(half - 1, 0)[None, :])
    rec = aatc.pack_records(c, bits)
    np.testing.assert_array_equal(aatc.unpack_records(rec, bits), c)
    # the first channel's field, read back by hand from the bit string
    b0 = int(bits[0])
    flat = np.unpackbits(rec, axis=1, bitorder="little")
    field = (flat[:, :b0].astype(np.int64) << np.arange(b0)).sum(axis=1)
    np.testing.assert_array_equal(field, c[:, 0] & ((1 << b0) - 1))


def test_allocation_with_sixteen_bit_cap():
    """b_max = 16: the budget is spent exactly, no width exceeds 16, a dominant channel
    takes more than 8 bits when its weighted variance calls for it, and the greedy result
    attains the minimum of sum_c W_c 4^-b_c over every allocation (brute force)."""
    import itertools
    from oracle.aatc import allocate_bits, allocation_objective
    w = np.array([4.0 ** 12, 1.0, 0.5, 0.25])
    b = allocate_bits(w, 20, 16)
    assert int(b.sum()) == 20 and b.max() <= 16 and b[0] > 8
    best = min(allocation_objective(w, np.array(c))
               for c in itertools.product(range(17), repeat=4) if sum(c) == 20)
    assert allocation_objective(w, b) == pytest.approx(best, rel=1e-12)
    # worked by hand: channel 0 wins every bit until 4^(12 - b0) reaches the others'
    # gains, then the ties go to the lowest index: (15, 2, 2, 1)
    assert b.tolist() == [15, 2, 2, 1]
