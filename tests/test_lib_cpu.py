"""Host-side checks of libaatc.so that need no GPU: exports, argument validation,
host calibration parity with the oracle, parameter packing."""
import ctypes
import os

import numpy as np
import pytest

import paper_2608_14191_amd as P
from kvsynth import workload
from oracle import aatc as ora

from helpers import abi_calibration

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "aatc.h")


def test_library_exports_every_declared_symbol():
    from paper_2608_14191_amd._lib import exported_symbols_declared_in_header
    names = exported_symbols_declared_in_header(HEADER)
    assert {"aatc_calibrate", "aatc_encode", "aatc_decode_attention",
            "aatc_append_decode_attention"} <= set(names)
    lib = P.library()
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    assert P.aatc_status_string(0) == "ok"
    assert "workspace" in P.aatc_status_string(5)


def _calib_cases():
    return [(1, 0, "k"), (1, 0, "v"), (2, 3, "k"), (2, 5, "v"), (3, 1, "k"), (5, 2, "k")]


@pytest.mark.parametrize("cfg,head,kind", _calib_cases())
def test_host_calibration_matches_oracle(cfg, head, kind):
    w = workload(cfg, n_tokens=64)
    x = w.calib(head, kind)
    avg = w.cfg["avg_bits"][0]
    qc = w.calib_queries(head) if (kind == "k" and w.cfg["query_weighted_k"]) else None
    g = w.group if qc is not None else 1
    c = P.aatc_calibrate(x, avg, q_calib=qc, q_group=g)
    o = ora.calibrate(x, avg, q_calib=qc, group=g)
    np.testing.assert_array_equal(c.bits_np, o.bits)
    np.testing.assert_array_equal(np.ctypeslib.as_array(c.perm), o.perm)
    np.testing.assert_array_equal(np.ctypeslib.as_array(c.bits_eig), o.bits_eig)
    np.testing.assert_array_equal(c.s16.view(np.uint16), o.s16.view(np.uint16))
    assert (c.budget_bits, c.record_bytes, c.d_active) == (o.budget, o.record_bytes, o.d_active)
    # the stored transform: on the 2^-22 grid on both sides; the eigensolvers differ by
    # ~1e-15, which moves an entry to the next grid point only at a rounding tie
    q = np.ldexp(c.T.astype(np.float64), 22)
    np.testing.assert_array_equal(q, np.rint(q))
    assert np.abs(c.T.astype(np.float64) - o.T32).max() <= 2.0 ** -22
    assert np.count_nonzero(c.T != o.T32) <= 2
    np.testing.assert_allclose(np.ctypeslib.as_array(c.sigma2), o.sigma2, rtol=1e-9,
                               atol=1e-12 * o.sigma2[0])
    np.testing.assert_allclose(np.ctypeslib.as_array(c.weight), o.weight, rtol=1e-9)


def test_host_calibration_value_weights_match_oracle():
    w = workload(2, n_tokens=64)
    x = w.calib(0, "v")
    w_o = np.random.default_rng(0).standard_normal((128, 96)).astype(np.float32)
    c = P.aatc_calibrate(x, 2.75, w_o=w_o)
    o = ora.calibrate(x, 2.75, w_o=w_o)
    np.testing.assert_array_equal(c.bits_np, o.bits)
    np.testing.assert_allclose(np.ctypeslib.as_array(c.weight), o.weight, rtol=1e-9)


def test_host_calibration_worked_rwf_example():
    """Diagonal covariance with variances 4, 1, 1/4, 1/16 repeated: the integer
    allocation follows the tie rule exactly (Sec. 5.2; see test_oracle_allocation)."""
    d = 128
    var = np.tile([4.0, 1.0, 0.25, 0.0625], d // 4) * np.repeat(4.0 ** -np.arange(32), 4)
    rng = np.random.default_rng(1)
    z, _ = np.linalg.qr(rng.standard_normal((512, d)))
    x = (z * np.sqrt(512) * np.sqrt(var)[None, :]).astype(np.float32)
    c = P.aatc_calibrate(x, 1.0)
    o = ora.calibrate(x, 1.0)
    np.testing.assert_array_equal(c.bits_np, o.bits)


@pytest.mark.parametrize("bad", ["d", "n", "bits", "pct", "both"])
def test_calibrate_validation(bad):
    x = np.zeros((16, 128), dtype=np.float32)
    kwargs = dict(avg_bits=2.0)
    if bad == "d":
        with pytest.raises(P.AatcError) as e:
            P.aatc_calibrate(np.zeros((16, 64), dtype=np.float32), 2.0)
        assert e.value.status == 2
        return
    if bad == "n":
        x = x[:1]
    if bad == "bits":
        kwargs = dict(avg_bits=9.0)
    if bad == "pct":
        kwargs = dict(avg_bits=2.0, percentile=1.5)
    if bad == "both":
        kwargs = dict(avg_bits=2.0, q_calib=np.ones((4, 128), np.float32),
                      w_o=np.ones((128, 4), np.float32))
    with pytest.raises(P.AatcError) as e:
        P.aatc_calibrate(x, **kwargs)
    assert e.value.status == 1


def test_calibrate_rejects_non_finite():
    x = np.ones((16, 128), dtype=np.float32)
    x[3, 7] = np.nan
    with pytest.raises(P.AatcError) as e:
        P.aatc_calibrate(x, 2.0)
    assert e.value.status == 3


def test_params_pack_validation():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((256, 128)).astype(np.float32)
    a = abi_calibration(ora.calibrate(x, 2.0))
    b = abi_calibration(ora.calibrate(x, 3.0))
    P.aatc_params_pack([a, a])
    with pytest.raises(P.AatcError):
        P.aatc_params_pack([a, b])                      # budgets differ
    bad = abi_calibration(ora.calibrate(x, 2.0))
    bad.bits[5], bad.bits[6] = bad.bits[6], bad.bits[5] + 1   # not non-increasing
    with pytest.raises(P.AatcError):
        P.aatc_params_pack([bad])
    # the stored transform must lie on the 2^-22 grid with |T| <= 1
    off = abi_calibration(ora.calibrate(x, 2.0))
    off.transform[7] = off.transform[7] + 2.0 ** -25
    with pytest.raises(P.AatcError):
        P.aatc_params_pack([off])
    big = abi_calibration(ora.calibrate(x, 2.0))
    big.transform[3] = 1.5
    with pytest.raises(P.AatcError):
        P.aatc_params_pack([big])


def test_params_pack_bf16_pair_copy_of_transform():
    """The parameter block's bf16-pair copy of T (the merge's matrix-core operands):
    unit ((4 w + kk) 2 + t) 64 + l holds term t of T[16 w + l % 16][32 kk + 8 (l / 16) ..
    + 7]; the first term is T rounded to bf16 (nearest even), the second the remainder
    rounded likewise, so the pair is within 2^-16 |T| + 2^-133 of T."""
    rng = np.random.default_rng(3)
    x = rng.standard_normal((512, 128)).astype(np.float32)
    cals = [abi_calibration(ora.calibrate(x + 0.1 * h, 2.75)) for h in range(2)]
    blk = P.aatc_params_pack(cals)
    hp_bytes = (P.aatc_params_bytes(2) - 256) // 2
    for h in range(2):
        base = 256 + h * hp_bytes
        T = np.frombuffer(blk, dtype=np.float32, count=128 * 128, offset=base).reshape(128, 128)
        assert np.array_equal(T, np.asarray(cals[h].transform, dtype=np.float32).reshape(128, 128))
        tm = np.frombuffer(blk, dtype=np.uint16, count=2 * 128 * 128,
                           offset=base + 128 * 128 * 4).reshape(8, 4, 2, 64, 8)
        def as_f32(b):
            return (b.astype(np.uint32) << 16).view(np.float32)
        hi = np.empty((128, 128), np.float32)
        lo = np.empty((128, 128), np.float32)
        for w in range(8):
            for kk in range(4):
                for l in range(64):
                    j, c0 = 16 * w + l % 16, 32 * kk + 8 * (l // 16)
                    hi[j, c0:c0 + 8] = as_f32(tm[w, kk, 0, l])
                    lo[j, c0:c0 + 8] = as_f32(tm[w, kk, 1, l])
        # the first term: nearest bf16 (ties even), by a direct search of the neighbours
        u = T.view(np.uint32)
        down = (u & 0xffff0000).view(np.float32)
        up = ((u & 0xffff0000) + 0x10000).astype(np.uint32).view(np.float32)
        d_down, d_up = np.abs(T - down), np.abs(up - T)
        even_down = ((u >> 16) & 1) == 0
        want = np.where((d_down < d_up) | ((d_down == d_up) & even_down), down, up)
        assert np.array_equal(hi, want)
        assert np.all(np.abs(T.astype(np.float64) - hi - lo) <= 2.0 ** -16 * np.abs(T) + 2.0 ** -133)


def _fake(addr=4096):
    return ctypes.c_void_p(addr)


def test_encode_and_decode_validate_before_launch():
    """Invalid requests are rejected on the host; nothing reaches the device."""
    L = P.library()
    p = _fake()
    # d != 128
    assert L.aatc_encode(p, 1, 64, p, 0, 1, 128, 0, p, p, 64, 0, None) == 2
    # pos + n_tok > cap
    assert L.aatc_encode(p, 1, 128, p, 0, 10, 128, 0, p, p, 64, 60, None) == 1
    # tiles need cap % 64 == 0
    assert L.aatc_encode(p, 1, 128, p, 0, 1, 128, 1, p, p, 100, 0, None) == 1
    # null codes
    assert L.aatc_encode(p, 1, 128, p, 0, 1, 128, 0, None, p, 64, 0, None) == 1
    # misaligned codes
    assert L.aatc_encode(p, 1, 128, p, 0, 1, 128, 0, _fake(4097), p, 64, 0, None) == 1
    # n_tok = 0 is a no-op
    assert L.aatc_encode(p, 1, 128, p, 0, 0, 128, 0, p, p, 64, 0, None) == 0
    ws = P.aatc_decode_workspace_bytes(1, 32, 8, 4096)
    assert ws > 0
    args = [p, p, 1, 32, 8, 128, p, 1, p, p, p, p, p, 4096, 44, 44, 0.088, p, p, ws, None]
    bad = list(args); bad[4] = 6                     # 32 % 6 != 0
    assert L.aatc_decode_attention(*bad) == 1
    bad = list(args); bad[13] = 100                  # cap not a multiple of 64
    assert L.aatc_decode_attention(*bad) == 1
    bad = list(args); bad[14] = 42                   # record size not a multiple of 4
    assert L.aatc_decode_attention(*bad) == 1
    bad = list(args); bad[15] = 260                  # record larger than 2048 bits (16 x 128)
    assert L.aatc_decode_attention(*bad) == 1
    bad = list(args); bad[19] = ws - 1               # workspace too small
    assert L.aatc_decode_attention(*bad) == 5
    bad = list(args); bad[5] = 64
    assert L.aatc_decode_attention(*bad) == 2


def test_append_decode_validates_before_launch():
    """The fused append + decode entry point checks the decode arguments and the new
    tokens on the host."""
    L = P.library()
    p = _fake()
    ws = P.aatc_decode_workspace_bytes(1, 32, 8, 4096)
    args = [p, p, 1, 32, 8, 128, p, 1, p, p, 1, p, p, p, p, p, 4096, 44, 44, 0.088, p, p, ws,
            None]
    bad = list(args); bad[8] = None                  # no new keys
    assert L.aatc_append_decode_attention(*bad) == 1
    bad = list(args); bad[10] = 2                    # f16 tokens are not accepted
    assert L.aatc_append_decode_attention(*bad) == 1
    bad = list(args); bad[9] = _fake(4097)           # misaligned bf16 values
    assert L.aatc_append_decode_attention(*bad) == 1
    bad = list(args); bad[16] = 100                  # cap not a multiple of 64
    assert L.aatc_append_decode_attention(*bad) == 1
    bad = list(args); bad[22] = ws - 1               # workspace too small
    assert L.aatc_append_decode_attention(*bad) == 5


def test_append_decode_binding_rejects_mixed_token_dtypes():
    """The binding raises the library's error type (status AATC_E_INVALID) when the new
    key and value tokens have different dtypes, before any pointer is touched."""
    import torch
    xk = torch.zeros((1, 8, 128), dtype=torch.bfloat16)
    xv = torch.zeros((1, 8, 128), dtype=torch.float32)
    with pytest.raises(P.AatcError) as e:
        P.aatc_append_decode_attention(None, None, 1, 32, 8, None, xk, xv, None, None, None,
                                       None, None, 64, 44, 44, 0.088, None, None)
    assert e.value.status == 1


def test_noalloc_entry_point_rejects_oversized_requests():
    """The static workspace takes at most 256 (sequence, KV head) rows and 32 MiB; larger
    requests return AATC_E_WORKSPACE before any launch (host checks only)."""
    L = P.library()
    p = _fake()
    args = [p, p, 40, 32, 8, 128, p, 1, p, p, 1, p, p, p, p, p, 4096, 44, 44, 0.088, p, None]
    assert L.aatc_append_decode_attention_noalloc(*args) == 5        # 320 rows
    args = [p, p, 32, 32, 8, 128, p, 1, p, p, 1, p, p, p, p, p, 1 << 20, 44, 44, 0.088, p, None]
    assert L.aatc_append_decode_attention_noalloc(*args) == 5        # partials beyond 32 MiB
    bad = [p, p, 1, 32, 8, 128, p, 1, None, p, 1, p, p, p, p, p, 4096, 44, 44, 0.088, p, None]
    assert L.aatc_append_decode_attention_noalloc(*bad) == 1         # no new keys


def test_calibrate_bits_matches_oracle_and_pads_records():
    """aatc_calibrate_bits (widths given, eigen order) against the oracle's calibration
    with the same widths; a padded record size is kept; params_pack takes heads with
    different budgets that share one record size, and rejects record sizes that differ."""
    w = workload(2, n_tokens=64)
    rng = np.random.default_rng(31)
    cals = []
    for head, budget in ((0, 300), (1, 352), (2, 290)):
        x = w.calib(head, "k")
        bits = ora.allocate_bits(np.arange(128, 0, -1) ** 1.5 * rng.uniform(0.5, 1.5, 128),
                                 budget, 8)
        c = P.aatc_calibrate_bits(x, bits, record_bytes=44)
        o = ora.calibrate(x, 0.0, bits_eig=bits, record_bytes=44)
        np.testing.assert_array_equal(np.ctypeslib.as_array(c.bits_eig), bits)
        np.testing.assert_array_equal(c.bits_np, o.bits)
        np.testing.assert_array_equal(np.ctypeslib.as_array(c.perm), o.perm)
        np.testing.assert_array_equal(c.s16.view(np.uint16), o.s16.view(np.uint16))
        assert (c.budget_bits, c.record_bytes, c.d_active) == (o.budget, 44, o.d_active) == \
            (budget, 44, int(np.count_nonzero(bits)))
        cals.append(c)
    P.aatc_params_pack(cals)                                  # budgets 300, 352, 290
    with pytest.raises(P.AatcError):
        P.aatc_calibrate_bits(w.calib(0, "k"), bits, record_bytes=32)   # 290 bits > 32 B
    small = P.aatc_calibrate_bits(w.calib(0, "k"), ora.allocate_bits(np.ones(128), 100, 8))
    assert small.record_bytes == 16
    with pytest.raises(P.AatcError):
        P.aatc_params_pack([cals[0], small])                  # record sizes differ


def _global_cases():
    rng = np.random.default_rng(2024)
    ints = rng.integers(0, 4, size=(5, 16)).astype(np.float64)      # many exact ties
    zero = rng.gamma(0.5, size=(4, 24))
    zero[1] = 0.0                                                   # percentile 0
    return [
        (rng.gamma(0.5, size=(5, 8)), rng.gamma(1.0, size=(5, 8)), 2.0, 8, 3, 1, True),
        (rng.gamma(0.3, size=(8, 512)), rng.gamma(1.0, size=(8, 512)), 2.75, 8, 3, 1, True),
        (rng.gamma(0.3, size=(8, 512)), None, 2.75, 8, 3, 0, False),
        (ints, ints[::-1].copy(), 1.5, 4, 0, 0, True),
        (zero, None, 3.0, 6, 1, 0, False),
        (rng.gamma(0.5, size=(2, 64)), None, 2.0, 8, 3, 1, False),  # all protected
        (rng.gamma(0.5, size=(1, 128)), rng.gamma(1.0, size=(1, 128)), 2.0, 8, 0, 0, True),
    ]


@pytest.mark.parametrize("case", range(7))
def test_allocate_global_matches_oracle(case):
    """aatc_allocate_global against the oracle, width for width."""
    s2, w, avg, b_max, n_prot, extra, norm = _global_cases()[case]
    want = ora.allocate_global(s2, w, avg, b_max, n_protect=n_prot, protect_extra=extra,
                               normalize_weight=norm)
    got = P.aatc_allocate_global(s2, w, avg, b_max, n_prot, extra, norm)
    np.testing.assert_array_equal(got.astype(np.int64), want)


def test_allocate_global_errors():
    s2 = np.ones((4, 8))
    for args in [(s2, None, 0.5, 8, 3, 1, False),      # protected layers exceed the total
                 (s2, None, 8.5, 8, 0, 0, False),      # the pool exceeds b_max
                 (s2, None, 2.0, 17, 3, 0, False),     # b_max above 16
                 (s2, None, 1e300, 8, 0, 0, False),    # an average beyond any width
                 (-s2, None, 2.0, 8, 3, 0, False),     # negative variance
                 (s2, np.full((4, 8), np.nan), 2.0, 8, 3, 0, False)]:
        with pytest.raises(P.AatcError):
            P.aatc_allocate_global(*args)


@pytest.mark.parametrize("cfg,head,kind", [(3, 0, "k"), (3, 2, "k"), (2, 1, "k"), (4, 0, "v")])
def test_host_calibration_sixteen_bit_cap_matches_oracle(cfg, head, kind):
    """b_max = 16 (App. E): the host allocation gives the oracle's widths, above 8 where
    the weighted variance calls for it (the Qwen-shape keys take 9 and 10 bits)."""
    w = workload(cfg, n_tokens=64)
    x = w.calib(head, kind)
    avg = 8.0 if cfg == 4 else w.cfg["avg_bits"][0]
    c = P.aatc_calibrate(x, avg, b_max=16)
    o = ora.calibrate(x, avg, b_max=16)
    np.testing.assert_array_equal(c.bits_np, o.bits)
    np.testing.assert_array_equal(c.s16.view(np.uint16), o.s16.view(np.uint16))
    assert c.quantizer == P.QUANT_MIDTREAD
    if cfg == 3:
        assert c.bits_np.max() > 8
    with pytest.raises(P.AatcError):
        P.aatc_calibrate(x, avg, b_max=17)


def test_params_pack_quantizer_reading():
    """The quantizer reading travels in the calibration: one reading per tensor, and only
    the two defined values are accepted."""
    w = workload(2, n_tokens=64)
    cals = [abi_calibration(ora.calibrate(w.calib(h, "k"), 2.75)) for h in range(2)]
    P.aatc_params_pack(cals)
    for c in cals:
        c.quantizer = P.QUANT_MIDRISE
    P.aatc_params_pack(cals)
    cals[1].quantizer = P.QUANT_MIDTREAD
    with pytest.raises(P.AatcError):
        P.aatc_params_pack(cals)
    cals[1].quantizer = 7
    with pytest.raises(P.AatcError):
        P.aatc_params_pack(cals)


@pytest.mark.parametrize("weights", ["var_only", "queries"])
def test_host_whitened_calibration_matches_oracle(weights):
    """aatc_calibrate_whitened (Cholesky, whitened Gram matrix, Jacobi) against the oracle's
    literal whitened SVD: widths, storage order and fp16 scales identical; transform within
    one grid step; and equal to aatc_calibrate on K = X W."""
    from kvsynth import layer_inputs, projection
    x = layer_inputs(11, 1024, 160)
    w = projection(11, 160, 128)
    kw = {}
    if weights == "queries":
        q = np.random.default_rng(3).standard_normal((2 * 300, 128)).astype(np.float32)
        kw = dict(q_calib=q, q_group=2)
    c = P.aatc_calibrate_whitened(x, w, 2.75, **kw)
    o = ora.calibrate_whitened(x, w, 2.75, q_calib=kw.get("q_calib"), group=kw.get("q_group", 1))
    np.testing.assert_array_equal(c.bits_np, o.bits)
    np.testing.assert_array_equal(np.ctypeslib.as_array(c.perm), o.perm)
    np.testing.assert_array_equal(c.s16.view(np.uint16), o.s16.view(np.uint16))
    assert np.abs(c.T.astype(np.float64) - o.T32).max() <= 2.0 ** -22
    k = (x.astype(np.float64) @ w.astype(np.float64)).astype(np.float32)
    c2 = P.aatc_calibrate(k, 2.75, **kw)
    np.testing.assert_array_equal(c.bits_np, c2.bits_np)


def test_host_whitened_calibration_errors():
    from kvsynth import projection
    w = projection(1, 32, 128)
    x = np.zeros((64, 32), dtype=np.float32)                  # Sigma_X = 0: not definite
    with pytest.raises(P.AatcError):
        P.aatc_calibrate_whitened(x, w, 2.75)
    with pytest.raises(ValueError):
        P.aatc_calibrate_whitened(np.ones((64, 16), np.float32), w, 2.75)
    with pytest.raises(P.AatcError):
        P.aatc_calibrate_whitened(np.ones((64, 32), np.float32), projection(1, 32, 64), 2.75)
