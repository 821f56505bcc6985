"""Host-side checks of the head-group entry points that need no GPU: calibration parity
with the oracle, parameter packing, argument validation before any launch."""
import ctypes

import numpy as np
import pytest

import paper_2608_14191_amd as P
from kvsynth import workload
from oracle import aatc as ora
from oracle import groups as og

from helpers import abi_group_calibration


def _group_calib(cfg, g, gkv, kind):
    w = workload(cfg, n_tokens=64)
    x = np.concatenate([w.calib(h, kind) for h in range(g * gkv, (g + 1) * gkv)], axis=1)
    return w, x


@pytest.mark.parametrize("cfg,g,gkv,kind", [(2, 1, 2, "k"), (2, 0, 2, "v"), (3, 0, 4, "k")])
def test_host_group_calibration_matches_oracle(cfg, g, gkv, kind):
    w, x = _group_calib(cfg, g, gkv, kind)
    avg = w.cfg["avg_bits"][0]
    c = P.aatc_calibrate_group(x, avg)
    o = og.calibrate_group(x, avg)
    d = 128 * gkv
    assert c.d == d == o.d
    np.testing.assert_array_equal(c.bits_np, o.bits)
    np.testing.assert_array_equal(np.ctypeslib.as_array(c.perm)[:d], o.perm)
    np.testing.assert_array_equal(c.s16.view(np.uint16), o.s16.view(np.uint16))
    assert (c.budget_bits, c.record_bytes, c.d_active) == (o.budget, o.record_bytes, o.d_active)
    q = np.ldexp(c.T.astype(np.float64), 22)
    np.testing.assert_array_equal(q, np.rint(q))
    assert np.abs(c.T.astype(np.float64) - o.T32).max() <= 2.0 ** -22
    assert np.count_nonzero(c.T != o.T32) <= 8


def test_host_group_calibration_query_weighted_matches_oracle():
    w, x = _group_calib(5, 1, 2, "k")
    gq = w.group
    qs = np.stack([w.calib_queries(h, n=256).reshape(gq, 256, 128).transpose(1, 0, 2)
                   for h in (2, 3)], axis=1)                 # [T, gkv, G_q, 128]
    qe = og.embed_group_queries(qs, 2).astype(np.float32)
    c = P.aatc_calibrate_group(x, 2.0, q_calib=qe, q_group=2 * gq)
    o = og.calibrate_group(x, 2.0, q_embedded=qe, n_q_heads=2 * gq)
    np.testing.assert_array_equal(c.bits_np, o.bits)
    np.testing.assert_allclose(np.ctypeslib.as_array(c.weight)[:256], o.weight, rtol=1e-9)


def test_group_calibration_errors():
    x = np.random.default_rng(0).standard_normal((64, 200)).astype(np.float32)
    with pytest.raises(P.AatcError) as e:
        P.aatc_calibrate_group(x, 2.0)                       # d not a multiple of 128
    assert e.value.status == 2
    x = np.random.default_rng(0).standard_normal((64, 640)).astype(np.float32)
    with pytest.raises(P.AatcError):
        P.aatc_calibrate_group(x, 2.0)                       # wider than 512


def test_group_params_pack_layout_and_validation():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal((600, 256)) * np.linspace(2, 0.01, 256)).astype(np.float32)
    o = og.calibrate_group(x, 3.0, quantizer="midrise")
    c = abi_group_calibration(o)
    buf = P.aatc_group_params_pack([c, c])
    assert buf.nbytes == P.aatc_group_params_bytes(2)
    hdr = buf[:16].view(np.int32)
    assert hdr[0] == 0x47544141 and hdr[1] == 2 and hdr[2] == 256 and hdr[3] == o.record_bytes
    gp = buf[256:]
    d = 256
    tqt = gp[:4 * d * d].view(np.int32).reshape(d, d)          # [c][j]
    np.testing.assert_array_equal(tqt, np.ldexp(o.T32.astype(np.float64), 22).T.astype(np.int64))
    t_off = 4 * 512 * 512
    t = gp[t_off:t_off + 4 * d * d].view(np.float32).reshape(d, d)
    np.testing.assert_array_equal(t, o.T32)
    bad = abi_group_calibration(o)
    bad.transform[5] = 0.1                                      # off the 2^-22 grid
    with pytest.raises(P.AatcError):
        P.aatc_group_params_pack([bad])
    bad = abi_group_calibration(o)
    bad.d = 200
    with pytest.raises(P.AatcError):
        P.aatc_group_params_pack([bad])
    other = abi_group_calibration(og.calibrate_group(x, 4.0))
    with pytest.raises(P.AatcError):
        P.aatc_group_params_pack([c, other])                    # record sizes differ


def _fake(addr=4096):
    return ctypes.c_void_p(addr)


def test_group_encode_and_decode_validate_before_launch():
    L = P.library()
    p = _fake()
    # gkv out of range, pos + n_tok > cap, misaligned codes, short token stride
    assert L.aatc_group_encode(p, 2, 5, p, 1, 1, 1024, p, p, 64, 0, None) == 1
    assert L.aatc_group_encode(p, 2, 4, p, 1, 10, 1024, p, p, 64, 60, None) == 1
    assert L.aatc_group_encode(p, 2, 4, p, 1, 1, 1024, _fake(4100), p, 64, 0, None) == 1
    assert L.aatc_group_encode(p, 2, 4, p, 1, 1, 1000, p, p, 64, 0, None) == 1
    assert L.aatc_group_encode(p, 2, 4, p, 1, 0, 1024, p, p, 64, 0, None) == 0   # no-op
    ws = P.aatc_group_decode_workspace_bytes(1, 32, 8, 4, 4096)
    assert ws > 0
    assert P.aatc_group_decode_workspace_bytes(1, 32, 8, 3, 4096) == 0
    args = [p, p, 1, 32, 8, 4, p, 1, p, p, p, p, p, 4096, 176, 176, 0.088, p, p, ws, None]
    bad = list(args); bad[5] = 3                       # 8 % 3 != 0
    assert L.aatc_group_decode_attention(*bad) == 1
    bad = list(args); bad[14] = 42                     # record size not whole dwords
    assert L.aatc_group_decode_attention(*bad) == 1
    bad = list(args); bad[15] = 516                    # record larger than the decode stages
    assert L.aatc_group_decode_attention(*bad) == 2
    bad = list(args); bad[3] = 80                      # 40 query heads per group
    bad[19] = P.aatc_group_decode_workspace_bytes(1, 80, 8, 4, 4096)
    assert L.aatc_group_decode_attention(*bad) == 2
    bad = list(args); bad[19] = ws - 1                 # workspace too small
    assert L.aatc_group_decode_attention(*bad) == 5
