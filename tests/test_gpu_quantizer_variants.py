"""GPU parity of the quantizer readings and widths (the midrise reading of Sec. 5.2's
quantizer, symmetric with errors of at most half a step as Sec. 4 and App. B describe it;
channel widths up to 16 bits as App. E allows): every encode path bit-exact against the
oracle, every decode path within the same tolerance as the default reading."""
import numpy as np
import pytest
import torch

import paper_2608_14191_amd as P
from oracle import aatc as ora

from helpers import alpha_cache, device_params, record_cache, tile_cache
from test_gpu_parity import (Case, _assert_heads_close, _check_codes, _decode, _gpu_caches,
                             _log, _oracle_decode, append_check)

pytestmark = pytest.mark.gpu


class VCase(Case):
    """A reduced workload whose calibrations use the given quantizer reading and width cap."""

    def __init__(self, quantizer="midtread", b_max=8, **kw):
        super().__init__(**kw)
        w = self.w
        if b_max != 8:
            qw = w.cfg["query_weighted_k"]
            self.cal_k = [ora.calibrate(w.calib(h, "k"), self.avg, b_max=b_max,
                                        q_calib=w.calib_queries(h) if qw else None,
                                        group=w.group) for h in range(w.n_kv_heads)]
            self.cal_v = [ora.calibrate(w.calib(h, "v"), self.avg, b_max=b_max)
                          for h in range(w.n_kv_heads)]
        for c in self.cal_k + self.cal_v:
            c.quantizer = quantizer
        # the heads of one tensor share the record size of the widest
        for cals in (self.cal_k, self.cal_v):
            rb = max(c.record_bytes for c in cals)
            for c in cals:
                c.record_bytes = rb


CASES = {
    # MFMA decode kernel (G <= 8, records <= 64 bytes)
    "midrise_cfg2_ragged_1000": dict(quantizer="midrise", cfg=2, n_tokens=1000),
    "midrise_cfg3_b2_gqa7": dict(quantizer="midrise", cfg=3, n_tokens=700, batch=2,
                                 lens=[700, 333]),
    "midrise_cfg5_zero_bit_keys": dict(quantizer="midrise", cfg=5, n_tokens=600),
    # keys of the Qwen shape take 9 and 10 bits once b_max is 16
    "bmax16_cfg3_wide_keys": dict(b_max=16, cfg=3, n_tokens=500, batch=2, lens=[500, 77]),
    "bmax16_midrise_cfg3": dict(quantizer="midrise", b_max=16, cfg=3, n_tokens=300),
    # generic VALU decode kernel (records over 64 bytes, or G > 8)
    "midrise_generic_6bit": dict(quantizer="midrise", cfg=4, n_tokens=400, avg_bits=6.0),
    "midrise_generic_gqa16": dict(quantizer="midrise", cfg=2, n_tokens=500, n_q_heads=32,
                                  n_kv_heads=2),
    "bmax16_generic_8bit": dict(b_max=16, quantizer="midrise", cfg=2, n_tokens=200,
                                avg_bits=8.0),
}


@pytest.mark.parametrize("name", list(CASES))
def test_variant_encode_bit_exact_and_decode_parity(name):
    _log(f"[case] {name}")
    case = VCase(**CASES[name])
    if "bmax16" in name:
        assert max(int(c.bits.max()) for c in case.cal_k + case.cal_v) > 8, "no wide channel"
    pk, pv, kc, ka, vc, va = _gpu_caches(case)
    _check_codes(case, kc, ka, vc, va)
    out, _ = _decode(case, pk, pv, kc, ka, vc, va)
    ref = _oracle_decode(case)
    for b in range(case.w.batch):
        err = _assert_heads_close(out[b], ref[b], f"seq {b}")
        _log(f"  seq {b} len {case.lens[b]} worst head rel_l2 {err:.3e}")


APPEND = {
    "midrise_cfg2_split_edges": dict(quantizer="midrise", cfg=2, n_tokens=1025, batch=3,
                                     lens=[1025, 700, 1]),
    "bmax16_midrise_cfg3": dict(quantizer="midrise", b_max=16, cfg=3, n_tokens=300, batch=2,
                                lens=[300, 65]),
    "midrise_generic_gqa16": dict(quantizer="midrise", cfg=2, n_tokens=300, n_q_heads=32,
                                  n_kv_heads=2),
}


@pytest.mark.parametrize("name", list(APPEND))
def test_variant_fused_append(name):
    _log(f"[append] {name}")
    append_check(VCase(**APPEND[name]))


@pytest.mark.parametrize("quantizer,b_max", [("midrise", 8), ("midrise", 16), ("midtread", 16)])
def test_variant_small_appends_and_unaligned_rows(quantizer, b_max):
    """The per-token kernel (appends of up to 16 tokens) and the unaligned-row kernel give
    the oracle's codes under either reading and width cap."""
    case = VCase(quantizer=quantizer, b_max=b_max, cfg=3, n_tokens=150)
    H, cap, n = case.w.n_kv_heads, case.cap, 150
    pk, pv = device_params(case.cal_k), device_params(case.cal_v)
    for kind, pp, cal, layout in (("k", pk, case.cal_k, P.LAYOUT_RECORDS),
                                  ("v", pv, case.cal_v, P.LAYOUT_TILES)):
        x = case.x_tokens(0, kind).reshape(n, H * 128)
        rb = cal[0].record_bytes
        for mode in ("appends", "unaligned"):
            codes = record_cache(H, cap, rb) if kind == "k" else tile_cache(H, cap, rb)
            al = alpha_cache(H, cap)
            if mode == "appends":
                pos = 0
                for m in [1, 16, 3, 64, 1, 65]:
                    P.aatc_encode(pp, H, x[pos:], m, H * 128, layout, codes, al, cap, pos)
                    pos += m
                assert pos == n
            else:
                xp = torch.zeros((n, H * 128 + 1), dtype=x.dtype, device=x.device)
                xp[:, :H * 128] = x
                P.aatc_encode(pp, H, xp, n, H * 128 + 1, layout, codes, al, cap, 0)
            torch.cuda.synchronize()
            for h in range(H):
                rec, a16 = case.oracle_encode(0, h, kind)
                got = codes[h, :n].cpu().numpy() if kind == "k" else \
                    ora.tiles_to_records(codes[h].cpu().numpy(), rb)[:n]
                np.testing.assert_array_equal(got, rec, err_msg=f"{kind} {mode} head {h}")
                np.testing.assert_array_equal(al[h, :n].cpu().numpy().view(np.uint16),
                                              a16.view(np.uint16))


def test_host_calibration_sixteen_bits_midrise_end_to_end():
    """aatc_calibrate (host) with b_max = 16, the midrise reading set on the calibrations,
    through encode and decode, against the oracle's pipeline on the same widths."""
    case = VCase(quantizer="midrise", b_max=16, cfg=3, n_tokens=400)
    w = case.w
    abi_k = [P.aatc_calibrate(w.calib(h, "k"), case.avg, b_max=16) for h in range(w.n_kv_heads)]
    abi_v = [P.aatc_calibrate(w.calib(h, "v"), case.avg, b_max=16) for h in range(w.n_kv_heads)]
    for c in abi_k + abi_v:
        c.quantizer = P.QUANT_MIDRISE
    for abi, cal in zip(abi_k + abi_v, case.cal_k + case.cal_v):
        np.testing.assert_array_equal(abi.bits_np, cal.bits)
    pk, pv = device_params(abi_k), device_params(abi_v)
    _, _, kc, ka, vc, va = _gpu_caches(case, pk, pv)
    _check_codes(case, kc, ka, vc, va)
    out, _ = _decode(case, pk, pv, kc, ka, vc, va)
    _assert_heads_close(out[0], _oracle_decode(case)[0])
