"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bar: bit-exact packed codes and fp16 token scales; decode attention within 2e-3
relative L2 of the oracle's exact fp64 attention over the decoded cache, for every query
head separately, and within 2e-3 of that head's largest output magnitude element by
element.
"""
import numpy as np
import pytest
import torch

import paper_2608_14191_amd as P
from kvsynth import workload
from oracle import aatc as ora

from helpers import (alpha_cache, device_params, oracle_tiles, record_cache, rel_l2,
                     stored_to_torch, tile_cache)

pytestmark = pytest.mark.gpu
TOL = 2e-3


def _log(msg):
    print(msg, flush=True)


def _assert_heads_close(got, ref, what=""):
    """Per query head: relative L2 <= TOL and max |error| <= TOL * max |ref|."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    worst = 0.0
    for j in range(ref.shape[0]):
        err = rel_l2(got[j], ref[j])
        worst = max(worst, err)
        assert err <= TOL, f"{what} query head {j}: rel L2 {err:.3e}"
        assert np.abs(got[j] - ref[j]).max() <= TOL * np.abs(ref[j]).max(), f"{what} head {j}"
    return worst


class Case:
    """Calibrations, stored tokens and queries of a (reduced) workload."""

    def __init__(self, cfg, n_tokens, batch=1, lens=None, avg_bits=None, **overrides):
        self.w = workload(cfg, n_tokens=n_tokens, batch=batch, **overrides)
        w = self.w
        self.avg = w.cfg["avg_bits"][0] if avg_bits is None else avg_bits
        self.lens = [n_tokens] * batch if lens is None else lens
        self.cap = max(64, -(-max(self.lens + [1]) // 64) * 64)
        qw = w.cfg["query_weighted_k"]
        self.cal_k = [ora.calibrate(w.calib(h, "k"), self.avg,
                                    q_calib=w.calib_queries(h) if qw else None,
                                    group=w.group) for h in range(w.n_kv_heads)]
        self.cal_v = [ora.calibrate(w.calib(h, "v"), self.avg) for h in range(w.n_kv_heads)]
        self.k = [[w.cache(b, h, "k", n=self.lens[b]) for h in range(w.n_kv_heads)]
                  for b in range(batch)]
        self.v = [[w.cache(b, h, "v", n=self.lens[b]) for h in range(w.n_kv_heads)]
                  for b in range(batch)]
        self.q = [w.queries(b) for b in range(batch)]

    def x_tokens(self, b, kind):
        """torch [len, H_kv, 128] (fp32 or bf16) of sequence b."""
        parts = self.k[b] if kind == "k" else self.v[b]
        arr = np.stack(parts, axis=1)
        return stored_to_torch(arr).cuda()

    def oracle_encode(self, b, h, kind):
        cal = (self.cal_k if kind == "k" else self.cal_v)[h]
        x = self.w.as_f32((self.k if kind == "k" else self.v)[b][h])
        rec, a16, _ = ora.encode(x, cal)
        return rec, a16


def _gpu_caches(case, params_k=None, params_v=None):
    w = case.w
    H, B, cap = w.n_kv_heads, w.batch, case.cap
    pk = device_params(case.cal_k) if params_k is None else params_k
    pv = device_params(case.cal_v) if params_v is None else params_v
    kc = record_cache(H, cap, case.cal_k[0].record_bytes, batch=B)
    ka = alpha_cache(H, cap, batch=B)
    vc = tile_cache(H, cap, case.cal_v[0].record_bytes, batch=B)
    va = alpha_cache(H, cap, batch=B)
    for b in range(B):
        n = case.lens[b]
        if n == 0:
            continue
        xk, xv = case.x_tokens(b, "k"), case.x_tokens(b, "v")
        P.aatc_encode(pk, H, xk, n, H * 128, P.LAYOUT_RECORDS, kc[b], ka[b], cap, 0)
        P.aatc_encode(pv, H, xv, n, H * 128, P.LAYOUT_TILES, vc[b], va[b], cap, 0)
    torch.cuda.synchronize()
    return pk, pv, kc, ka, vc, va


def _check_codes(case, kc, ka, vc, va):
    for b in range(case.w.batch):
        n = case.lens[b]
        for h in range(case.w.n_kv_heads):
            rk, ak = case.oracle_encode(b, h, "k")
            rv, av = case.oracle_encode(b, h, "v")
            got = kc[b, h, :n].cpu().numpy()
            bad = np.argwhere(np.any(got != rk, axis=1))
            assert bad.size == 0, f"seq {b} head {h}: key records differ at tokens {bad[:5].ravel()}"
            np.testing.assert_array_equal(ka[b, h, :n].cpu().numpy().view(np.uint16),
                                          ak.view(np.uint16))
            np.testing.assert_array_equal(vc[b, h].cpu().numpy(), oracle_tiles(rv, case.cap))
            np.testing.assert_array_equal(va[b, h, :n].cpu().numpy().view(np.uint16),
                                          av.view(np.uint16))


def _decode(case, pk, pv, kc, ka, vc, va):
    w = case.w
    B, H, HQ = w.batch, w.n_kv_heads, w.n_q_heads
    q = stored_to_torch(np.stack(case.q)).cuda()
    lens = torch.tensor(case.lens, dtype=torch.int32, device="cuda")
    out = torch.full((B, HQ, 128), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.zeros(P.aatc_decode_workspace_bytes(B, HQ, H, case.cap), dtype=torch.uint8,
                     device="cuda")
    P.aatc_decode_attention(pk, pv, B, HQ, H, q, kc, ka, vc, va, lens, case.cap,
                            case.cal_k[0].record_bytes, case.cal_v[0].record_bytes,
                            1 / np.sqrt(128), out, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy(), ws


def _oracle_decode(case):
    outs = []
    for b in range(case.w.batch):
        n = case.lens[b]
        q32 = case.w.as_f32(case.q[b])
        if n == 0:
            outs.append(np.zeros_like(q32, dtype=np.float64))
            continue
        enc_k = [case.oracle_encode(b, h, "k") for h in range(case.w.n_kv_heads)]
        enc_v = [case.oracle_encode(b, h, "v") for h in range(case.w.n_kv_heads)]
        outs.append(ora.decode_attention(q32, case.cal_k, case.cal_v, [e[0] for e in enc_k],
                                         [e[1] for e in enc_k], [e[0] for e in enc_v],
                                         [e[1] for e in enc_v], n))
    return np.stack(outs)


CASES = {
    "cfg1_single_head_512": dict(cfg=1, n_tokens=512),
    "cfg2_llama_ragged_1000": dict(cfg=2, n_tokens=1000),
    "cfg3_qwen_b2_ragged": dict(cfg=3, n_tokens=700, batch=2, lens=[700, 333]),
    "cfg5_long_qweighted_zero_bits": dict(cfg=5, n_tokens=1100, batch=2, lens=[1100, 65]),
    "cfg4_llama_4bit_300": dict(cfg=4, n_tokens=300, avg_bits=4.0),
    # outside the MFMA kernel's range: the generic kernel runs these
    "generic_gqa16": dict(cfg=2, n_tokens=700, n_q_heads=32, n_kv_heads=2),
    "generic_6bit": dict(cfg=4, n_tokens=400, avg_bits=6.0),
}


@pytest.mark.parametrize("name", list(CASES))
def test_encode_bit_exact_and_decode_parity(name):
    _log(f"[case] {name}")
    case = Case(**CASES[name])
    pk, pv, kc, ka, vc, va = _gpu_caches(case)
    _check_codes(case, kc, ka, vc, va)
    out, _ = _decode(case, pk, pv, kc, ka, vc, va)
    ref = _oracle_decode(case)
    for b in range(case.w.batch):
        if case.lens[b] == 0:
            assert np.all(out[b] == 0)
            continue
        err = _assert_heads_close(out[b], ref[b], f"seq {b}")
        _log(f"  seq {b} len {case.lens[b]} worst head rel_l2 {err:.3e}")


def test_encode_incremental_appends_match_bulk():
    """Decode-step appends (1 token, odd chunks, partial tiles) give the same caches."""
    case = Case(cfg=2, n_tokens=300)
    H, cap = case.w.n_kv_heads, case.cap
    pk, pv = device_params(case.cal_k), device_params(case.cal_v)
    xk, xv = case.x_tokens(0, "k"), case.x_tokens(0, "v")
    kc = record_cache(H, cap, case.cal_k[0].record_bytes)
    vc = tile_cache(H, cap, case.cal_v[0].record_bytes)
    ka, va = alpha_cache(H, cap), alpha_cache(H, cap)
    vc.fill_(0xA5)          # stale bytes beyond the written tokens must not matter
    pos = 0
    for n in [1, 1, 5, 16, 41, 1, 64, 3, 100, 68]:      # 16: largest per-token append
        P.aatc_encode(pk, H, xk[pos:], n, H * 128, P.LAYOUT_RECORDS, kc, ka, cap, pos)
        P.aatc_encode(pv, H, xv[pos:], n, H * 128, P.LAYOUT_TILES, vc, va, cap, pos)
        pos += n
    assert pos == 300
    torch.cuda.synchronize()
    for h in range(H):
        rk, ak = case.oracle_encode(0, h, "k")
        rv, av = case.oracle_encode(0, h, "v")
        np.testing.assert_array_equal(kc[h, :300].cpu().numpy(), rk)
        got = ora.tiles_to_records(vc[h].cpu().numpy(), rv.shape[1])
        np.testing.assert_array_equal(got[:300], rv)
        np.testing.assert_array_equal(va[h, :300].cpu().numpy().view(np.uint16), av.view(np.uint16))


def test_encode_unaligned_rows_match_oracle():
    """Token rows that are not 16-byte aligned take the VALU encode path: same codes."""
    case = Case(cfg=2, n_tokens=200)
    H, cap, n = case.w.n_kv_heads, case.cap, 200
    pk, pv = device_params(case.cal_k), device_params(case.cal_v)
    caches = {}
    for kind, pp, cal, layout in (("k", pk, case.cal_k, P.LAYOUT_RECORDS),
                                  ("v", pv, case.cal_v, P.LAYOUT_TILES)):
        x = case.x_tokens(0, kind).reshape(n, H * 128)
        xp = torch.zeros((n, H * 128 + 1), dtype=x.dtype, device=x.device)
        xp[:, :H * 128] = x
        rb = cal[0].record_bytes
        codes = record_cache(H, cap, rb) if kind == "k" else tile_cache(H, cap, rb)
        al = alpha_cache(H, cap)
        P.aatc_encode(pp, H, xp, n, H * 128 + 1, layout, codes, al, cap, 0)
        caches[kind] = (codes, al)
    torch.cuda.synchronize()
    for h in range(H):
        rk, ak = case.oracle_encode(0, h, "k")
        rv, av = case.oracle_encode(0, h, "v")
        np.testing.assert_array_equal(caches["k"][0][h, :n].cpu().numpy(), rk)
        np.testing.assert_array_equal(caches["k"][1][h, :n].cpu().numpy().view(np.uint16), ak.view(np.uint16))
        got = ora.tiles_to_records(caches["v"][0][h].cpu().numpy(), rv.shape[1])
        np.testing.assert_array_equal(got[:n], rv)
        np.testing.assert_array_equal(caches["v"][1][h, :n].cpu().numpy().view(np.uint16), av.view(np.uint16))


def test_decode_edge_lengths():
    """Empty, single-token, tile-edge and ragged lengths in one batch."""
    lens = [0, 1, 63, 64, 65, 511, 512, 513]
    case = Case(cfg=2, n_tokens=513, batch=len(lens), lens=lens)
    pk, pv, kc, ka, vc, va = _gpu_caches(case)
    out, _ = _decode(case, pk, pv, kc, ka, vc, va)
    ref = _oracle_decode(case)
    assert np.all(out[0] == 0)
    for b in range(1, len(lens)):
        _assert_heads_close(out[b], ref[b], f"seq {b} len {lens[b]}")


def test_decode_repeatable_and_workspace_reusable():
    case = Case(cfg=3, n_tokens=640, batch=1)
    pk, pv, kc, ka, vc, va = _gpu_caches(case)
    o1, ws = _decode(case, pk, pv, kc, ka, vc, va)
    o2, _ = _decode(case, pk, pv, kc, ka, vc, va)
    np.testing.assert_array_equal(o1, o2)


def test_end_to_end_with_host_calibration():
    """aatc_calibrate (host C++) -> encode -> decode against the oracle pipeline."""
    case = Case(cfg=5, n_tokens=800)
    w = case.w
    abi_k = [P.aatc_calibrate(w.calib(h, "k"), case.avg, q_calib=w.calib_queries(h),
                              q_group=w.group) for h in range(w.n_kv_heads)]
    abi_v = [P.aatc_calibrate(w.calib(h, "v"), case.avg) for h in range(w.n_kv_heads)]
    pk, pv = device_params(abi_k), device_params(abi_v)
    pk_, pv_, kc, ka, vc, va = _gpu_caches(case, pk, pv)
    out, _ = _decode(case, pk, pv, kc, ka, vc, va)
    ref = _oracle_decode(case)
    _assert_heads_close(out[0], ref[0])


APPEND_CASES = {
    # new token first in a 1024-token split, last in a split, mid-tile, alone, no token
    "cfg2_split_edges": dict(cfg=2, n_tokens=1025, batch=5, lens=[1025, 1024, 700, 1, 0]),
    "cfg3_gqa7_ragged": dict(cfg=3, n_tokens=600, batch=2, lens=[600, 129]),
    "cfg4_4bit_wide_records": dict(cfg=4, n_tokens=200, avg_bits=4.0),
    "generic_gqa16": dict(cfg=2, n_tokens=300, n_q_heads=32, n_kv_heads=2),
}


@pytest.mark.parametrize("name", list(APPEND_CASES))
def test_append_decode_matches_encode_then_decode(name):
    """One aatc_append_decode_attention call gives the codes of encoding the new token and
    the outputs of decoding the updated cache (oracle and separate calls)."""
    _log(f"[append] {name}")
    append_check(Case(**APPEND_CASES[name]))


def append_check(case):
    """The fused append + decode of each sequence's last token against the oracle's codes
    and attention and against separate encode + decode calls."""
    w = case.w
    B, H, HQ, cap = w.batch, w.n_kv_heads, w.n_q_heads, case.cap
    rk, rv = case.cal_k[0].record_bytes, case.cal_v[0].record_bytes
    pk, pv, _, _, _, _ = _gpu_caches(case)
    kc = record_cache(H, cap, rk, batch=B).fill_(0xA5)       # stale bytes everywhere
    vc = tile_cache(H, cap, rv, batch=B).fill_(0x5A)
    ka, va = alpha_cache(H, cap, batch=B), alpha_cache(H, cap, batch=B)
    xk_new = torch.zeros((B, H, 128), dtype=torch.bfloat16 if w.dtype == "bf16" else torch.float32)
    xv_new = torch.zeros_like(xk_new)
    for b in range(B):
        n = case.lens[b]
        if n == 0:
            continue
        xk, xv = case.x_tokens(b, "k"), case.x_tokens(b, "v")
        if n > 1:
            P.aatc_encode(pk, H, xk, n - 1, H * 128, P.LAYOUT_RECORDS, kc[b], ka[b], cap, 0)
            P.aatc_encode(pv, H, xv, n - 1, H * 128, P.LAYOUT_TILES, vc[b], va[b], cap, 0)
        xk_new[b], xv_new[b] = xk[n - 1].cpu(), xv[n - 1].cpu()
    q = stored_to_torch(np.stack(case.q)).cuda()
    lens = torch.tensor(case.lens, dtype=torch.int32, device="cuda")
    out = torch.full((B, HQ, 128), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.zeros(P.aatc_decode_workspace_bytes(B, HQ, H, cap), dtype=torch.uint8,
                     device="cuda")
    P.aatc_append_decode_attention(pk, pv, B, HQ, H, q, xk_new.cuda(), xv_new.cuda(), kc, ka,
                                   vc, va, lens, cap, rk, rv, 1 / np.sqrt(128), out, ws)
    torch.cuda.synchronize()
    for b in range(B):
        n = case.lens[b]
        for h in range(H):
            ok_, oa = case.oracle_encode(b, h, "k")
            ov_, ova = case.oracle_encode(b, h, "v")
            np.testing.assert_array_equal(kc[b, h, :n].cpu().numpy(), ok_)
            np.testing.assert_array_equal(ka[b, h, :n].cpu().numpy().view(np.uint16), oa.view(np.uint16))
            got_v = ora.tiles_to_records(vc[b, h].cpu().numpy(), rv)[:n]
            np.testing.assert_array_equal(got_v, ov_)
            np.testing.assert_array_equal(va[b, h, :n].cpu().numpy().view(np.uint16), ova.view(np.uint16))
    got = out.cpu().numpy()
    ref = _oracle_decode(case)
    sep, _ = _decode(case, pk, pv, kc, ka, vc, va)
    for b in range(B):
        if case.lens[b] == 0:
            assert np.all(got[b] == 0)
            continue
        _assert_heads_close(got[b], ref[b], f"seq {b} len {case.lens[b]}")
        assert rel_l2(got[b], sep[b]) <= 1e-5, (b, case.lens[b])


FULL_SIZE = {
    # the benchmark's workload and launch (append the last token, decode all 32768):
    # every KV head
    "cfg2_llama_32k": dict(cfg=2, sample=[(0, h) for h in range(8)]),
    # every KV head of two of the eight sequences
    "cfg3_qwen_16k_b8": dict(cfg=3, sample=[(b, h) for b in (3, 7) for h in range(4)]),
    # the largest decode workload: 4 x 131072 tokens, 2.0 bits, zero-bit key channels,
    # 128 splits per (sequence, KV head) into one merge; every KV head of two sequences
    "cfg5_long_131k_b4": dict(cfg=5, sample=[(b, h) for b in (0, 3) for h in range(8)]),
}
# generating 4 x 8 x 131072 stored tokens per tensor takes about a minute on the host
_FULL_SLOW = {"cfg5_long_131k_b4"}


@pytest.mark.parametrize("name", [pytest.param(n, marks=pytest.mark.timeout(600))
                                  if n in _FULL_SLOW else
                                  pytest.param(n, marks=pytest.mark.timeout(300))
                                  for n in FULL_SIZE])
def test_full_size_sampled(name):
    """Full-size workloads through aatc_append_decode_attention: the packed caches of
    sampled (sequence, KV head) pairs are bit-exact, including the appended token, and
    the outputs of their query heads are within TOL of the oracle."""
    spec = FULL_SIZE[name]
    full = workload(spec["cfg"])
    _log(f"[full] {name}: batch {full.batch}, {full.n_tokens} tokens, "
         f"{full.n_q_heads}/{full.n_kv_heads} heads")
    case = Case(cfg=spec["cfg"], n_tokens=full.n_tokens, batch=full.batch)
    _log(f"  generated, bits k {case.cal_k[0].record_bytes * 8} v {case.cal_v[0].record_bytes * 8}")
    w = case.w
    B, H, HQ, cap = w.batch, w.n_kv_heads, w.n_q_heads, case.cap
    rk, rv = case.cal_k[0].record_bytes, case.cal_v[0].record_bytes
    pk, pv = device_params(case.cal_k), device_params(case.cal_v)
    kc, vc = record_cache(H, cap, rk, batch=B), tile_cache(H, cap, rv, batch=B)
    ka, va = alpha_cache(H, cap, batch=B), alpha_cache(H, cap, batch=B)
    xk_new = torch.zeros((B, H, 128), dtype=torch.bfloat16 if w.dtype == "bf16" else torch.float32)
    xv_new = torch.zeros_like(xk_new)
    for b in range(B):
        n = case.lens[b]
        xk, xv = case.x_tokens(b, "k"), case.x_tokens(b, "v")
        P.aatc_encode(pk, H, xk, n - 1, H * 128, P.LAYOUT_RECORDS, kc[b], ka[b], cap, 0)
        P.aatc_encode(pv, H, xv, n - 1, H * 128, P.LAYOUT_TILES, vc[b], va[b], cap, 0)
        xk_new[b], xv_new[b] = xk[n - 1].cpu(), xv[n - 1].cpu()
        del xk, xv
    q = stored_to_torch(np.stack(case.q)).cuda()
    lens = torch.tensor(case.lens, dtype=torch.int32, device="cuda")
    out = torch.full((B, HQ, 128), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.zeros(P.aatc_decode_workspace_bytes(B, HQ, H, cap), dtype=torch.uint8,
                     device="cuda")
    P.aatc_append_decode_attention(pk, pv, B, HQ, H, q, xk_new.cuda(), xv_new.cuda(), kc, ka,
                                   vc, va, lens, cap, rk, rv, 1 / np.sqrt(128), out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert np.all(np.isfinite(got))
    g = HQ // H
    for b, h in spec["sample"]:
        n = case.lens[b]
        ok_, oa = case.oracle_encode(b, h, "k")
        ov_, ova = case.oracle_encode(b, h, "v")
        np.testing.assert_array_equal(kc[b, h, :n].cpu().numpy(), ok_)
        np.testing.assert_array_equal(ka[b, h, :n].cpu().numpy().view(np.uint16), oa.view(np.uint16))
        np.testing.assert_array_equal(ora.tiles_to_records(vc[b, h].cpu().numpy(), rv)[:n], ov_)
        np.testing.assert_array_equal(va[b, h, :n].cpu().numpy().view(np.uint16), ova.view(np.uint16))
        kh = ora.decode_tokens(ok_, oa, case.cal_k[h])
        vh = ora.decode_tokens(ov_, ova, case.cal_v[h])
        q32 = w.as_f32(case.q[b])[h * g:(h + 1) * g]
        ref = ora.softmax_attention(q32, kh, vh, 1 / np.sqrt(128))
        err = _assert_heads_close(got[b, h * g:(h + 1) * g], ref, f"seq {b} kv head {h}")
        _log(f"  seq {b} kv head {h}: worst query head rel_l2 {err:.3e}")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("avg_bits", [2.75, 4.0])
def test_full_size_prefill_encode_sampled(avg_bits):
    """The prefill workload at full size (65536 new tokens x 8 KV heads, one aatc_encode
    per tensor, as the benchmark launches it): every head's key records, value tiles and
    scales are bit-exact against the oracle at both budgets."""
    full = workload(4)
    _log(f"[full] prefill encode: {full.n_tokens} tokens, {full.n_kv_heads} heads, "
         f"{avg_bits} bits")
    case = Case(cfg=4, n_tokens=full.n_tokens, avg_bits=avg_bits)
    w = case.w
    H, cap, n = w.n_kv_heads, case.cap, case.lens[0]
    rk, rv = case.cal_k[0].record_bytes, case.cal_v[0].record_bytes
    pk, pv = device_params(case.cal_k), device_params(case.cal_v)
    kc, vc = record_cache(H, cap, rk), tile_cache(H, cap, rv)
    ka, va = alpha_cache(H, cap), alpha_cache(H, cap)
    xk, xv = case.x_tokens(0, "k"), case.x_tokens(0, "v")
    P.aatc_encode(pk, H, xk, n, H * 128, P.LAYOUT_RECORDS, kc, ka, cap, 0)
    P.aatc_encode(pv, H, xv, n, H * 128, P.LAYOUT_TILES, vc, va, cap, 0)
    torch.cuda.synchronize()
    for h in range(H):
        ok_, oa = case.oracle_encode(0, h, "k")
        ov_, ova = case.oracle_encode(0, h, "v")
        got = kc[h, :n].cpu().numpy()
        bad = np.argwhere(np.any(got != ok_, axis=1))
        assert bad.size == 0, f"head {h}: key records differ at tokens {bad[:5].ravel()}"
        np.testing.assert_array_equal(ka[h, :n].cpu().numpy().view(np.uint16), oa.view(np.uint16))
        np.testing.assert_array_equal(vc[h].cpu().numpy(), oracle_tiles(ov_, cap))
        np.testing.assert_array_equal(va[h, :n].cpu().numpy().view(np.uint16), ova.view(np.uint16))
        _log(f"  head {h}: records {rk} / {rv} B bit-exact")
