"""GPU parity of the head-group path (Sec. 5.1, the remark on head groups; Sec. 5.2, one
token scale per head group; Sec. 6 setup: G = 2 groups of four KV heads for Llama, one
group of four for Qwen) against the oracle, through the C ABI.

Bar: bit-exact records and fp16 token scales against ``oracle.groups.encode_group``;
decode outputs within 2e-3 relative L2 (and max-abs) per query head of
``oracle.groups.group_attention`` over the oracle's own records.
"""
import numpy as np
import pytest
import torch

import paper_2608_14191_amd as P
from kvsynth import workload
from oracle import groups as og

from helpers import alpha_cache, group_device_params, rel_l2, stored_to_torch

pytestmark = pytest.mark.gpu

TOL = 2e-3


def _log(msg):
    print(msg, flush=True)


def _assert_heads_close(got, ref, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    worst = 0.0
    for j in range(ref.shape[0]):
        err = rel_l2(got[j], ref[j])
        worst = max(worst, err)
        assert err <= TOL, f"{what} query head {j}: rel L2 {err:.3e}"
        assert np.abs(got[j] - ref[j]).max() <= TOL * np.abs(ref[j]).max(), f"{what} head {j}"
    return worst


class GCase:
    """Synthetic group workload: calibrations per group from the configuration's
    calibration draws, cached tokens per sequence."""

    def __init__(self, cfg, gkv, lens, avg_bits=None, quantizer="midtread", b_max=8,
                 **overrides):
        self.w = workload(cfg, n_tokens=max(max(lens), 1), batch=len(lens), **overrides)
        w = self.w
        self.gkv, self.lens = gkv, list(lens)
        self.H, self.HQ = w.n_kv_heads, w.n_q_heads
        self.ng = self.H // gkv
        avg = w.cfg["avg_bits"][0] if avg_bits is None else avg_bits
        self.cal = {}
        for kind in ("k", "v"):
            self.cal[kind] = [
                og.calibrate_group(
                    np.concatenate([w.calib(h, kind) for h in range(g * gkv, (g + 1) * gkv)],
                                   axis=1), avg, b_max=b_max, quantizer=quantizer)
                for g in range(self.ng)]
        self.R = {k: self.cal[k][0].record_bytes for k in ("k", "v")}
        self.cap = max(64, -(-max(lens) // 64) * 64)
        self._tok = {}

    def tokens(self, b, kind):
        """Stored tokens [n, H, 128] of sequence b (bf16 bits or fp32)."""
        key = (b, kind)
        if key not in self._tok:
            n = self.lens[b]
            self._tok[key] = np.stack([self.w.cache(b, h, kind, n=n) for h in range(self.H)],
                                      axis=1)
        return self._tok[key]

    def oracle_encode(self, b, kind, g, x=None):
        x = self.tokens(b, kind) if x is None else x
        xg = og.group_tokens(self.w.as_f32(x), g, self.gkv)
        rec, a16, _ = og.encode_group(xg, self.cal[kind][g])
        return rec, a16

    def gpu_encode(self, params, kind, tokens=None):
        B, ng, cap = len(self.lens), self.ng, self.cap
        codes = torch.zeros((B, ng, cap, self.R[kind]), dtype=torch.uint8, device="cuda")
        alpha = alpha_cache(ng, cap, batch=B)
        for b in range(B):
            n = self.lens[b]
            if n == 0:
                continue
            x = stored_to_torch(self.tokens(b, kind) if tokens is None else tokens[b]).cuda()
            P.aatc_group_encode(params, ng, self.gkv, x.contiguous(), n, self.H * 128, codes[b],
                                alpha[b], cap, 0)
        return codes, alpha

    def queries(self):
        return np.stack([self.w.queries(b) for b in range(len(self.lens))])


def _run(case, tokens_k=None, tokens_v=None, check_codes=True):
    pk, pv = group_device_params(case.cal["k"]), group_device_params(case.cal["v"])
    kc, ka = case.gpu_encode(pk, "k", tokens_k)
    vc, va = case.gpu_encode(pv, "v", tokens_v)
    torch.cuda.synchronize()
    B = len(case.lens)
    orec = {}
    for b in range(B):
        n = case.lens[b]
        for kind, (c, a, toks) in (("k", (kc, ka, tokens_k)), ("v", (vc, va, tokens_v))):
            for g in range(case.ng):
                if n == 0:
                    orec[(b, kind, g)] = (np.zeros((0, case.R[kind]), np.uint8),
                                          np.zeros(0, np.float16))
                    continue
                rec, a16 = case.oracle_encode(b, kind, g, None if toks is None else toks[b])
                orec[(b, kind, g)] = (rec, a16)
                if check_codes:
                    got = c[b, g, :n].cpu().numpy()
                    bad = np.argwhere(np.any(got != rec, axis=1))
                    assert bad.size == 0, f"seq {b} {kind} group {g}: records differ at {bad[:5].ravel()}"
                    np.testing.assert_array_equal(a[b, g, :n].cpu().numpy().view(np.uint16),
                                                  a16.view(np.uint16))
    q = case.queries()
    qt = stored_to_torch(q).cuda()
    lens = torch.tensor(case.lens, dtype=torch.int32, device="cuda")
    out = torch.full((B, case.HQ, 128), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(P.aatc_group_decode_workspace_bytes(B, case.HQ, case.H, case.gkv, case.cap),
                     dtype=torch.uint8, device="cuda")
    P.aatc_group_decode_attention(pk, pv, B, case.HQ, case.H, case.gkv, qt, kc, ka, vc, va, lens,
                                  case.cap, case.R["k"], case.R["v"], 1 / np.sqrt(128), out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    worst = 0.0
    for b in range(B):
        n = case.lens[b]
        if n == 0:
            assert np.all(got[b] == 0)
            continue
        ref = og.group_attention(case.w.as_f32(q[b]), case.H, case.gkv, case.cal["k"],
                                 case.cal["v"], [orec[(b, "k", g)][0] for g in range(case.ng)],
                                 [orec[(b, "k", g)][1] for g in range(case.ng)],
                                 [orec[(b, "v", g)][0] for g in range(case.ng)],
                                 [orec[(b, "v", g)][1] for g in range(case.ng)], n)
        worst = max(worst, _assert_heads_close(got[b], ref, f"seq {b} len {n}"))
    return got, worst, (pk, pv, kc, ka, vc, va)


CASES = {
    # Llama shape: 8 KV heads in 2 groups of 4 (512 channels, 16 query heads per group);
    # lengths across the 256-token splits and the 64-token chunks, and a one-token row
    "llama_g2": dict(cfg=2, gkv=4, lens=[300, 257, 1]),
    # Qwen shape: 4 KV heads in one group, 28 query heads per group
    "qwen_g1": dict(cfg=3, gkv=4, lens=[200, 64]),
    # groups of two (256 channels), the midrise reading, 6 bits with widths up to 16
    "gkv2_midrise_6bit": dict(cfg=2, gkv=2, lens=[130, 0], avg_bits=6.0,
                              quantizer="midrise", b_max=16),
    # groups of three (384 channels), fp32 tokens and queries, query-weighting off
    "gkv3_fp32": dict(cfg=1, gkv=3, lens=[96], n_kv_heads=6, n_q_heads=12),
    # 8 bits over 512 channels: 512-byte records, the split kernel that stages 64-token
    # chunks (the whole split's records do not fit in LDS)
    "llama_g2_8bit_records_512b": dict(cfg=2, gkv=4, lens=[300, 129], avg_bits=8.0),
    # key codes of 12 bits (the widest the matrix-core split takes: exact in fp16)
    "gkv2_12bit_codes": dict(cfg=2, gkv=2, lens=[200, 45], avg_bits=8.0, b_max=12),
    # key codes of 15 bits: the matrix-core split kernel runs its VALU body instead
    "gkv2_15bit_codes": dict(cfg=2, gkv=2, lens=[140, 33], avg_bits=10.0, b_max=16),
}


@pytest.mark.timeout(300)
@pytest.mark.parametrize("name", list(CASES))
def test_group_encode_bit_exact_and_decode_parity(name):
    spec = dict(CASES[name])
    cfg, gkv, lens = spec.pop("cfg"), spec.pop("gkv"), spec.pop("lens")
    _log(f"[group] {name}: cfg {cfg}, gkv {gkv}, lens {lens}")
    case = GCase(cfg, gkv, lens, **spec)
    _, worst, _ = _run(case)
    _log(f"  worst query head rel_l2 {worst:.3e}")


@pytest.mark.timeout(300)
def test_group_of_one_head_matches_the_per_head_path():
    """gkv = 1: the group path is the per-head method, so its key records and scales equal
    those of aatc_encode (RECORDS) and its outputs those of aatc_decode_attention."""
    from helpers import device_params, record_cache, tile_cache
    case = GCase(2, 1, [200])
    _log("[group] gkv 1 against the per-head path")
    got, _, (pk, pv, kc, ka, vc, va) = _run(case)
    from oracle import aatc as ora
    cal_k = [ora.calibrate(case.w.calib(h, "k"), case.w.cfg["avg_bits"][0]) for h in range(8)]
    cal_v = [ora.calibrate(case.w.calib(h, "v"), case.w.cfg["avg_bits"][0]) for h in range(8)]
    hk, hv = device_params(cal_k), device_params(cal_v)
    cap, n = case.cap, 200
    kc2, vc2 = record_cache(8, cap, case.R["k"], batch=1), tile_cache(8, cap, case.R["v"], batch=1)
    ka2, va2 = alpha_cache(8, cap, batch=1), alpha_cache(8, cap, batch=1)
    xk = stored_to_torch(case.tokens(0, "k")).cuda().contiguous()
    xv = stored_to_torch(case.tokens(0, "v")).cuda().contiguous()
    P.aatc_encode(hk, 8, xk, n, 8 * 128, P.LAYOUT_RECORDS, kc2[0], ka2[0], cap, 0)
    P.aatc_encode(hv, 8, xv, n, 8 * 128, P.LAYOUT_TILES, vc2[0], va2[0], cap, 0)
    torch.cuda.synchronize()
    assert torch.equal(kc[0, :, :n].cpu(), kc2[0, :, :n].cpu())
    assert torch.equal(ka[0, :, :n].cpu(), ka2[0, :, :n].cpu())
    assert torch.equal(va[0, :, :n].cpu(), va2[0, :, :n].cpu())
    q = stored_to_torch(case.queries()).cuda()
    lens = torch.tensor([n], dtype=torch.int32, device="cuda")
    out = torch.zeros((1, 32, 128), dtype=torch.float32, device="cuda")
    ws = torch.zeros(P.aatc_decode_workspace_bytes(1, 32, 8, cap), dtype=torch.uint8,
                     device="cuda")
    P.aatc_decode_attention(hk, hv, 1, 32, 8, q, kc2, ka2, vc2, va2, lens, cap, case.R["k"],
                            case.R["v"], 1 / np.sqrt(128), out, ws)
    torch.cuda.synchronize()
    for j in range(32):
        assert rel_l2(got[0, j], out[0, j].cpu().numpy()) <= 1e-5, j


@pytest.mark.timeout(300)
def test_group_edge_tokens_bit_exact():
    """A zero token, a scale that rounds to an fp16 subnormal, a saturating scale and
    tokens with elements far below the largest (not exact in 22-bit fixed point, so the
    fp64 sums are not exact and the interval test or the exact accumulator decides)."""
    case = GCase(2, 4, [80])
    toks = {}
    for kind in ("k", "v"):
        x = case.w.as_f32(case.tokens(0, kind)).copy()
        x[5] = 0.0
        x[17] *= 2.0 ** -20
        x[33] *= 2.0 ** 17
        x[50, :, 3] = 2.0 ** -30
        x[51, :2, :] *= 2.0 ** -40
        x[52, 1, 7] = 2.0 ** 20
        from kvsynth.gen import f32_to_bf16_bits
        toks[kind] = [f32_to_bf16_bits(x.astype(np.float32))]
    _log("[group] edge tokens")
    _run(case, tokens_k=toks["k"], tokens_v=toks["v"])


@pytest.mark.timeout(300)
def test_group_decode_repeatable_and_reports_mismatched_records():
    case = GCase(3, 4, [150])
    got, _, (pk, pv, kc, ka, vc, va) = _run(case)
    q = stored_to_torch(case.queries()).cuda()
    lens = torch.tensor(case.lens, dtype=torch.int32, device="cuda")
    ws = torch.empty(P.aatc_group_decode_workspace_bytes(1, case.HQ, case.H, 4, case.cap),
                     dtype=torch.uint8, device="cuda")
    out = torch.empty((1, case.HQ, 128), dtype=torch.float32, device="cuda")
    P.aatc_group_decode_attention(pk, pv, 1, case.HQ, case.H, 4, q, kc, ka, vc, va, lens,
                                  case.cap, case.R["k"], case.R["v"], 1 / np.sqrt(128), out, ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy(), got)
    # caches of another record size than the parameter blocks give NaN outputs
    kc_wide = torch.zeros((1, 1, case.cap, case.R["k"] + 4), dtype=torch.uint8, device="cuda")
    P.aatc_group_decode_attention(pk, pv, 1, case.HQ, case.H, 4, q, kc_wide, ka, vc, va, lens,
                                  case.cap, case.R["k"] + 4, case.R["v"], 1 / np.sqrt(128), out,
                                  ws)
    torch.cuda.synchronize()
    assert torch.isnan(out).all()


@pytest.mark.timeout(600)
def test_full_size_llama_groups():
    """The Llama shape at full length as the benchmark launches it: 32768 tokens, 8 KV heads
    in two groups of four, 32 query heads, 2.75 bits.  Every record and scale of group 0 is
    compared with the oracle (and sampled tokens of group 1), and group 0's 16 query heads
    with the oracle's attention over the whole length."""
    n = 32768
    case = GCase(2, 4, [n])
    _log(f"[group] full size: {n} tokens, 2 groups of 4 KV heads")
    pk, pv = group_device_params(case.cal["k"]), group_device_params(case.cal["v"])
    kc, ka = case.gpu_encode(pk, "k")
    vc, va = case.gpu_encode(pv, "v")
    q = case.queries()
    lens = torch.tensor([n], dtype=torch.int32, device="cuda")
    out = torch.empty((1, 32, 128), dtype=torch.float32, device="cuda")
    ws = torch.empty(P.aatc_group_decode_workspace_bytes(1, 32, 8, 4, case.cap),
                     dtype=torch.uint8, device="cuda")
    P.aatc_group_decode_attention(pk, pv, 1, 32, 8, 4, stored_to_torch(q).cuda(), kc, ka, vc,
                                  va, lens, case.cap, case.R["k"], case.R["v"],
                                  1 / np.sqrt(128), out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert np.all(np.isfinite(got))
    orec = {}
    for kind, c, a in (("k", kc, ka), ("v", vc, va)):
        rec, a16 = case.oracle_encode(0, kind, 0)
        orec[kind] = (rec, a16)
        np.testing.assert_array_equal(c[0, 0, :n].cpu().numpy(), rec)
        np.testing.assert_array_equal(a[0, 0, :n].cpu().numpy().view(np.uint16), a16.view(np.uint16))
        idx = np.r_[0:64, n // 2:n // 2 + 64, n - 64:n]
        x1 = case.tokens(0, kind)[idx]
        r1, a1 = case.oracle_encode(0, kind, 1, x=x1)
        np.testing.assert_array_equal(c[0, 1, idx].cpu().numpy(), r1)
        np.testing.assert_array_equal(a[0, 1, idx].cpu().numpy().view(np.uint16), a1.view(np.uint16))
        _log(f"  {kind}: group 0 records bit-exact, group 1 sampled bit-exact")
    # group 0 = KV heads 0..3 = query heads 0..15
    from oracle import aatc as ora
    kh = ora.decode_tokens(orec["k"][0], orec["k"][1], case.cal["k"][0])
    vh = ora.decode_tokens(orec["v"][0], orec["v"][1], case.cal["v"][0])
    q32 = case.w.as_f32(q[0])
    for j in range(16):
        k = j // 4
        blk = slice(128 * k, 128 * (k + 1))
        ref = ora.softmax_attention(q32[j:j + 1], kh[:, blk], vh[:, blk], 1 / np.sqrt(128))
        _assert_heads_close(got[0, j:j + 1], ref, f"query head {j}")
    _log("  group 0 query heads within tolerance")


@pytest.mark.timeout(300)
def test_group_incremental_appends_match_bulk():
    """Tokens appended a few at a time at increasing positions (as decode steps append them)
    give the same records and scales as one bulk encode, and leave the other positions of
    the cache untouched."""
    case = GCase(2, 4, [150])
    pk = group_device_params(case.cal["k"])
    bulk, abulk = case.gpu_encode(pk, "k")
    x = stored_to_torch(case.tokens(0, "k")).cuda().contiguous()
    cap, ng = case.cap, case.ng
    inc = torch.full((ng, cap, case.R["k"]), 0xA5, dtype=torch.uint8, device="cuda")
    ainc = torch.full((ng, cap), 0x1234, dtype=torch.int16, device="cuda")
    pos = 0
    for n in (1, 2, 5, 16, 17, 1, 40, 68):
        P.aatc_group_encode(pk, ng, 4, x[pos:pos + n], n, 8 * 128, inc, ainc, cap, pos)
        pos += n
    assert pos == 150
    torch.cuda.synchronize()
    assert torch.equal(inc[:, :150].cpu(), bulk[0, :, :150].cpu())
    assert torch.equal(ainc[:, :150].cpu(), abulk[0, :, :150].cpu())
    assert bool((inc[:, 150:] == 0xA5).all()) and bool((ainc[:, 150:] == 0x1234).all())


@pytest.mark.timeout(300)
def test_group_end_to_end_with_host_calibration():
    """aatc_calibrate_group (host C++) -> aatc_group_params_pack -> encode -> decode against
    the oracle pipeline on the oracle's own calibrations (groups of two, 256 channels)."""
    case = GCase(2, 2, [260, 90])
    w = case.w
    abi = {kind: [P.aatc_calibrate_group(
        np.concatenate([w.calib(h, kind) for h in range(2 * g, 2 * g + 2)], axis=1),
        w.cfg["avg_bits"][0]) for g in range(case.ng)] for kind in ("k", "v")}
    for kind in ("k", "v"):
        assert abi[kind][0].record_bytes == case.R[kind]
    pk, pv = group_device_params(abi["k"]), group_device_params(abi["v"])
    kc, ka = case.gpu_encode(pk, "k")
    vc, va = case.gpu_encode(pv, "v")
    q = case.queries()
    lens = torch.tensor(case.lens, dtype=torch.int32, device="cuda")
    out = torch.empty((2, case.HQ, 128), dtype=torch.float32, device="cuda")
    ws = torch.empty(P.aatc_group_decode_workspace_bytes(2, case.HQ, case.H, 2, case.cap),
                     dtype=torch.uint8, device="cuda")
    P.aatc_group_decode_attention(pk, pv, 2, case.HQ, case.H, 2, stored_to_torch(q).cuda(), kc,
                                  ka, vc, va, lens, case.cap, case.R["k"], case.R["v"],
                                  1 / np.sqrt(128), out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    for b in range(2):
        n = case.lens[b]
        recs = {(kind, g): case.oracle_encode(b, kind, g) for kind in ("k", "v")
                for g in range(case.ng)}
        ref = og.group_attention(case.w.as_f32(q[b]), case.H, 2, case.cal["k"], case.cal["v"],
                                 [recs[("k", g)][0] for g in range(case.ng)],
                                 [recs[("k", g)][1] for g in range(case.ng)],
                                 [recs[("v", g)][0] for g in range(case.ng)],
                                 [recs[("v", g)][1] for g in range(case.ng)], n)
        _assert_heads_close(got[b], ref, f"seq {b}")


@pytest.mark.timeout(300)
def test_group_long_sequence_of_one_repeated_token():
    """300000 copies of one token (1172 splits: the merge takes its split weights in two
    passes): every score is equal, so each query head's output is its KV head's block of
    the token's reconstruction, which the oracle gives from that one token."""
    n = 300_000
    case = GCase(3, 4, [1])
    H, HQ, gkv, cap = case.H, case.HQ, 4, n + 32
    tok_k, tok_v = case.tokens(0, "k")[:1], case.tokens(0, "v")[:1]
    pk, pv = group_device_params(case.cal["k"]), group_device_params(case.cal["v"])
    caches = {}
    for kind, tok, params in (("k", tok_k, pk), ("v", tok_v, pv)):
        x = stored_to_torch(tok).cuda().expand(n, H, 128).contiguous()
        codes = torch.zeros((1, 1, cap, case.R[kind]), dtype=torch.uint8, device="cuda")
        alpha = alpha_cache(1, cap, batch=1)
        P.aatc_group_encode(params, 1, gkv, x, n, H * 128, codes[0], alpha[0], cap, 0)
        caches[kind] = (codes, alpha)
        del x
    q = case.queries()[:1]
    lens = torch.tensor([n], dtype=torch.int32, device="cuda")
    out = torch.empty((1, HQ, 128), dtype=torch.float32, device="cuda")
    ws = torch.empty(P.aatc_group_decode_workspace_bytes(1, HQ, H, gkv, cap), dtype=torch.uint8,
                     device="cuda")
    P.aatc_group_decode_attention(pk, pv, 1, HQ, H, gkv, stored_to_torch(q).cuda(),
                                  caches["k"][0], caches["k"][1], caches["v"][0],
                                  caches["v"][1], lens, cap, case.R["k"], case.R["v"],
                                  1 / np.sqrt(128), out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()[0]
    rec, a16 = case.oracle_encode(0, "v", 0, x=tok_v)
    from oracle import aatc as ora
    vhat = ora.decode_tokens(rec, a16, case.cal["v"][0])[0]            # [512]
    gq = HQ // H
    for j in range(HQ):
        k = j // gq
        ref = vhat[128 * k:128 * (k + 1)]
        assert rel_l2(got[j], ref) <= 1e-5, j
