"""GPU parity of every encode path on the tokens that stress the exact transform.

The transform of a token is the exact product with the stored transform, rounded once
(Sec. 5.1; Alg. 1 "project").  The matrix-core encode computes it from a fixed-point form
of the token that is exact for most tokens, certifies the others, and redoes the few it
cannot certify with an exact routine; the per-token and VALU kernels and the decode
kernel's fused append take their own routes.  These tests put the same tokens through all
of them:
  - edge tokens: all zero, a scale that rounds to an fp16 subnormal, a saturating scale
    (alpha = 65504), one element far below the others (not exact in fixed point);
  - a crafted transform whose channel-0 sum lies at an fp16 halfway point of the scale up
    to a term of 2^-24 that the fixed-point form loses: only the exact routine gets alpha
    (and so every code) right.
Bar: bit-exact records, value tiles and fp16 scales against the oracle.
"""
import numpy as np
import pytest
import torch

import paper_2608_14191_amd as P
from kvsynth import workload
from kvsynth.gen import bf16_bits_to_f32, f32_to_bf16_bits
from oracle import aatc as ora

from helpers import (alpha_cache, device_params, oracle_tiles, record_cache, rel_l2,
                     stored_to_torch, tile_cache)

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)


def _bf16(a):
    return f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


def _edge_tokens(base_bits: np.ndarray) -> np.ndarray:
    """bf16 tokens [n, H, 128] with edge rows planted at fixed positions."""
    x = bf16_bits_to_f32(base_bits).copy()
    x[5] = 0.0                                  # zero token: alpha = 0, all codes 0
    x[17] *= 2.0 ** -20                         # alpha rounds to an fp16 subnormal
    x[33] *= 2.0 ** 17                          # alpha saturates at 65504
    x[50, :, 3] = 2.0 ** -30                    # one element far below the others
    x[51, :, :64] *= 2.0 ** -40                 # half the token far below the other half
    return _bf16(x)


def _crafted_calibration() -> "ora.Calibration":
    """Channels 0..63 at 4 bits with s = 1, 64..127 dropped; T = I except column 0 =
    e0 + 2^-10 e2 + e3."""
    d = 128
    t = np.eye(d, dtype=np.float32)
    t[2, 0] = 2.0 ** -10
    t[3, 0] = 1.0
    bits = np.array([4] * 64 + [0] * 64, dtype=np.int64)
    s16 = np.where(bits > 0, 1.0, 0.0).astype(np.float16)
    return ora.Calibration(d=d, budget=256, record_bytes=32, d_active=64, bits=bits,
                           perm=np.arange(d), T64=t.astype(np.float64), T32=t, s16=s16,
                           sigma2=np.ones(d), weight=np.ones(d), bits_eig=bits)


def _crafted_tokens(n: int, H: int, seed: int) -> np.ndarray:
    """Tokens whose channel-0 sum is 1 + 2^-11 (+-) 2^-24 (1 + 2^-7): the fixed-point form
    drops the last term (far below the token's largest element), and with it the fp32
    rounding that decides the fp16 scale (the halfway point 1 + 2^-11 ties to 1)."""
    rng = np.random.default_rng(seed)
    x = (rng.uniform(-0.25, 0.25, size=(n, H, 128))).astype(np.float32)
    x[:, :, 0] = 1.0
    x[:, :, 2] = 0.5
    sign = np.where(np.arange(n) % 2 == 0, 1.0, -1.0)[:, None]
    x[:, :, 3] = sign * 2.0 ** -24 * (1 + 2.0 ** -7)
    return _bf16(x)


def _oracle(cal, x_bits_h):
    rec, a16, _ = ora.encode(bf16_bits_to_f32(x_bits_h), cal)
    return rec, a16


def _check(cals, x_bits, rec_k, alpha, layout, cap, lo=0, hi=None):
    """Compare one tensor's cache (all heads) with the oracle for tokens [lo, hi)."""
    n = x_bits.shape[0] if hi is None else hi
    for h, cal in enumerate(cals):
        want_rec, want_a = _oracle(cal, x_bits[:n, h])
        if layout == P.LAYOUT_RECORDS:
            got = rec_k[h, :n].cpu().numpy()
        else:
            got = ora.tiles_to_records(rec_k[h].cpu().numpy(), cal.record_bytes)[:n]
        bad = np.argwhere(np.any(got[lo:n] != want_rec[lo:n], axis=1)).ravel() + lo
        assert bad.size == 0, f"head {h}: records differ at tokens {bad[:8]}"
        ga = alpha[h, lo:n].cpu().numpy().view(np.uint16)
        np.testing.assert_array_equal(ga, want_a[lo:n].view(np.uint16), err_msg=f"head {h}")


def _encode_paths(pp, cals, x_bits, layout, cap):
    """Encode [n, H, 128] bf16 tokens by the three encode paths; returns their caches."""
    H = x_bits.shape[1]
    n = x_bits.shape[0]
    rb = cals[0].record_bytes
    x = torch.from_numpy(x_bits.view(np.int16).copy()).view(torch.bfloat16).cuda()
    out = {}
    mk = (lambda: record_cache(H, cap, rb)) if layout == P.LAYOUT_RECORDS else \
        (lambda: tile_cache(H, cap, rb))
    # matrix-core kernel: aligned rows, more than 16 tokens
    c, a = mk(), alpha_cache(H, cap)
    P.aatc_encode(pp, H, x, n, H * 128, layout, c, a, cap, 0)
    out["mfma"] = (c, a)
    # VALU kernel: rows padded by one element (not 16-byte aligned)
    xp = torch.zeros((n, H * 128 + 1), dtype=x.dtype, device=x.device)
    xp[:, :H * 128] = x.reshape(n, H * 128)
    c, a = mk(), alpha_cache(H, cap)
    P.aatc_encode(pp, H, xp, n, H * 128 + 1, layout, c, a, cap, 0)
    out["valu"] = (c, a)
    # per-token kernel: appends of at most 16 tokens
    c, a = mk(), alpha_cache(H, cap)
    for p0 in range(0, n, 16):
        k = min(16, n - p0)
        P.aatc_encode(pp, H, x[p0:], k, H * 128, layout, c, a, cap, p0)
    out["token"] = (c, a)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("kind", ["k", "v"])
def test_edge_tokens_every_encode_path(kind):
    w = workload(2, n_tokens=192)
    H, n, cap = w.n_kv_heads, 192, 192
    cals = [ora.calibrate(w.calib(h, kind), 2.75) for h in range(H)]
    x_bits = _edge_tokens(np.stack([w.cache(0, h, kind) for h in range(H)], axis=1))
    pp = device_params(cals)
    layout = P.LAYOUT_RECORDS if kind == "k" else P.LAYOUT_TILES
    for path, (c, a) in _encode_paths(pp, cals, x_bits, layout, cap).items():
        _log(f"[edge] {kind} {path}")
        _check(cals, x_bits, c, a, layout, cap)
    # the planted scales are what the test means them to be
    _, a_sub = _oracle(cals[0], x_bits[:, 0])
    assert 0 < a_sub[17].astype(np.float32) < 2.0 ** -14
    assert a_sub[33].astype(np.float32) == 65504.0 and a_sub[5] == 0


@pytest.mark.parametrize("kind", ["k", "v"])
def test_certificate_failures_take_the_exact_route(kind):
    """Every token of the crafted transform fails the scale certificate in the
    matrix-core kernel; all paths must still give the oracle's scales and codes."""
    H, n, cap = 2, 96, 128
    cals = [_crafted_calibration() for _ in range(H)]
    x_bits = _crafted_tokens(n, H, seed=1 if kind == "k" else 2)
    # the oracle's scales alternate 1 + 2^-10 (sum above the tie) and 1 (below)
    _, a16 = _oracle(cals[0], x_bits[:, 0])
    np.testing.assert_array_equal(a16[:4].astype(np.float32), [1 + 2.0 ** -10, 1, 1 + 2.0 ** -10, 1])
    pp = device_params(cals)
    layout = P.LAYOUT_RECORDS if kind == "k" else P.LAYOUT_TILES
    for path, (c, a) in _encode_paths(pp, cals, x_bits, layout, cap).items():
        _log(f"[crafted] {kind} {path}")
        _check(cals, x_bits, c, a, layout, cap)


@pytest.mark.parametrize("which", ["edge", "crafted"])
def test_fused_append_exact_transform(which):
    """The decode kernel's fused append encodes the step's token: edge tokens and crafted
    near-tie tokens (certificate failures in the merging workgroup) give the oracle's
    codes, and the attention output stays within tolerance."""
    if which == "edge":
        w = workload(2, n_tokens=256)
        H, HQ = w.n_kv_heads, w.n_q_heads
        cal_k = [ora.calibrate(w.calib(h, "k"), 2.75) for h in range(H)]
        cal_v = [ora.calibrate(w.calib(h, "v"), 2.75) for h in range(H)]
        xk = _edge_tokens(np.stack([w.cache(0, h, "k", n=256) for h in range(H)], axis=1))
        xv = _edge_tokens(np.stack([w.cache(0, h, "v", n=256) for h in range(H)], axis=1))
        q = np.stack([w.queries(0)])
        new_pos = [5, 17, 33, 50, 51, 100]        # each edge token appended in its step
    else:
        H, HQ = 2, 8
        cal_k = [_crafted_calibration() for _ in range(H)]
        cal_v = [_crafted_calibration() for _ in range(H)]
        xk = _crafted_tokens(256, H, seed=3)
        xv = _crafted_tokens(256, H, seed=4)
        rng = np.random.default_rng(5)
        q = _bf16(rng.standard_normal((1, HQ, 128)) * 2)
        new_pos = [0, 1, 63, 64, 200]
    cap = 256
    rk, rv = cal_k[0].record_bytes, cal_v[0].record_bytes
    pk, pv = device_params(cal_k), device_params(cal_v)
    B = len(new_pos)
    kc, vc = record_cache(H, cap, rk, batch=B), tile_cache(H, cap, rv, batch=B)
    ka, va = alpha_cache(H, cap, batch=B), alpha_cache(H, cap, batch=B)
    xk_t = torch.from_numpy(xk.view(np.int16).copy()).view(torch.bfloat16).cuda()
    xv_t = torch.from_numpy(xv.view(np.int16).copy()).view(torch.bfloat16).cuda()
    for b, p in enumerate(new_pos):
        if p > 0:
            P.aatc_encode(pk, H, xk_t, p, H * 128, P.LAYOUT_RECORDS, kc[b], ka[b], cap, 0)
            P.aatc_encode(pv, H, xv_t, p, H * 128, P.LAYOUT_TILES, vc[b], va[b], cap, 0)
    xk_new = torch.stack([xk_t[p] for p in new_pos])
    xv_new = torch.stack([xv_t[p] for p in new_pos])
    qt = torch.from_numpy(np.repeat(q, B, axis=0).view(np.int16).copy()).view(torch.bfloat16).cuda()
    lens = torch.tensor([p + 1 for p in new_pos], dtype=torch.int32, device="cuda")
    out = torch.full((B, HQ, 128), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.zeros(P.aatc_decode_workspace_bytes(B, HQ, H, cap), dtype=torch.uint8, device="cuda")
    P.aatc_append_decode_attention(pk, pv, B, HQ, H, qt, xk_new, xv_new, kc, ka, vc, va, lens,
                                   cap, rk, rv, 1 / np.sqrt(128), out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    q32 = bf16_bits_to_f32(q[0])
    for b, p in enumerate(new_pos):
        n = p + 1
        _log(f"[append {which}] token {p}")
        enc_k = [_oracle(cal_k[h], xk[:n, h]) for h in range(H)]
        enc_v = [_oracle(cal_v[h], xv[:n, h]) for h in range(H)]
        for h in range(H):
            np.testing.assert_array_equal(kc[b, h, :n].cpu().numpy(), enc_k[h][0])
            np.testing.assert_array_equal(ka[b, h, :n].cpu().numpy().view(np.uint16),
                                          enc_k[h][1].view(np.uint16))
            np.testing.assert_array_equal(ora.tiles_to_records(vc[b, h].cpu().numpy(), rv)[:n],
                                          enc_v[h][0])
            np.testing.assert_array_equal(va[b, h, :n].cpu().numpy().view(np.uint16),
                                          enc_v[h][1].view(np.uint16))
        ref = ora.decode_attention(q32, cal_k, cal_v, [e[0] for e in enc_k], [e[1] for e in enc_k],
                                   [e[0] for e in enc_v], [e[1] for e in enc_v], n)
        g = HQ // H
        for j in range(HQ):
            if np.linalg.norm(ref[j]) > 0:
                assert rel_l2(got[b, j], ref[j]) <= 2e-3, (p, j, rel_l2(got[b, j], ref[j]))
            else:
                assert np.abs(got[b, j]).max() <= 1e-30, (p, j)
