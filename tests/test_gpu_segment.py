"""GPU parity of the full-precision segment (Sec. 6 experimental setup; App. E "AATC": the
first 4 tokens and the recent window of 128 tokens at input precision, the oldest 16 window
tokens quantized whenever the window is full): aatc_decode_attention_segmented over caches
laid out by that policy, against the oracle's exact attention over the union."""
import numpy as np
import pytest
import torch

import paper_2608_14191_amd as P
from kvsynth import workload
from oracle import aatc as ora

from helpers import alpha_cache, device_params, record_cache, rel_l2, stored_to_torch, tile_cache

pytestmark = pytest.mark.gpu
SEG_CAP = 4 + 128


def _log(msg):
    print(msg, flush=True)


def _run(w, cal_k, cal_v, lens, cap, seg_dtype=torch.bfloat16):
    """Caches by the policy for each sequence length, decode, oracle; returns worst error."""
    B, H, HQ = len(lens), w.n_kv_heads, w.n_q_heads
    rk, rv = cal_k[0].record_bytes, cal_v[0].record_bytes
    pk, pv = device_params(cal_k), device_params(cal_v)
    kc, vc = record_cache(H, cap, rk, batch=B), tile_cache(H, cap, rv, batch=B)
    ka, va = alpha_cache(H, cap, batch=B), alpha_cache(H, cap, batch=B)
    seg_k = torch.zeros((B, H, SEG_CAP, 128), dtype=seg_dtype, device="cuda")
    seg_v = torch.zeros_like(seg_k)
    n_comp, n_seg, parts = [], [], []
    for b, n in enumerate(lens):
        comp, seg = ora.segment_split(n)
        c, g = P.aatc_segment_counts(n)
        assert (c, g) == (comp.size, seg.size)
        xk = np.stack([w.cache(b, h, "k", n=n) for h in range(H)], axis=1)   # [n, H, 128]
        xv = np.stack([w.cache(b, h, "v", n=n) for h in range(H)], axis=1)
        if comp.size:
            tk = stored_to_torch(xk[comp]).cuda()
            tv = stored_to_torch(xv[comp]).cuda()
            P.aatc_encode(pk, H, tk, comp.size, H * 128, P.LAYOUT_RECORDS, kc[b], ka[b], cap, 0)
            P.aatc_encode(pv, H, tv, comp.size, H * 128, P.LAYOUT_TILES, vc[b], va[b], cap, 0)
        if seg.size:
            seg_k[b, :, :seg.size] = stored_to_torch(xk[seg]).cuda().transpose(0, 1).to(seg_dtype)
            seg_v[b, :, :seg.size] = stored_to_torch(xv[seg]).cuda().transpose(0, 1).to(seg_dtype)
        n_comp.append(comp.size)
        n_seg.append(seg.size)
        parts.append((comp, seg, xk, xv))
    q = stored_to_torch(np.stack([w.queries(b) for b in range(B)])).cuda()
    lt = torch.tensor(n_comp, dtype=torch.int32, device="cuda")
    st = torch.tensor(n_seg, dtype=torch.int32, device="cuda")
    out = torch.full((B, HQ, 128), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.zeros(P.aatc_decode_workspace_bytes(B, HQ, H, cap), dtype=torch.uint8, device="cuda")
    P.aatc_decode_attention_segmented(pk, pv, B, HQ, H, q, kc, ka, vc, va, lt, cap, rk, rv,
                                      1 / np.sqrt(128), seg_k, seg_v, st, SEG_CAP, out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    worst = 0.0
    for b, (comp, seg, xk, xv) in enumerate(parts):
        enc_k = [ora.encode(w.as_f32(xk[comp, h]), cal_k[h]) for h in range(H)]
        enc_v = [ora.encode(w.as_f32(xv[comp, h]), cal_v[h]) for h in range(H)]
        sk = [torch.from_numpy(w.as_f32(xk[seg, h])).to(seg_dtype).float().numpy() for h in range(H)]
        sv = [torch.from_numpy(w.as_f32(xv[seg, h])).to(seg_dtype).float().numpy() for h in range(H)]
        ref = ora.attention_with_segment(w.as_f32(w.queries(b)), cal_k, cal_v,
                                         [e[0] for e in enc_k], [e[1] for e in enc_k],
                                         [e[0] for e in enc_v], [e[1] for e in enc_v],
                                         comp.size, sk, sv)
        for j in range(HQ):
            err = rel_l2(got[b, j], ref[j])
            worst = max(worst, err)
            assert err <= 2e-3, (lens[b], j, err)
    return worst


@pytest.mark.parametrize("cfg", [2, 3])
def test_segmented_decode_around_flushes(cfg):
    """Lengths on both sides of the flushes (131 | 132, 147 | 148), only the sink, one
    token, and a long sequence; bf16 and fp32 segments."""
    lens = [1, 4, 5, 131, 132, 147, 148, 1000]
    w = workload(cfg, n_tokens=1000, batch=len(lens))
    H = w.n_kv_heads
    cal_k = [ora.calibrate(w.calib(h, "k"), 2.75) for h in range(H)]
    cal_v = [ora.calibrate(w.calib(h, "v"), 2.75) for h in range(H)]
    for dt in (torch.bfloat16, torch.float32):
        worst = _run(w, cal_k, cal_v, lens, 1024, dt)
        _log(f"[segment] cfg {cfg} {dt}: worst query head rel_l2 {worst:.2e}")


def test_segmented_decode_step_by_step_across_flushes():
    """Appending token by token with the policy (the flush encodes the window's oldest 16
    tokens at the end of the compressed cache): caches and outputs match the oracle at
    every step from 128 to 166 tokens."""
    w = workload(2, n_tokens=166, batch=1)
    H, HQ, cap = w.n_kv_heads, w.n_q_heads, 256
    cal_k = [ora.calibrate(w.calib(h, "k"), 2.75) for h in range(H)]
    cal_v = [ora.calibrate(w.calib(h, "v"), 2.75) for h in range(H)]
    rk, rv = cal_k[0].record_bytes, cal_v[0].record_bytes
    pk, pv = device_params(cal_k), device_params(cal_v)
    kc, vc = record_cache(H, cap, rk, batch=1), tile_cache(H, cap, rv, batch=1)
    ka, va = alpha_cache(H, cap, batch=1), alpha_cache(H, cap, batch=1)
    xk = np.stack([w.cache(0, h, "k") for h in range(H)], axis=1)
    xv = np.stack([w.cache(0, h, "v") for h in range(H)], axis=1)
    tk, tv = stored_to_torch(xk).cuda(), stored_to_torch(xv).cuda()
    q = stored_to_torch(np.stack([w.queries(0)])).cuda()
    ws = torch.zeros(P.aatc_decode_workspace_bytes(1, HQ, H, cap), dtype=torch.uint8, device="cuda")
    out = torch.zeros((1, HQ, 128), dtype=torch.float32, device="cuda")
    n_comp = 0
    for n in range(128, 167):
        comp, seg = ora.segment_split(n)
        if comp.size > n_comp:                           # the flush: 16 tokens at once
            k0 = comp[n_comp]
            P.aatc_encode(pk, H, tk[k0:], comp.size - n_comp, H * 128, P.LAYOUT_RECORDS,
                          kc[0], ka[0], cap, n_comp)
            P.aatc_encode(pv, H, tv[k0:], comp.size - n_comp, H * 128, P.LAYOUT_TILES,
                          vc[0], va[0], cap, n_comp)
            n_comp = comp.size
        seg_k = tk[seg].transpose(0, 1).contiguous()[None]
        seg_v = tv[seg].transpose(0, 1).contiguous()[None]
        lt = torch.tensor([n_comp], dtype=torch.int32, device="cuda")
        st = torch.tensor([seg.size], dtype=torch.int32, device="cuda")
        P.aatc_decode_attention_segmented(pk, pv, 1, HQ, H, q, kc, ka, vc, va, lt, cap, rk, rv,
                                          1 / np.sqrt(128), seg_k, seg_v, st, seg.size, out, ws)
        torch.cuda.synchronize()
        enc_k = [ora.encode(w.as_f32(xk[comp, h]), cal_k[h]) for h in range(H)]
        enc_v = [ora.encode(w.as_f32(xv[comp, h]), cal_v[h]) for h in range(H)]
        for h in range(H):
            np.testing.assert_array_equal(kc[0, h, :n_comp].cpu().numpy(), enc_k[h][0])
            np.testing.assert_array_equal(
                ora.tiles_to_records(vc[0, h].cpu().numpy(), rv)[:n_comp], enc_v[h][0])
        ref = ora.attention_with_segment(w.as_f32(w.queries(0)), cal_k, cal_v,
                                         [e[0] for e in enc_k], [e[1] for e in enc_k],
                                         [e[0] for e in enc_v], [e[1] for e in enc_v], n_comp,
                                         [w.as_f32(xk[seg, h]) for h in range(H)],
                                         [w.as_f32(xv[seg, h]) for h in range(H)])
        got = out.cpu().numpy()[0]
        for j in range(HQ):
            assert rel_l2(got[j], ref[j]) <= 2e-3, (n, j)
    _log(f"[segment] steps 128..166 ok, {n_comp} tokens compressed at the end")
