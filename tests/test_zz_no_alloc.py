"""aatc_append_decode_attention_noalloc (the library's static workspace) against
aatc_append_decode_attention (a caller workspace): two calls in a row, the second smaller,
give bit-identical outputs and caches."""
import numpy as np
import pytest
import torch

import paper_2608_14191_amd as P
from kvsynth import workload
from oracle import aatc as ora

from helpers import alpha_cache, device_params, record_cache, stored_to_torch, tile_cache

pytestmark = pytest.mark.gpu


def _step(w, cal_k, cal_v, pk, pv, lens, cap, noalloc):
    B, H, HQ = len(lens), w.n_kv_heads, w.n_q_heads
    rk, rv = cal_k[0].record_bytes, cal_v[0].record_bytes
    kc, vc = record_cache(H, cap, rk, batch=B), tile_cache(H, cap, rv, batch=B)
    ka, va = alpha_cache(H, cap, batch=B), alpha_cache(H, cap, batch=B)
    xk_new = torch.zeros((B, H, 128), dtype=torch.bfloat16, device="cuda")
    xv_new = torch.zeros_like(xk_new)
    for b, n in enumerate(lens):
        xk = stored_to_torch(np.stack([w.cache(b, h, "k", n=n) for h in range(H)], axis=1)).cuda()
        xv = stored_to_torch(np.stack([w.cache(b, h, "v", n=n) for h in range(H)], axis=1)).cuda()
        if n > 1:
            P.aatc_encode(pk, H, xk, n - 1, H * 128, P.LAYOUT_RECORDS, kc[b], ka[b], cap, 0)
            P.aatc_encode(pv, H, xv, n - 1, H * 128, P.LAYOUT_TILES, vc[b], va[b], cap, 0)
        xk_new[b], xv_new[b] = xk[n - 1], xv[n - 1]
    q = stored_to_torch(np.stack([w.queries(b) for b in range(B)])).cuda()
    lt = torch.tensor(lens, dtype=torch.int32, device="cuda")
    out = torch.full((B, HQ, 128), float("nan"), dtype=torch.float32, device="cuda")
    if noalloc:
        P.aatc_append_decode_attention_noalloc(pk, pv, B, HQ, H, q, xk_new, xv_new, kc, ka, vc,
                                               va, lt, cap, rk, rv, 1 / np.sqrt(128), out)
    else:
        ws = torch.zeros(P.aatc_decode_workspace_bytes(B, HQ, H, cap), dtype=torch.uint8,
                         device="cuda")
        P.aatc_append_decode_attention(pk, pv, B, HQ, H, q, xk_new, xv_new, kc, ka, vc, va, lt,
                                       cap, rk, rv, 1 / np.sqrt(128), out, ws)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in (out, kc, ka, vc, va)]


def test_noalloc_matches_workspace_entry_point_twice():
    w = workload(2, n_tokens=2100, batch=3)
    H = w.n_kv_heads
    cal_k = [ora.calibrate(w.calib(h, "k"), 2.75) for h in range(H)]
    cal_v = [ora.calibrate(w.calib(h, "v"), 2.75) for h in range(H)]
    pk, pv = device_params(cal_k), device_params(cal_v)
    for lens, cap in (([2100, 1025, 64], 2112), ([300], 320)):   # the second call smaller
        print(f"[noalloc] lens {lens} cap {cap}", flush=True)
        want = _step(w, cal_k, cal_v, pk, pv, lens, cap, noalloc=False)
        got = _step(w, cal_k, cal_v, pk, pv, lens, cap, noalloc=True)
        assert np.all(np.isfinite(got[0]))
        for a, b in zip(got, want):
            np.testing.assert_array_equal(a.view(np.uint8), b.view(np.uint8))
