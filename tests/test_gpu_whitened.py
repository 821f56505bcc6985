"""GPU end to end from the paper's form of the calibration (Sec. 5.1 Step 1): host
calibration from layer inputs X and projections W_K, W_V (aatc_calibrate_whitened), the
cache of K = X W_K and V = X W_V encoded and decoded on the GPU, against the oracle on the
same calibrations."""
import numpy as np
import pytest
import torch

import paper_2608_14191_amd as P
from kvsynth import f32_to_bf16_bits, bf16_bits_to_f32, layer_inputs, projection
from oracle import aatc as ora

from helpers import alpha_cache, device_params, oracle_tiles, record_cache, rel_l2, tile_cache

pytestmark = pytest.mark.gpu


def _oracle_cal(c):
    bits = c.bits_np
    return ora.Calibration(d=128, budget=c.budget_bits, record_bytes=c.record_bytes,
                           d_active=c.d_active, bits=bits, perm=np.arange(128),
                           T64=c.T.astype(np.float64), T32=c.T, s16=c.s16,
                           sigma2=np.ones(128), weight=np.ones(128), bits_eig=bits)


def test_whitened_calibration_end_to_end():
    H, G, dm, n, cap = 2, 4, 256, 700, 768
    x_cal = layer_inputs(21, 2048, dm)
    x_new = layer_inputs(22, n, dm)
    wk = [projection(100 + h, dm, 128) for h in range(H)]
    wv = [projection(200 + h, dm, 128) for h in range(H)]
    cal_k = [P.aatc_calibrate_whitened(x_cal, wk[h], 2.75) for h in range(H)]
    cal_v = [P.aatc_calibrate_whitened(x_cal, wv[h], 2.75) for h in range(H)]
    for h in range(H):                   # the oracle's literal whitened SVD allocates the same
        o = ora.calibrate_whitened(x_cal, wk[h], 2.75)
        np.testing.assert_array_equal(cal_k[h].bits_np, o.bits)
    # cache tokens in bf16, as a model would hand them over
    kb = [f32_to_bf16_bits((x_new.astype(np.float64) @ wk[h]).astype(np.float32)) for h in range(H)]
    vb = [f32_to_bf16_bits((x_new.astype(np.float64) @ wv[h]).astype(np.float32)) for h in range(H)]
    pk, pv = device_params(cal_k), device_params(cal_v)
    rk, rv = cal_k[0].record_bytes, cal_v[0].record_bytes
    assert all(c.record_bytes == rk for c in cal_k) and all(c.record_bytes == rv for c in cal_v)
    kc, vc = record_cache(H, cap, rk), tile_cache(H, cap, rv)
    ka, va = alpha_cache(H, cap), alpha_cache(H, cap)

    def tok(bits):
        return torch.from_numpy(np.stack(bits, axis=1).view(np.int16).copy()).view(torch.bfloat16).cuda()
    P.aatc_encode(pk, H, tok(kb), n, H * 128, P.LAYOUT_RECORDS, kc, ka, cap, 0)
    P.aatc_encode(pv, H, tok(vb), n, H * 128, P.LAYOUT_TILES, vc, va, cap, 0)
    rng = np.random.default_rng(4)
    qf = (rng.standard_normal((H * G, 128)) * 0.3).astype(np.float32)
    qb = f32_to_bf16_bits(qf)
    q = torch.from_numpy(qb.view(np.int16).copy()).view(torch.bfloat16).cuda()[None]
    lens = torch.tensor([n], dtype=torch.int32, device="cuda")
    out = torch.zeros((1, H * G, 128), dtype=torch.float32, device="cuda")
    ws = torch.zeros(P.aatc_decode_workspace_bytes(1, H * G, H, cap), dtype=torch.uint8, device="cuda")
    P.aatc_decode_attention(pk, pv, 1, H * G, H, q, kc, ka, vc, va, lens, cap, rk, rv,
                            128 ** -0.5, out, ws)
    torch.cuda.synchronize()
    ok_, ov_ = [_oracle_cal(c) for c in cal_k], [_oracle_cal(c) for c in cal_v]
    enc_k = [ora.encode(bf16_bits_to_f32(kb[h]), ok_[h]) for h in range(H)]
    enc_v = [ora.encode(bf16_bits_to_f32(vb[h]), ov_[h]) for h in range(H)]
    for h in range(H):
        np.testing.assert_array_equal(kc[h, :n].cpu().numpy(), enc_k[h][0])
        np.testing.assert_array_equal(ka[h, :n].cpu().numpy().view(np.uint16), enc_k[h][1].view(np.uint16))
        np.testing.assert_array_equal(vc[h].cpu().numpy(), oracle_tiles(enc_v[h][0], cap))
    ref = ora.decode_attention(bf16_bits_to_f32(qb), ok_, ov_, [e[0] for e in enc_k],
                               [e[1] for e in enc_k], [e[0] for e in enc_v],
                               [e[1] for e in enc_v], n)
    got = out[0].cpu().numpy()
    for j in range(H * G):
        assert rel_l2(got[j], ref[j]) <= 2e-3, j
