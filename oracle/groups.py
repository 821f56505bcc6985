"""AATC head-group transforms -- TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's experiments compress several KV heads with one transform (Sec. 5.1, the
remark on head groups: the heads are merged into G groups, each with its own block B_i;
Sec. 5.2: the token scale is taken per head group; Sec. 6 setup: G = 2 groups for
Llama's 8 KV heads and G = 1 for Qwen's 4, so each group spans 512 key dimensions).

Reading used here and by the GPU path:
  * A group is ``gkv`` consecutive KV heads; group g holds KV heads g gkv .. g gkv + gkv - 1.
    Its token is the concatenation of those heads' vectors, d_g = 128 gkv elements, head
    kk of the group at elements [128 kk, 128 kk + 128).
  * Calibration, transform, allocation (B = round(avg_bits d_g) bits per token and
    group), scales, quantizer and record packing are those of ``oracle.aatc`` applied to
    the d_g-element vectors: one transform, one token scale alpha and one record per
    (token, group).
  * Key weights sum over every query head of the group (eq. waterfilling-keys with the
    GQA remark of App. B): a query of KV head k enters as the d_g vector that is zero
    outside block k % gkv.  Value weights take the rows of W_O that read the group.
  * Decode attention: query head j reads KV head k = j // (H_q / H_kv); its keys and
    values are block k % gkv of the reconstructed tokens of group k // gkv.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

from . import aatc

HEAD_DIM = 128


def group_tokens(x: np.ndarray, g: int, gkv: int) -> np.ndarray:
    """Tokens of group g: x [n, H_kv, 128] -> [n, 128 gkv] (KV heads g gkv .. concatenated)."""
    x = np.asarray(x)
    n, hkv, d = x.shape
    if d != HEAD_DIM or hkv % gkv or not 0 <= g < hkv // gkv:
        raise ValueError("bad group")
    return x[:, g * gkv:(g + 1) * gkv, :].reshape(n, gkv * d)


def embed_group_queries(q: np.ndarray, gkv: int) -> np.ndarray:
    """Calibration queries of one group for the key weights.

    q: [T, gkv, G_q, 128], the G_q query heads of each of the group's KV heads over T
    tokens.  Returns [T gkv G_q, 128 gkv]: each query placed in its KV head's block, zero
    elsewhere, stacked so that ``aatc.key_weights(p, ., gkv * G_q)`` averages over tokens
    and sums over the group's query heads."""
    q = np.asarray(q, dtype=np.float64)
    t, k, gq, d = q.shape
    if k != gkv or d != HEAD_DIM:
        raise ValueError("bad query shape")
    out = np.zeros((t, gkv, gq, gkv * d))
    for kk in range(gkv):
        out[:, kk, :, kk * d:(kk + 1) * d] = q[:, kk]
    return out.reshape(t * gkv * gq, gkv * d)


def calibrate_group(x_group: np.ndarray, avg_bits: float, b_max: int = 8,
                    percentile: float = 0.99, q_embedded: Optional[np.ndarray] = None,
                    n_q_heads: int = 1, w_o: Optional[np.ndarray] = None,
                    quantizer: str = "midtread") -> aatc.Calibration:
    """Alg. 1 (calibration) for one group and tensor: ``aatc.calibrate`` on the group's
    d_g-element tokens (x_group [n, d_g]); ``q_embedded`` from ``embed_group_queries``
    (with ``n_q_heads`` = the group's query heads) or ``w_o`` [d_g, d_out]."""
    return aatc.calibrate(x_group, avg_bits, b_max=b_max, percentile=percentile,
                          q_calib=q_embedded, group=n_q_heads, w_o=w_o, quantizer=quantizer)


def encode_group(x_group: np.ndarray, cal: aatc.Calibration):
    """Records [n, R], token scales alpha16 [n] (one per token and group) and codes of the
    group's tokens [n, d_g] (``aatc.encode`` on the concatenated vectors)."""
    return aatc.encode(np.asarray(x_group, dtype=np.float32), cal)


def group_attention(q32: np.ndarray, n_kv_heads: int, gkv: int,
                    cal_k: Sequence[aatc.Calibration], cal_v: Sequence[aatc.Calibration],
                    k_rec, k_alpha, v_rec, v_alpha, seq_len: int,
                    scale: Optional[float] = None) -> np.ndarray:
    """Exact attention of one sequence's query heads over its group-compressed cache.

    q32: [H_q, 128]; cal_k / cal_v: one Calibration per group; k_rec / v_rec: per group
    records [>= seq_len, R]; k_alpha / v_alpha: per group fp16 token scales.  Query head j
    reads KV head k = j // (H_q / H_kv), block k % gkv of group k // gkv.  Returns
    [H_q, 128] fp64."""
    q32 = np.asarray(q32)
    hq, d = q32.shape
    if d != HEAD_DIM or n_kv_heads % gkv or hq % n_kv_heads:
        raise ValueError("bad shapes")
    gq = hq // n_kv_heads
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    out = np.zeros((hq, d))
    for g in range(n_kv_heads // gkv):
        kg = aatc.decode_tokens(k_rec[g][:seq_len], k_alpha[g][:seq_len], cal_k[g])
        vg = aatc.decode_tokens(v_rec[g][:seq_len], v_alpha[g][:seq_len], cal_v[g])
        for kk in range(gkv):
            k = g * gkv + kk
            blk = slice(kk * d, (kk + 1) * d)
            out[k * gq:(k + 1) * gq] = aatc.softmax_attention(
                q32[k * gq:(k + 1) * gq], kg[:, blk], vg[:, blk], scale)
    return out
