"""Distortion theory of the paper, for Monte-Carlo and deterministic pins.

TEST INFRASTRUCTURE ONLY.  Implements, in fp64:

* the softmax response along the ray theta -> softmax(s + theta * alpha) and its first
  three derivatives (Remark "Softmax derivatives along the ray", eq. g3-ray);
* the second-order expansion of the attention-weight perturbation
  delta_a = delta_a1 + delta_a2 + r (eq. softmax-2nd) with the exact remainder r;
* the output error split o - o^ = -(E_K + E_V + E_x) (App. A, Step 1);
* the leading distortion terms D_K and D_V of Theorem 1 (eq.
  distortion-decomposition), and the factorized form of D_K (eq.
  factorized-distortion).
"""
from __future__ import annotations

import numpy as np


def softmax(s: np.ndarray) -> np.ndarray:
    s = np.asarray(s, dtype=np.float64)
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def ray_derivatives(s: np.ndarray, alpha: np.ndarray, theta: float):
    """g_i(theta) = softmax(s + theta alpha)_i and g', g'', g''' (eq. g3-ray).

    With weights a~(theta), mean abar = sum a~ alpha, central moments m2, m3:
      g'   = a~_i (alpha_i - abar)
      g''  = a~_i ((alpha_i - abar)^2 - m2)
      g''' = a~_i ((alpha_i - abar)^3 - 3 (alpha_i - abar) m2 - m3)
    """
    at = softmax(np.asarray(s) + theta * np.asarray(alpha))
    abar = np.sum(at * alpha)
    dev = alpha - abar
    m2 = np.sum(at * dev ** 2)
    m3 = np.sum(at * dev ** 3)
    return at, at * dev, at * (dev ** 2 - m2), at * (dev ** 3 - 3.0 * dev * m2 - m3)


def delta_a_expansion(s: np.ndarray, alpha: np.ndarray):
    """Exact delta_a = softmax(s + alpha) - softmax(s) and its split (eq. softmax-2nd).

    delta_a1 = a_i (alpha_i - abar); delta_a2 = 1/2 a_i ((alpha_i - abar)^2 -
    sum_l a_l (alpha_l - abar)^2); r = delta_a - delta_a1 - delta_a2.
    """
    a = softmax(s)
    da = softmax(np.asarray(s) + np.asarray(alpha)) - a
    abar = np.sum(a * alpha)
    dev = alpha - abar
    da1 = a * dev
    da2 = 0.5 * a * (dev ** 2 - np.sum(a * dev ** 2))
    return da, da1, da2, da - da1 - da2


def output_error_terms(a, da, v, dv, w_o):
    """E_K = sum_i da_i v_i W_O, E_V = sum_i a_i dv_i W_O, E_x = sum_i da_i dv_i W_O."""
    e_k = (da @ v) @ w_o
    e_v = (a @ dv) @ w_o
    e_x = (da @ dv) @ w_o
    return e_k, e_v, e_x


def leading_distortion(q, k, v, w_o, var_dk, var_dv, scale: float = 1.0):
    """(D_K, D_V) of Theorem 1 for per-element error variances var_dk, var_dv [T, d].

    D_K = sum_{i,c} a_i^2 ||v_i W_O - o||^2 q_c^2 E[dk_ic^2] with q already including
    the logit scale; D_V = sum_{i,c} a_i^2 E[dv_ic^2] ||W_O,c||^2.
    """
    qs = np.asarray(q, dtype=np.float64) * scale
    a = softmax(k @ qs)
    o = (a @ v) @ w_o
    u = v @ w_o - o[None, :]
    d_k = np.sum((a ** 2) * np.sum(u ** 2, axis=1) * (var_dk @ (qs ** 2)))
    d_v = np.sum((a ** 2)[:, None] * var_dv * np.sum(w_o ** 2, axis=1)[None, :])
    return float(d_k), float(d_v)


def factorized_key_distortion(q, k, v, w_o, var_dk_channel, scale: float = 1.0):
    """D_K = (sum_i a_i^2 ||u_i||^2) (sum_c q_c^2 E[dk_c^2]) (eq. factorized-distortion),
    valid when the key error variance depends on the channel only."""
    qs = np.asarray(q, dtype=np.float64) * scale
    a = softmax(k @ qs)
    o = (a @ v) @ w_o
    u = v @ w_o - o[None, :]
    return float(np.sum(a ** 2 * np.sum(u ** 2, axis=1)) * np.sum(qs ** 2 * var_dk_channel))


def monte_carlo_distortion(q, k, v, w_o, half_k, half_v, n_draws, rng, scale=1.0,
                           chunk=20000):
    """Empirical E||o - o^||^2 under i.i.d. uniform errors on [-half, half].

    The errors satisfy Assumptions 1-2 (zero-mean, independent, symmetric, bounded).
    Returns a dict with the mean distortion, its standard error, the mean of the
    cross term E_K . E_V (and its standard error) and the largest ratio
    max_i |r_i| / A0^3 and sum_i |r_i| / A0^3 seen (Lemma 1), where A0 bounds |alpha_l|
    on that draw.
    """
    q = np.asarray(q, dtype=np.float64)
    qs = q * scale
    t, d = k.shape
    a = softmax(k @ qs)
    o = (a @ v) @ w_o
    tot = tot2 = cross = cross2 = 0.0
    worst_max = worst_sum = 0.0
    done = 0
    while done < n_draws:
        m = min(chunk, n_draws - done)
        dk = rng.uniform(-half_k, half_k, size=(m, t, d))
        dv = rng.uniform(-half_v, half_v, size=(m, t, d))
        alpha = dk @ qs                                    # [m, t] logit perturbations
        s = k @ qs
        ah = softmax(s[None, :] + alpha)
        oh = np.einsum("mt,mtd->md", ah, v[None] + dv) @ w_o
        err = np.sum((o[None, :] - oh) ** 2, axis=1)
        tot += err.sum()
        tot2 += (err ** 2).sum()
        da = ah - a[None, :]
        e_k = (da @ v) @ w_o
        e_v = np.einsum("t,mtd->md", a, dv) @ w_o
        c = np.sum(e_k * e_v, axis=1)
        cross += c.sum()
        cross2 += (c ** 2).sum()
        # Lemma 1 on every draw, with A0 = max_l |alpha_l| (the proof only uses that).
        a0 = np.max(np.abs(alpha), axis=1)
        abar = alpha @ a
        dev = alpha - abar[:, None]
        da1 = a[None, :] * dev
        da2 = 0.5 * a[None, :] * (dev ** 2 - (dev ** 2) @ a[:, None])
        r = da - da1 - da2
        ok = a0 > 0
        if np.any(ok):
            worst_max = max(worst_max, float(np.max(np.max(np.abs(r[ok]), axis=1) / a0[ok] ** 3)))
            worst_sum = max(worst_sum, float(np.max(np.sum(np.abs(r[ok]), axis=1) / a0[ok] ** 3)))
        done += m
    mean = tot / n_draws
    se = np.sqrt(max(tot2 / n_draws - mean ** 2, 0.0) / n_draws)
    cm = cross / n_draws
    cse = np.sqrt(max(cross2 / n_draws - cm ** 2, 0.0) / n_draws)
    return dict(d_emp=mean, d_se=se, cross_kv=cm, cross_kv_se=cse,
                lemma_max_ratio=worst_max, lemma_sum_ratio=worst_sum)
