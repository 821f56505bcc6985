"""Seeded generators for the five KV workloads the path is measured on.

Every key/value vector of KV head ``h`` is drawn as ``x = D U diag(sqrt(lam)) z``:

* ``z ~ N(0, I_d)``;
* ``lam_i = i**-p`` for ``i = 1..d`` (``p`` differs between keys and values);
* ``U`` is a Haar-random orthogonal matrix seeded per head (QR of a Gaussian matrix with
  the signs of ``diag(R)`` folded into ``Q``);
* ``D`` multiplies a few seeded "outlier" coordinates of the keys by a gain.

Values are rounded to the workload's storage type: float32, or bfloat16 (fp64 -> fp32
round-to-nearest-even, then fp32 -> bf16 round-to-nearest-even).  bf16 data is carried
as ``uint16`` bit patterns.

Queries are ``query_gain`` times a fresh draw from the key generator of their KV head.
With gain 8 the logits ``q.k/sqrt(d)`` have a standard deviation of about 3: the
attention rows are peaked without being one-hot.

Random streams: ``numpy.random.default_rng([config_id, head, stream, index])``.
The streams are 0 = basis U, 1 = outlier coordinates, 2 = calibration keys,
3 = calibration values, 4 = cached keys, 5 = cached values, 6 = decode queries,
7 = calibration queries.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

# Stream identifiers (see module docstring).
S_BASIS, S_OUTLIER, S_CAL_K, S_CAL_V, S_CACHE_K, S_CACHE_V, S_QUERY, S_CAL_Q = range(8)

CONFIGS: Dict[int, dict] = {
    1: dict(name="single_head_512", batch=1, n_q_heads=1, n_kv_heads=1, d=128,
            n_tokens=512, dtype="f32", p_k=1.5, p_v=0.8, avg_bits=(2.75,),
            query_weighted_k=False),
    2: dict(name="llama31_8b_decode_b1_32k", batch=1, n_q_heads=32, n_kv_heads=8, d=128,
            n_tokens=32768, dtype="bf16", p_k=1.5, p_v=0.8, avg_bits=(2.75,),
            query_weighted_k=False),
    3: dict(name="qwen25_7b_decode_b8_16k", batch=8, n_q_heads=28, n_kv_heads=4, d=128,
            n_tokens=16384, dtype="bf16", p_k=2.0, p_v=0.8, avg_bits=(2.75,),
            query_weighted_k=False),
    4: dict(name="llama31_8b_prefill_64k", batch=1, n_q_heads=32, n_kv_heads=8, d=128,
            n_tokens=65536, dtype="bf16", p_k=1.5, p_v=0.8, avg_bits=(2.75, 4.0),
            query_weighted_k=False),
    5: dict(name="llama31_8b_decode_b4_128k", batch=4, n_q_heads=32, n_kv_heads=8, d=128,
            n_tokens=131072, dtype="bf16", p_k=1.5, p_v=0.8, avg_bits=(2.0,),
            query_weighted_k=True),
}
for _c in CONFIGS.values():
    _c.setdefault("n_outliers", 4)
    _c.setdefault("outlier_gain", 10.0)
    _c.setdefault("n_calib", 2048)
    _c.setdefault("b_max", 8)
    _c.setdefault("query_gain", 8.0)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even); return bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def haar_orthogonal(rng: np.random.Generator, d: int) -> np.ndarray:
    """Haar-distributed orthogonal d x d matrix (QR of a Gaussian, signs folded in)."""
    g = rng.standard_normal((d, d))
    q, r = np.linalg.qr(g)
    return q * np.sign(np.diag(r))[None, :]


def _spectrum(d: int, p: float) -> np.ndarray:
    return np.arange(1, d + 1, dtype=np.float64) ** (-p)


@dataclasses.dataclass
class HeadBasis:
    u: np.ndarray            # [d, d] orthogonal
    outliers: np.ndarray     # [n_outliers] coordinate indices (keys only)


@dataclasses.dataclass
class Workload:
    """One of the configurations, with its draws available per (head, sequence)."""

    config_id: int
    cfg: dict
    n_tokens: int            # cached tokens per sequence (may be reduced for tests)
    batch: int

    @property
    def d(self) -> int:
        return self.cfg["d"]

    @property
    def n_kv_heads(self) -> int:
        return self.cfg["n_kv_heads"]

    @property
    def n_q_heads(self) -> int:
        return self.cfg["n_q_heads"]

    @property
    def group(self) -> int:
        return self.cfg["n_q_heads"] // self.cfg["n_kv_heads"]

    @property
    def dtype(self) -> str:
        return self.cfg["dtype"]

    def _rng(self, head: int, stream: int, index: int = 0) -> np.random.Generator:
        return np.random.default_rng([self.config_id, head, stream, index])

    def basis(self, head: int) -> HeadBasis:
        u = haar_orthogonal(self._rng(head, S_BASIS), self.d)
        idx = self._rng(head, S_OUTLIER).choice(self.d, size=self.cfg["n_outliers"],
                                                replace=False)
        return HeadBasis(u=u, outliers=np.sort(idx))

    def _draw(self, rng: np.random.Generator, head: int, n: int, kind: str) -> np.ndarray:
        """fp64 draws [n, d] of keys ('k') or values ('v') for one head."""
        b = self.basis(head)
        p = self.cfg["p_k"] if kind == "k" else self.cfg["p_v"]
        lam = _spectrum(self.d, p)
        z = rng.standard_normal((n, self.d))
        x = (z * np.sqrt(lam)[None, :]) @ b.u.T
        if kind == "k":
            x[:, b.outliers] *= self.cfg["outlier_gain"]
        return x

    def _store(self, x: np.ndarray):
        """Round fp64 draws to the storage type: float32 array or bf16 bit array."""
        x32 = x.astype(np.float32)
        if self.dtype == "bf16":
            return f32_to_bf16_bits(x32)
        return x32

    def as_f32(self, stored: np.ndarray) -> np.ndarray:
        """Exact float32 view of stored values (bf16 bits are widened)."""
        if stored.dtype == np.uint16:
            return bf16_bits_to_f32(stored)
        return np.asarray(stored, dtype=np.float32)

    # -- calibration draws (one separate 2048-token draw per head and tensor) --
    def calib(self, head: int, kind: str) -> np.ndarray:
        stream = S_CAL_K if kind == "k" else S_CAL_V
        x = self._draw(self._rng(head, stream), head, self.cfg["n_calib"], kind)
        return self.as_f32(self._store(x))

    def calib_queries(self, head: int, n: Optional[int] = None) -> np.ndarray:
        """Calibration queries of the GQA group of ``head``: [group * n, d] float32."""
        n = self.cfg["n_calib"] if n is None else n
        x = self._draw(self._rng(head, S_CAL_Q), head, self.group * n, "k")
        return self.as_f32(self._store(self.cfg["query_gain"] * x))

    # -- cached tokens --
    def cache(self, seq: int, head: int, kind: str, n: Optional[int] = None,
              start: int = 0) -> np.ndarray:
        """Stored cache tokens [n, d] (float32 or bf16 bits) of one (sequence, head).

        Tokens are drawn in blocks of 4096 from per-block streams, so any token range
        can be produced without drawing the tokens before it.
        """
        n = self.n_tokens - start if n is None else n
        stream = S_CACHE_K if kind == "k" else S_CACHE_V
        out = []
        blk = 4096
        t = start
        while t < start + n:
            b0 = t // blk
            rng = self._rng(head, stream, seq * 1_000_003 + b0)
            x = self._draw(rng, head, blk, kind)
            lo = t - b0 * blk
            hi = min(blk, start + n - b0 * blk)
            out.append(self._store(x[lo:hi]))
            t = b0 * blk + hi
        return np.concatenate(out, axis=0) if out else self._store(np.zeros((0, self.d)))

    def queries(self, seq: int) -> np.ndarray:
        """Decode queries [n_q_heads, d] of one sequence (float32 or bf16 bits)."""
        rows = []
        for h in range(self.n_kv_heads):
            x = self._draw(self._rng(h, S_QUERY, seq), h, self.group, "k")
            rows.append(self.cfg["query_gain"] * x)
        return self._store(np.concatenate(rows, axis=0))


def workload(config_id: int, n_tokens: Optional[int] = None,
             batch: Optional[int] = None, **overrides) -> Workload:
    """Workload of a configuration, optionally with fewer cached tokens or sequences, or
    other fields of the configuration replaced (e.g. n_q_heads)."""
    cfg = dict(CONFIGS[config_id], **overrides)
    return Workload(config_id=config_id, cfg=cfg,
                    n_tokens=cfg["n_tokens"] if n_tokens is None else n_tokens,
                    batch=cfg["batch"] if batch is None else batch)


# ---------------------------------------------------------------------------------------
# Layer inputs and a projection, for the calibration form that starts from the layer's
# input activations X and its key or value projection W (K = X W).
# ---------------------------------------------------------------------------------------
S_LAYER_X, S_LAYER_W = 8, 9


def layer_inputs(seed: int, n: int, d_model: int, p: float = 1.0) -> np.ndarray:
    """[n, d_model] float32 calibration activations with a decaying spectrum: rows are
    U diag(sqrt(lam)) z with lam_i = i**-p and a Haar-random U."""
    u = haar_orthogonal(np.random.default_rng([seed, 0, S_LAYER_X, 0]), d_model)
    lam = np.arange(1, d_model + 1, dtype=np.float64) ** -p
    z = np.random.default_rng([seed, 0, S_LAYER_X, 1]).standard_normal((n, d_model))
    return ((z * np.sqrt(lam)[None, :]) @ u.T).astype(np.float32)


def projection(seed: int, d_model: int, d: int) -> np.ndarray:
    """[d_model, d] float32 projection with Gaussian entries of variance 1 / d_model."""
    g = np.random.default_rng([seed, 0, S_LAYER_W, 0]).standard_normal((d_model, d))
    return (g / np.sqrt(d_model)).astype(np.float32)
