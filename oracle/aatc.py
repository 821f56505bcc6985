"""AATC oracle: calibration, encoding and exact decode attention (NumPy, fp64).

TEST INFRASTRUCTURE ONLY (see the package docstring).  Citations name the paper's
sections, equations, algorithms and tables ("KV Cache Compression Through the Lens of
Transform Coding").

What is computed, step by step
------------------------------
Calibration (Alg. 1, offline part; Sec. 5.1 and 5.2), per KV head and tensor (K or V):
  1. Sigma = X^T X / n, the uncentered empirical covariance of the calibration
     samples (Sec. 5.1).
  2. Its eigendecomposition, sorted by decreasing eigenvalue.  The PCA basis P is the
     decorrelating transform.  The Proposition of App. D shows it spans the same
     channels as the whitening-based SVD; the two differ only by a per-channel scale,
     which changes neither the codes nor the products w_c * sigma_c^2 used by the
     allocation.
  3. Attention-aware channel weights (eq. waterfilling-keys and its GQA remark in
     App. B for keys; the value weight of Sec. 5.2).  w = 1 when no queries / W_O are
     given ("AATC var-only", Sec. 6).
  4. Integer reverse water-filling: minimize sum_c W_c 2^(-2 b_c) with W_c =
     w_c sigma_c^2, subject to sum_c b_c = B and b_c in {0..b_max} (eq.
     waterfilling-keys; Alg. 1).
  5. Per-channel scale s_c = 99th percentile of |h_c| over the calibration tokens
     (Sec. 5.2, "The right scaling").
Encoding (Alg. 1, online part; Sec. 5.2), per token and head:
  6. h = T^T x (eq. transformed-cache): the exact product of the token with the stored
     transform, rounded once to fp32.
  7. alpha = max_c |h_c / s_c| over the stored channels; the signed uniform quantizer
     with step Delta_c = 2 alpha s_c / 2^b_c (Sec. 5.2), in one of two readings:
     "midtread", the printed qtz/dqtz pair (levels k Delta), or "midrise", the
     symmetric quantizer of Sec. 4's remark and App. B's noise model (levels
     (k + 1/2) Delta, error at most half a step over the whole range).
  8. Bit packing of the codes (layout defined below; the paper is silent on it).
Decode attention (Alg. 1, online part; Def. 1):
  9. Reconstruct K = H^ T^T and V = H^ T^T, then o = softmax(q K^T / sqrt(d)) V in fp64.

Readings where the paper is silent or ambiguous (each listed in the design doc)
----------------------------------------------------------------------------
* The integer allocation (the paper names an unspecified "dynamic program"): greedy
  marginal allocation, one bit at a time to argmax_c W_c 4^(-b_c) among channels
  below b_max, ties to the lowest eigen index.  This is exactly optimal for the
  separable convex problem and spends exactly B = round(avg_bits * d) bits.
* Var-only weights are w = 1 on the orthonormal PCA coefficients (W_c = eigenvalue),
  the reconstruction-error criterion the paper equates with per-layer KVTC.
* alpha is taken over the stored channels only (zero-bit channels are not cached).
* Stored transform: the fp64 eigenvectors rounded to multiples of 2^-22 (every entry
  is then exactly an fp32 number).  The transform of a token is the exact real product
  sum_j x_j T_jc of the token as given (bf16 or fp32 values) with that stored matrix,
  rounded once to fp32 (nearest, ties to even): a result with a plain definition that
  does not depend on any order of summation.  The quantizer is the fp32 sequence of
  ``quantize``.  alpha and s_c are stored as fp16.
* Storage order of channels: stable sort by bit width, widest first (eigen order
  breaks ties), so dropped channels form a suffix.
* Quantizer: the printed formula (midtread) puts a level at 0, lets the top cell absorb
  values up to a full step above the largest level, and at b = 1 has the levels
  {-alpha s, 0}.  That contradicts the passages that call the quantizer symmetric with
  errors of at most half a step (Sec. 4, the remark after Assumption 1; App. B, the
  noise model).  The midrise reading satisfies them: code = clamp(floor(h / Delta),
  -2^(b-1), 2^(b-1) - 1), h^ = (code + 1/2) Delta.  Both are offered; midtread is the
  default.  Widths go up to b_max = 16 (App. E allows 0 to 16 bits per channel).

Parity unpinned (spec choices with no value in the paper to check against): the
percentile interpolation (linear between order statistics), the storage order and
the packing layout.  The tests pin them to worked examples of this spec.
"""
from __future__ import annotations

import dataclasses
from fractions import Fraction
from typing import Optional

import numpy as np

# The stored transform's entries are multiples of 2^-T_FRAC_BITS (see module docstring).
T_FRAC_BITS = 22
TILE_TOKENS = 64     # tokens per tile of the value-cache layout
FP16_MAX = 65504.0
MAX_BITS = 16        # widest channel code (App. E: 0 to 16 bits per channel)
QUANTIZERS = ("midtread", "midrise")


# --------------------------------------------------------------------------------------
# Calibration
# --------------------------------------------------------------------------------------
def covariance(x: np.ndarray) -> np.ndarray:
    """Uncentered empirical covariance Sigma = X^T X / n (Sec. 5.1)."""
    x = np.asarray(x, dtype=np.float64)
    return x.T @ x / x.shape[0]


def pca_basis(sigma: np.ndarray):
    """Eigenvectors of Sigma by decreasing eigenvalue, sign-canonicalized.

    Returns (P, lam): columns of P are orthonormal eigenvectors; lam the eigenvalues
    (the channel variances sigma_c^2 of Sec. 5.1 / App. B).  The sign of each column
    makes its largest-magnitude entry positive (the lowest row index wins a tie).
    """
    lam, vec = np.linalg.eigh(sigma)
    order = np.argsort(-lam, kind="stable")
    lam = lam[order]
    vec = vec[:, order]
    for c in range(vec.shape[1]):
        col = vec[:, c]
        j = int(np.argmax(np.abs(col)))   # first index of the maximum magnitude
        if col[j] < 0:
            vec[:, c] = -col
    return vec, lam


def key_weights(p: np.ndarray, q_calib: np.ndarray, group: int) -> np.ndarray:
    """w_c = (1/T) sum over the group's query heads and tokens of (P_c^T q)^2.

    eq. waterfilling-keys, with the GQA remark of App. B (sum over the query heads
    that share this KV head).  ``q_calib`` stacks the group's calibration queries,
    [group * T, d].
    """
    proj = np.asarray(q_calib, dtype=np.float64) @ p
    t = q_calib.shape[0] // group
    return (proj ** 2).sum(axis=0) / t


def value_weights(p: np.ndarray, w_o: np.ndarray) -> np.ndarray:
    """w_c = || (P^T W_O)_c ||^2, the value weight of Sec. 5.2 (W_O rows of this head)."""
    m = p.T @ np.asarray(w_o, dtype=np.float64)
    return (m ** 2).sum(axis=1)


def rwf_continuous(var: np.ndarray, avg_bits: float):
    """Classical reverse water-filling, closed form (Sec. 3.1, eq. bit-allocation).

    b_i = max(0, 1/2 log2(var_i / lam)) with the water level lam set so that the mean
    of b equals avg_bits.  Returns (lam, b).  The active set is found by trying the k
    largest variances, k = d .. 1.
    """
    var = np.asarray(var, dtype=np.float64)
    d = var.size
    order = np.argsort(-var, kind="stable")
    v = var[order]
    for k in range(d, 0, -1):
        # sum_{i<k} 1/2 log2(v_i / lam) = d * avg_bits
        log2_lam = (np.sum(np.log2(v[:k])) - 2.0 * d * avg_bits) / k
        lam = 2.0 ** log2_lam
        if v[k - 1] > lam and (k == d or v[k] <= lam):
            b = np.zeros(d)
            b[order[:k]] = 0.5 * np.log2(v[:k] / lam)
            return lam, b
    raise ValueError("no water level found")


def allocate_bits(w_var: np.ndarray, budget: int, b_max: int) -> np.ndarray:
    """Integer reverse water-filling by greedy marginal allocation (reading of Sec. 5.2).

    Each of the ``budget`` bits goes to argmax_c W_c 4^(-b_c) over channels with
    b_c < b_max (first index on ties).  Adding a bit to channel c lowers the objective
    sum_c W_c 2^(-2 b_c) by 3/4 W_c 4^(-b_c); those gains shrink geometrically per
    channel, so the greedy result is a global optimum of the separable problem.
    """
    w_var = np.asarray(w_var, dtype=np.float64)
    d = w_var.size
    if budget > d * b_max or budget < 0:
        raise ValueError("budget outside [0, d * b_max]")
    b = np.zeros(d, dtype=np.int64)
    for _ in range(budget):
        gain = np.where(b < b_max, np.ldexp(w_var, -2 * b), -np.inf)
        c = int(np.argmax(gain))
        b[c] += 1
    return b


def allocate_global(sigma2, weight, avg_bits: float, b_max: int, n_protect: int = 3,
                    protect_extra: int = 0, normalize_weight: bool = False,
                    pct: float = 95.0) -> np.ndarray:
    """One tensor's (keys' or values') widths over all layers at once.

    The water-filling problem of Sec. 5.2 sums the distortion over layers under a single
    budget; App. E adds two rules for it: each layer's variances (and, for the keys, its
    weights) are divided by that layer's own 95th percentile, which removes the activation
    scale that differs between layers, and the first three layers are protected with a
    fixed budget of the average width (values) or the average plus one bit (keys).
    Readings (the paper gives no formula):
      - the total budget is round(avg_bits m L) bits for L layers of m channels; the
        protected layers take round((avg_bits + protect_extra) m) each and the other
        layers share what is left, by the greedy of ``allocate_bits`` over all their
        channels (first (layer, channel) on ties);
      - inside a protected layer the same greedy runs on its own channels;
      - the percentile interpolates linearly; a layer whose percentile is 0 is not scaled.
    ``sigma2`` and ``weight`` are [L][m] (``weight`` None means 1).  Returns bits [L][m].
    """
    s2 = np.asarray(sigma2, dtype=np.float64)
    if s2.ndim != 2:
        raise ValueError("sigma2 must be [layers][channels]")
    n_layers, m = s2.shape
    w = np.ones_like(s2) if weight is None else np.asarray(weight, dtype=np.float64)
    if w.shape != s2.shape or not (np.all(s2 >= 0) and np.all(w >= 0)):
        raise ValueError("weights and variances must be non-negative and of one shape")

    def per_layer_scaled(a):
        p = np.percentile(a, pct, axis=1, keepdims=True)
        return a / np.where(p > 0, p, 1.0)

    w_var = (per_layer_scaled(w) if normalize_weight else w) * per_layer_scaled(s2)
    n_prot = min(n_protect, n_layers)
    total = int(np.floor(avg_bits * m * n_layers + 0.5))
    prot = int(np.floor((avg_bits + protect_extra) * m + 0.5))
    bits = np.zeros((n_layers, m), dtype=np.int64)
    for layer in range(n_prot):
        bits[layer] = allocate_bits(w_var[layer], prot, b_max)
    if n_layers > n_prot:
        rest = total - n_prot * prot
        bits[n_prot:] = allocate_bits(w_var[n_prot:].ravel(), rest, b_max).reshape(-1, m)
    return bits


def allocation_objective(w_var: np.ndarray, bits: np.ndarray) -> float:
    """sum_c W_c 2^(-2 b_c) (eq. waterfilling-keys)."""
    return float(np.sum(np.ldexp(np.asarray(w_var, dtype=np.float64), -2 * np.asarray(bits))))


def stored_transform(t64: np.ndarray) -> np.ndarray:
    """The transform as stored: each entry rounded to the nearest multiple of 2^-22 (ties
    to even).  For |t| <= 1 that is at most 23 significant bits, so the result is exact
    in fp32; it is returned as float32."""
    t = np.asarray(t64, dtype=np.float64)
    return np.ldexp(np.rint(np.ldexp(t, T_FRAC_BITS)), -T_FRAC_BITS).astype(np.float32)


def to_f16(x) -> np.ndarray:
    """Round to fp16 (nearest, ties to even), saturating at the largest finite value."""
    x = np.asarray(x, dtype=np.float64)
    return np.clip(x, -FP16_MAX, FP16_MAX).astype(np.float16)


@dataclasses.dataclass
class Calibration:
    """Calibration artifact of one (KV head, K or V); channels in storage order."""

    d: int
    budget: int               # B = sum of bits
    record_bytes: int         # R = 4 * ceil(B / 32)
    d_active: int             # channels with at least one bit
    bits: np.ndarray          # [d] int64, storage order, non-increasing
    perm: np.ndarray          # [d] eigen index of each storage channel
    T64: np.ndarray           # [d, d] fp64, column c = eigenvector of storage channel c
    T32: np.ndarray           # [d, d] the stored transform: T64 on the 2^-22 grid (fp32)
    s16: np.ndarray           # [d] fp16 per-channel scales (0 for dropped channels)
    sigma2: np.ndarray        # [d] eigenvalues, eigen order
    weight: np.ndarray        # [d] channel weights, eigen order
    bits_eig: np.ndarray      # [d] bits, eigen order
    quantizer: str = "midtread"   # "midtread" (the printed formula) or "midrise"


def calibrate(x_calib: np.ndarray, avg_bits: float, b_max: int = 8,
              percentile: float = 0.99, q_calib: Optional[np.ndarray] = None,
              group: int = 1, w_o: Optional[np.ndarray] = None,
              bits_eig: Optional[np.ndarray] = None,
              record_bytes: Optional[int] = None,
              quantizer: str = "midtread") -> Calibration:
    """Alg. 1 (calibration) for one KV head and one tensor.

    ``q_calib`` (keys) or ``w_o`` (values) select the attention-aware weights; with
    neither, w = 1 (var-only).  The budget is B = round(avg_bits * d) bits per token.
    With ``bits_eig`` the widths (eigen order) are given instead of allocated, as when one
    budget is allocated over several heads and layers (``allocate_global``); then
    ``avg_bits`` is not used.  ``record_bytes`` pads the records to a larger size (the heads
    of one tensor share the record size of the widest).  ``quantizer`` names the reading of
    the quantizer that encode and decode use (it changes neither the widths nor the scales).
    """
    if quantizer not in QUANTIZERS:
        raise ValueError(f"quantizer must be one of {QUANTIZERS}")
    if not 1 <= b_max <= MAX_BITS:
        raise ValueError(f"b_max must be in 1..{MAX_BITS}")
    x = np.asarray(x_calib, dtype=np.float64)
    n, d = x.shape
    if n < 2:
        raise ValueError("need at least 2 calibration samples")
    budget = (int(np.sum(bits_eig)) if bits_eig is not None
              else int(np.floor(avg_bits * d + 0.5)))
    p, lam = pca_basis(covariance(x))
    if q_calib is not None:
        w = key_weights(p, q_calib, group)
    elif w_o is not None:
        w = value_weights(p, w_o)
    else:
        w = np.ones(d)
    w_var = w * lam
    if bits_eig is None:
        bits_eig = allocate_bits(w_var, budget, b_max)
    bits_eig = np.asarray(bits_eig, dtype=np.int64)
    perm = np.argsort(-bits_eig, kind="stable")
    bits = bits_eig[perm]
    t64 = p[:, perm]
    t32 = stored_transform(t64)
    # Per-channel scale: 99th percentile of |h_c| over the calibration tokens.
    h = x @ t64
    s = np.zeros(d)
    for c in range(d):
        if bits[c] > 0:
            s[c] = np.percentile(np.abs(h[:, c]), 100.0 * percentile)
    s16 = to_f16(s)
    s16[bits == 0] = 0
    min_rb = 4 * ((budget + 31) // 32)
    if record_bytes is not None and (record_bytes < min_rb or record_bytes % 4):
        raise ValueError("record_bytes below the budget or not whole dwords")
    return Calibration(d=d, budget=budget,
                       record_bytes=min_rb if record_bytes is None else int(record_bytes),
                       d_active=int(np.count_nonzero(bits)), bits=bits, perm=perm,
                       T64=t64, T32=t32, s16=s16, sigma2=lam, weight=w,
                       bits_eig=bits_eig, quantizer=quantizer)


def whitened_svd(x_in: np.ndarray, w_proj: np.ndarray):
    """Sec. 5.1, Step 1 (whitening-based decorrelation), literally:

    Sigma_X = X^T X / T; Sigma_X = L L^T (Cholesky); W~ = L^T W; W~ = U S P^T (reduced
    SVD); A = L^-T U sqrt(S), B = sqrt(S) P^T, so that W = A B (eq. AB-factorization) and
    the cache holds H = X A (eq. transformed-cache).  Singular values decreasing; each
    column of P signed so its largest-magnitude entry is positive (U and A follow).
    Returns (A [d_model, d], B [d, d], S [d], P [d, d])."""
    x = np.asarray(x_in, dtype=np.float64)
    w = np.asarray(w_proj, dtype=np.float64)
    sig_x = covariance(x)
    chol = np.linalg.cholesky(sig_x)
    u, s, pt = np.linalg.svd(chol.T @ w, full_matrices=False)
    p = pt.T
    for c in range(p.shape[1]):
        j = int(np.argmax(np.abs(p[:, c])))
        if p[j, c] < 0:
            p[:, c] = -p[:, c]
            u[:, c] = -u[:, c]
    a_mat = np.linalg.solve(chol.T, u) * np.sqrt(s)[None, :]
    b_mat = np.sqrt(s)[:, None] * p.T
    return a_mat, b_mat, s, p


def calibrate_whitened(x_in: np.ndarray, w_proj: np.ndarray, avg_bits: float,
                       b_max: int = 8, percentile: float = 0.99,
                       q_calib: Optional[np.ndarray] = None, group: int = 1,
                       w_o: Optional[np.ndarray] = None,
                       quantizer: str = "midtread") -> Calibration:
    """Alg. 1 (calibration) from the layer's input activations X [T, d_model] and its key
    or value projection W [d_model, d], in the paper's form (Sec. 5.1 Step 1, Sec. 5.2):

    1. the whitened SVD (``whitened_svd``): A, B, S, P;
    2. channel variances of H = X A: var(h_c) = S_c (A^T Sigma_X A = S);
    3. weights from B: keys w_c = (1/T) sum over the group's queries of (B_c q)^2
       (eq. waterfilling-keys), values w_c = ||(B W_O)_c||^2 (Sec. 5.2); without either,
       w_c = ||B_c||^2 = S_c (var-only as the reconstruction error of K or V, the reading
       the PCA form uses);
    4. the integer allocation of w_c S_c (as in ``allocate_bits``);
    5. the cache stores K = X W in the basis P: h_c = (K P)_c = sqrt(S_c) (X A)_c, which
       differs from H only by a per-channel scale that changes no code (App. B); so the
       stored transform is P in storage order and s_c the 99th percentile of |(K P)_c|.
    """
    x = np.asarray(x_in, dtype=np.float64)
    a_mat, b_mat, s, p = whitened_svd(x, w_proj)
    d = b_mat.shape[0]
    if q_calib is not None:
        t = q_calib.shape[0] // group
        w = ((np.asarray(q_calib, dtype=np.float64) @ b_mat.T) ** 2).sum(axis=0) / t
    elif w_o is not None:
        w = ((b_mat @ np.asarray(w_o, dtype=np.float64)) ** 2).sum(axis=1)
    else:
        # var-only (reading: the key/value reconstruction error, as for the PCA form):
        # an error in h_c reaches K through row c of B, ||B_c||^2 = S_c
        w = s.copy()
    budget = int(np.floor(avg_bits * d + 0.5))
    bits_eig = allocate_bits(w * s, budget, b_max)
    k = x @ np.asarray(w_proj, dtype=np.float64)
    return _storage_calibration(k, p, s * s, w * s / (s * s), bits_eig, budget, percentile,
                                None, quantizer)


def _storage_calibration(k, p, lam, weight, bits_eig, budget, percentile, record_bytes,
                         quantizer) -> Calibration:
    """Storage order, stored transform and scales of a calibration whose basis P (eigen
    order), channel variances lam and widths (eigen order) are known; k holds the
    calibration samples in the original coordinates."""
    d = p.shape[0]
    bits_eig = np.asarray(bits_eig, dtype=np.int64)
    perm = np.argsort(-bits_eig, kind="stable")
    bits = bits_eig[perm]
    t64 = p[:, perm]
    t32 = stored_transform(t64)
    h = np.asarray(k, dtype=np.float64) @ t64
    s = np.zeros(d)
    for c in range(d):
        if bits[c] > 0:
            s[c] = np.percentile(np.abs(h[:, c]), 100.0 * percentile)
    s16 = to_f16(s)
    s16[bits == 0] = 0
    min_rb = 4 * ((budget + 31) // 32)
    if record_bytes is not None and (record_bytes < min_rb or record_bytes % 4):
        raise ValueError("record_bytes below the budget or not whole dwords")
    return Calibration(d=d, budget=budget,
                       record_bytes=min_rb if record_bytes is None else int(record_bytes),
                       d_active=int(np.count_nonzero(bits)), bits=bits, perm=perm,
                       T64=t64, T32=t32, s16=s16, sigma2=lam, weight=weight,
                       bits_eig=bits_eig, quantizer=quantizer)


# --------------------------------------------------------------------------------------
# Encoding
# --------------------------------------------------------------------------------------
def round_to_f32(q: Fraction) -> np.float32:
    """The fp32 number nearest to the rational q (ties to even), with fp32 subnormals and
    overflow to infinity: the rounding IEEE 754 defines, written out on exact integers."""
    q = Fraction(q)
    if q == 0:
        return np.float32(0.0)
    neg = q < 0
    a = -q if neg else q
    e = a.numerator.bit_length() - a.denominator.bit_length()   # 2^(e-1) < a < 2^(e+1)
    if a < Fraction(2) ** e:
        e -= 1                                                  # now 2^e <= a < 2^(e+1)
    quantum = Fraction(2) ** (max(e, -126) - 23)                # 24 significant bits,
    m = round(a / quantum)                                      # fewer below 2^-126
    v = m * quantum
    if v >= Fraction(2) ** 128:
        return np.float32(-np.inf if neg else np.inf)
    return np.float32(-float(v) if neg else float(v))           # exact: v is an fp32 value


def exact_dot_f32(x, t) -> np.float32:
    """fl32(sum_j x_j t_j) with the sum taken in exact rational arithmetic."""
    acc = Fraction(0)
    for xj, tj in zip(np.asarray(x, dtype=np.float64), np.asarray(t, dtype=np.float64)):
        acc += Fraction(float(xj)) * Fraction(float(tj))
    return round_to_f32(acc)


def transform(x32: np.ndarray, t32: np.ndarray) -> np.ndarray:
    """h = T^T x per token (eq. transformed-cache; Alg. 1 "project"): h_c is the exact
    value of sum_j x_j T_jc rounded once to fp32 (nearest, ties to even).  An exact zero
    is +0.

    x: [n, d] fp32 values (bf16 tokens widened exactly); t: [d, m] the stored transform,
    multiples of 2^-22 with |t| <= 1.  The sum is formed exactly in integers: with
    Tq = t 2^22 and, per token, x_j = 2^-S (X_j + 2^-31 Y_j) with integers X_j, Y_j (S puts
    max |X| in [2^30, 2^31); |Y| <= 2^30), the sum is 2^-(S+22+31) (2^31 H + L) with
    H = X Tq and L = Y Tq exact in int64 (|X| <= 2^31 and |Tq| <= 2^22, so every product
    is at most 2^53 and a sum of d <= 512 of them stays below 2^62).
      - Where L = 0 (every element a multiple of 2^-S, as for bf16 tokens whose elements
        are all above 2^-23 of the largest) the result is the int64 H converted to fp32,
        which rounds once, to nearest with ties to even (pinned by the tests), times the
        power of two, exact for normal results.
      - Elsewhere the integer 2^31 H + L is rounded by ``round_to_f32``.
      - Tokens whose elements are not all multiples of 2^-(S+31), and results in the fp32
        subnormal range, are redone from the definition in exact rational arithmetic.
    """
    x = np.asarray(x32, dtype=np.float32)
    t = np.asarray(t32, dtype=np.float32)
    n, d = x.shape
    if d > 512:
        raise ValueError("at most 512 elements per token")
    tq_f = np.ldexp(t.astype(np.float64), T_FRAC_BITS)
    if not (np.all(tq_f == np.rint(tq_f)) and np.all(np.abs(tq_f) <= 2.0 ** T_FRAC_BITS)):
        raise ValueError("the transform must be on the 2^-22 grid with |t| <= 1")
    tq = tq_f.astype(np.int64)
    xd = x.astype(np.float64)
    m = np.max(np.abs(xd), axis=1) if d else np.zeros(n)
    e = np.frexp(m)[1] - 1                                   # 2^e <= m < 2^(e+1)
    S = np.where(m > 0, 30 - e, 0)
    v = np.ldexp(xd, S[:, None])                             # exact (power-of-two scale)
    X = np.rint(v)
    Yf = np.ldexp(v - X, 31)                                 # v - X is exact
    Y = np.rint(Yf)
    split_ok = np.all(Y == Yf, axis=1)
    H = X.astype(np.int64) @ tq
    h = np.ldexp(H.astype(np.float32), -(S + T_FRAC_BITS)[:, None])
    rows = np.flatnonzero(split_ok & np.any(Y != 0, axis=1))
    if rows.size:
        L = Y[rows].astype(np.int64) @ tq
        for r, i in enumerate(rows):
            for c in range(t.shape[1]):
                V = int(H[i, c]) * 2 ** 31 + int(L[r, c])
                h[i, c] = round_to_f32(Fraction(V, 2 ** int(S[i] + T_FRAC_BITS + 31))
                                       if S[i] + T_FRAC_BITS + 31 >= 0 else
                                       Fraction(V * 2 ** int(-(S[i] + T_FRAC_BITS + 31))))
    redo = ~split_ok[:, None] | ((np.abs(h) < np.float32(2.0 ** -126)) & (h != 0))
    for i, c in np.argwhere(redo):
        h[i, c] = exact_dot_f32(x[i], t[:, c])
    h[h == 0] = 0.0
    return h


def inverse_f32(v: np.ndarray) -> np.ndarray:
    """fp32 1/v rounded to nearest, and 0 where v == 0."""
    v = np.asarray(v, dtype=np.float32)
    safe = np.where(v != 0, v, np.float32(1))
    return np.where(v != 0, np.float32(1) / safe, np.float32(0)).astype(np.float32)


def quantize(h32: np.ndarray, bits: np.ndarray, s16: np.ndarray, kind: str = "midtread"):
    """Signed uniform quantizer with per-token scale alpha (Sec. 5.2).

    For each token: alpha = max_c |h_c / s_c| over channels with b_c >= 1; with
    Delta_c = 2 alpha s_c / 2^b_c the code is clamp(floor(h_c / Delta_c + 1/2),
    -2^(b-1), 2^(b-1) - 1) (midtread, the printed formula) or clamp(floor(h_c / Delta_c),
    -2^(b-1), 2^(b-1) - 1) (midrise, whose level is (code + 1/2) Delta_c).
    The canonical fp32 evaluation is r = h * (1/s), alpha16 = fp16(max |r|),
    y = r * (1/alpha16), x = y * 2^(b-1) (exact), code = floor(x + 1/2) taken exactly
    (midtread) or floor(x) (midrise).
    Returns (code [n, d] int64 with 0 for dropped channels, alpha16 [n] fp16).
    """
    h = np.asarray(h32, dtype=np.float32)
    bits = np.asarray(bits, dtype=np.int64)
    keep = bits > 0
    inv_s = inverse_f32(np.asarray(s16, dtype=np.float16).astype(np.float32))
    r = (h * inv_s[None, :]).astype(np.float32)
    if np.any(keep):
        alpha = np.max(np.abs(r[:, keep]), axis=1)
    else:
        alpha = np.zeros(h.shape[0], dtype=np.float32)
    alpha16 = to_f16(alpha)
    inv_a = inverse_f32(alpha16.astype(np.float32))
    y = (r * inv_a[:, None]).astype(np.float32)
    x = np.ldexp(y, np.maximum(bits - 1, 0)[None, :]).astype(np.float32)
    f = np.floor(x)
    if kind == "midrise":
        code = f
    elif kind == "midtread":
        code = f + ((x - f) >= np.float32(0.5))
    else:
        raise ValueError(f"unknown quantizer {kind!r}")
    half = np.left_shift(1, np.maximum(bits - 1, 0))
    lo = np.where(keep, -half, 0)
    hi = np.where(keep, half - 1, 0)
    code = np.clip(code.astype(np.int64), lo[None, :], hi[None, :])
    return code.astype(np.int64), alpha16


def dequantize(code: np.ndarray, alpha16: np.ndarray, bits: np.ndarray,
               s16: np.ndarray, kind: str = "midtread") -> np.ndarray:
    """h^_c = Delta_c * code_c = alpha s_c 2^(1-b_c) code_c (midtread) or
    Delta_c * (code_c + 1/2) (midrise); 0 for b_c = 0."""
    bits = np.asarray(bits, dtype=np.int64)
    keep = bits > 0
    s = np.asarray(s16, dtype=np.float16).astype(np.float64)
    a = np.asarray(alpha16, dtype=np.float16).astype(np.float64)
    step = np.where(keep, s * np.ldexp(1.0, 1 - bits), 0.0)
    level = np.asarray(code, dtype=np.float64)
    if kind == "midrise":
        level = level + 0.5
    elif kind != "midtread":
        raise ValueError(f"unknown quantizer {kind!r}")
    return a[:, None] * step[None, :] * level


# --------------------------------------------------------------------------------------
# Packing (the paper does not specify one; this is the layout the path defines)
# --------------------------------------------------------------------------------------
def pack_records(code: np.ndarray, bits: np.ndarray, rbytes: Optional[int] = None) -> np.ndarray:
    """Token-major records: the codes of one token as one LSB-first bit string.

    Channel c (storage order) occupies bits [o_c, o_c + b_c) with o_c = sum of the
    earlier widths and holds the b_c-bit two's complement pattern of its code, least
    significant bit first; bit i of the record is bit i % 8 of byte i // 8.  The record
    is zero-padded to R = 4 * ceil(B / 32) bytes, or to ``rbytes`` if given.
    """
    code = np.asarray(code, dtype=np.int64)
    bits = np.asarray(bits, dtype=np.int64)
    n = code.shape[0]
    budget = int(bits.sum())
    rbytes = 4 * ((budget + 31) // 32) if rbytes is None else int(rbytes)
    flat = np.zeros((n, 8 * rbytes), dtype=np.uint8)
    off = 0
    for c, b in enumerate(bits):
        pattern = np.mod(code[:, c], 1 << int(b))           # two's complement, b bits
        for k in range(int(b)):
            flat[:, off + k] = (pattern >> k) & 1
        off += int(b)
    return np.packbits(flat, axis=1, bitorder="little")


def unpack_records(rec: np.ndarray, bits: np.ndarray) -> np.ndarray:
    """Inverse of ``pack_records``: signed codes [n, d] (0 for dropped channels)."""
    bits = np.asarray(bits, dtype=np.int64)
    flat = np.unpackbits(np.asarray(rec, dtype=np.uint8), axis=1, bitorder="little")
    code = np.zeros((rec.shape[0], bits.size), dtype=np.int64)
    off = 0
    for c, b in enumerate(bits):
        b = int(b)
        if b == 0:
            continue
        u = np.zeros(rec.shape[0], dtype=np.int64)
        for k in range(b):
            u |= flat[:, off + k].astype(np.int64) << k
        code[:, c] = np.where(u >= (1 << (b - 1)), u - (1 << b), u)
        off += b
    return code


def _tile_token_of_bit() -> np.ndarray:
    """Token (0..63) of each (word W, bit p) position of a value tile: t = 16 d + 4 g + i
    is stored in word W = d // 2 at bit p = 8 i + 2 g + d % 2."""
    tok = np.zeros((2, 32), dtype=np.int64)
    for t in range(TILE_TOKENS):
        d, g, i = t // 16, (t // 4) % 4, t % 4
        tok[d // 2, 8 * i + 2 * g + d % 2] = t
    return tok


def records_to_tiles(rec: np.ndarray) -> np.ndarray:
    """Value-cache layout: tiles of 64 tokens, bit-transposed.

    Record bit v of the 64 tokens of tile j is stored in two little-endian 32-bit words
    (j, v, W), W = 0, 1.  Token t = 16 d + 4 g + i of the tile (d, g, i in 0..3) sits
    in word W = d // 2 at bit 8 i + 2 g + d % 2.  A tile is 8R words x 2 = 64 R bytes,
    the same bytes as its 64 records.  The token count must be a multiple of 64.
    Returns uint8 [n_tiles, 64 R].
    """
    rec = np.asarray(rec, dtype=np.uint8)
    n, rbytes = rec.shape
    if n % TILE_TOKENS:
        raise ValueError("token count must be a multiple of 64")
    flat = np.unpackbits(rec, axis=1, bitorder="little")              # [n, 8R]
    nt = n // TILE_TOKENS
    tok = _tile_token_of_bit()                                        # [2, 32]
    b = flat.reshape(nt, TILE_TOKENS, 8 * rbytes)[:, tok, :]          # [nt, 2, 32, 8R]
    b = b.transpose(0, 3, 1, 2)                                       # [nt, 8R, 2, 32]
    return np.packbits(b, axis=-1, bitorder="little").reshape(nt, 64 * rbytes)


def tiles_to_records(tiles: np.ndarray, rbytes: int) -> np.ndarray:
    """Inverse of ``records_to_tiles``: records [64 * n_tiles, R]."""
    tiles = np.asarray(tiles, dtype=np.uint8)
    nt = tiles.shape[0]
    b = np.unpackbits(tiles.reshape(nt, 8 * rbytes, 2, 4), axis=-1, bitorder="little")
    b = b.transpose(0, 2, 3, 1)                                       # [nt, 2, 32, 8R]
    flat = np.zeros((nt, TILE_TOKENS, 8 * rbytes), dtype=np.uint8)
    flat[:, _tile_token_of_bit(), :] = b
    return np.packbits(flat.reshape(nt * TILE_TOKENS, 8 * rbytes), axis=1, bitorder="little")


def encode(x32: np.ndarray, cal: Calibration):
    """Encode tokens [n, d] of one head: (records [n, R] uint8, alpha16 [n], codes [n, d])."""
    h = transform(x32, cal.T32)
    code, alpha16 = quantize(h, cal.bits, cal.s16, cal.quantizer)
    return pack_records(code, cal.bits, cal.record_bytes), alpha16, code


def decode_tokens(rec: np.ndarray, alpha16: np.ndarray, cal: Calibration) -> np.ndarray:
    """Reconstructed tokens [n, d] in the original coordinates: x^ = T h^ (fp64), with the
    stored transform that encoded them."""
    h = dequantize(unpack_records(rec, cal.bits), alpha16, cal.bits, cal.s16, cal.quantizer)
    return h @ np.asarray(cal.T32, dtype=np.float64).T


# --------------------------------------------------------------------------------------
# Decode attention
# --------------------------------------------------------------------------------------
def softmax_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float) -> np.ndarray:
    """One decode row per query: o = softmax(q k^T * scale) v, fp64 (Def. 1, no mask
    inside the cache: the decode row attends to every cached token)."""
    q = np.asarray(q, dtype=np.float64)
    s = (q @ np.asarray(k, dtype=np.float64).T) * scale
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p /= p.sum(axis=-1, keepdims=True)
    return p @ np.asarray(v, dtype=np.float64)


def decode_attention(q32: np.ndarray, cal_k, cal_v, k_rec, k_alpha, v_rec, v_alpha,
                     seq_len: int, scale: Optional[float] = None) -> np.ndarray:
    """Attention of one sequence's queries over its compressed cache (Alg. 1, online).

    q32: [H_q, d] fp32 queries; cal_k / cal_v: per-KV-head Calibration lists;
    k_rec / v_rec: per-head records [>= seq_len, R]; k_alpha / v_alpha: per-head fp16
    token scales.  Query head j reads KV head j // (H_q / H_kv).  Returns [H_q, d] fp64.
    """
    hq, d = q32.shape
    hkv = len(cal_k)
    g = hq // hkv
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    out = np.zeros((hq, d))
    for h in range(hkv):
        kh = decode_tokens(k_rec[h][:seq_len], k_alpha[h][:seq_len], cal_k[h])
        vh = decode_tokens(v_rec[h][:seq_len], v_alpha[h][:seq_len], cal_v[h])
        out[h * g:(h + 1) * g] = softmax_attention(q32[h * g:(h + 1) * g], kh, vh, scale)
    return out


# --------------------------------------------------------------------------------------
# Full-precision sink and recent window (Sec. 6 experimental setup; App. E, "AATC")
# --------------------------------------------------------------------------------------
def segment_split(n_tokens: int, sink: int = 4, window: int = 128, step: int = 16):
    """Which of a sequence's first ``n_tokens`` tokens are compressed and which stay at
    input precision, by playing the paper's policy token by token: the first ``sink``
    tokens are kept; later tokens enter the recent window, and whenever the window holds
    ``window`` tokens its oldest ``step`` are quantized (appended to the compressed cache).
    Returns (compressed token indices in cache order, segment token indices)."""
    kept = list(range(min(sink, n_tokens)))
    compressed, win = [], []
    for t in range(len(kept), n_tokens):
        win.append(t)
        if len(win) == window:
            compressed.extend(win[:step])
            win = win[step:]
    return np.array(compressed, dtype=np.int64), np.array(kept + win, dtype=np.int64)


def attention_with_segment(q32, cal_k, cal_v, k_rec, k_alpha, v_rec, v_alpha, n_comp: int,
                           seg_k, seg_v, scale: Optional[float] = None) -> np.ndarray:
    """Exact softmax attention of each query head over the union of its KV head's
    ``n_comp`` compressed tokens (decoded: records, fp16 scales, calibration) and its
    segment tokens kept at input precision (``seg_k[h]``, ``seg_v[h]``: [n, d] fp32 values).
    Query head j reads KV head j // (H_q / H_kv).  Returns [H_q, d] fp64."""
    hq, d = q32.shape
    hkv = len(cal_k)
    g = hq // hkv
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    out = np.zeros((hq, d))
    for h in range(hkv):
        kh = decode_tokens(k_rec[h][:n_comp], k_alpha[h][:n_comp], cal_k[h])
        vh = decode_tokens(v_rec[h][:n_comp], v_alpha[h][:n_comp], cal_v[h])
        kk = np.concatenate([kh, np.asarray(seg_k[h], dtype=np.float64)], axis=0)
        vv = np.concatenate([vh, np.asarray(seg_v[h], dtype=np.float64)], axis=0)
        if kk.shape[0] == 0:
            continue
        out[h * g:(h + 1) * g] = softmax_attention(q32[h * g:(h + 1) * g], kk, vv, scale)
    return out
