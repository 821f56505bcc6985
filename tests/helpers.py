"""Shared test helpers: convert oracle calibrations to the C ABI struct and build
compressed caches through the HIP path."""
from __future__ import annotations

import numpy as np

from oracle import aatc as ora


def abi_calibration(cal: "ora.Calibration"):
    """ctypes aatc_calibration holding an oracle calibration (host memory)."""
    import paper_2608_14191_amd as P
    c = P.Calibration()
    c.d = cal.d
    c.budget_bits = cal.budget
    c.record_bytes = cal.record_bytes
    c.d_active = cal.d_active
    c.quantizer = P.QUANT_MIDRISE if cal.quantizer == "midrise" else P.QUANT_MIDTREAD
    np.ctypeslib.as_array(c.transform)[:] = cal.T32.reshape(-1)
    np.ctypeslib.as_array(c.bits)[:] = cal.bits
    np.ctypeslib.as_array(c.scale_f16)[:] = cal.s16.view(np.uint16)
    np.ctypeslib.as_array(c.perm)[:] = cal.perm
    np.ctypeslib.as_array(c.sigma2)[:] = cal.sigma2
    np.ctypeslib.as_array(c.weight)[:] = cal.weight
    np.ctypeslib.as_array(c.bits_eig)[:] = cal.bits_eig
    return c


def device_params(cals, device="cuda"):
    """Device parameter block (torch uint8) of per-head calibrations (oracle or ABI)."""
    import torch
    import paper_2608_14191_amd as P
    abi = [c if isinstance(c, P.Calibration) else abi_calibration(c) for c in cals]
    host = P.aatc_params_pack(abi)
    return torch.from_numpy(host).to(device)


def abi_group_calibration(cal: "ora.Calibration"):
    """ctypes aatc_group_calibration holding an oracle calibration of a head group."""
    import paper_2608_14191_amd as P
    d = cal.d
    c = P.GroupCalibration()
    c.d = d
    c.budget_bits = cal.budget
    c.record_bytes = cal.record_bytes
    c.d_active = cal.d_active
    c.quantizer = P.QUANT_MIDRISE if cal.quantizer == "midrise" else P.QUANT_MIDTREAD
    np.ctypeslib.as_array(c.transform)[:d * d] = cal.T32.reshape(-1)
    np.ctypeslib.as_array(c.bits)[:d] = cal.bits
    np.ctypeslib.as_array(c.scale_f16)[:d] = cal.s16.view(np.uint16)
    np.ctypeslib.as_array(c.perm)[:d] = cal.perm
    np.ctypeslib.as_array(c.sigma2)[:d] = cal.sigma2
    np.ctypeslib.as_array(c.weight)[:d] = cal.weight
    np.ctypeslib.as_array(c.bits_eig)[:d] = cal.bits_eig
    return c


def group_device_params(cals, device="cuda"):
    """Device parameter block (torch uint8) of per-group calibrations (oracle or ABI)."""
    import torch
    import paper_2608_14191_amd as P
    abi = [c if isinstance(c, P.GroupCalibration) else abi_group_calibration(c) for c in cals]
    host = P.aatc_group_params_pack(abi)
    return torch.from_numpy(host).to(device)


def stored_to_torch(arr):
    """float32 array or bf16 bit array -> torch tensor of the same values (CPU)."""
    import torch
    if arr.dtype == np.uint16:
        return torch.from_numpy(arr.view(np.int16).copy()).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32))


def record_cache(n_heads, cap, rbytes, batch=None, device="cuda"):
    import torch
    shape = (n_heads, cap, rbytes) if batch is None else (batch, n_heads, cap, rbytes)
    return torch.zeros(shape, dtype=torch.uint8, device=device)


def tile_cache(n_heads, cap, rbytes, batch=None, device="cuda"):
    import torch
    nt = cap // 64
    shape = (n_heads, nt, 64 * rbytes) if batch is None else (batch, n_heads, nt, 64 * rbytes)
    return torch.zeros(shape, dtype=torch.uint8, device=device)


def alpha_cache(n_heads, cap, batch=None, device="cuda"):
    import torch
    shape = (n_heads, cap) if batch is None else (batch, n_heads, cap)
    return torch.zeros(shape, dtype=torch.int16, device=device)


def oracle_tiles(rec: np.ndarray, cap: int) -> np.ndarray:
    """Oracle records [n, R] of one head -> tile bytes [cap/64, 64R] (zero beyond n)."""
    full = np.zeros((cap, rec.shape[1]), dtype=np.uint8)
    full[:rec.shape[0]] = rec
    return ora.records_to_tiles(full)


def rel_l2(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))
