"""ctypes binding of libaatc.so: the C ABI of include/aatc.h, argument marshalling only.

Every function here has the name of the C entry point it calls.  Device buffers are
torch tensors on a HIP device; their pointers and the current HIP stream are handed to
the library, which does all the work.  If libaatc.so is missing, importing this module
raises ImportError: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np

from .build import LIB

HEAD_DIM = 128
MAX_BITS = 16
TILE_TOKENS = 64

OK, E_INVALID, E_UNSUPPORTED, E_NUMERIC, E_DEVICE, E_WORKSPACE = range(6)
QUANT_MIDTREAD, QUANT_MIDRISE = 0, 1
F32, BF16, F16 = 0, 1, 2
LAYOUT_RECORDS, LAYOUT_TILES = 0, 1


class AatcError(RuntimeError):
    def __init__(self, func: str, status: int):
        super().__init__(f"{func}: {_status_string(status)} (status {status})")
        self.status = status


class Calibration(ctypes.Structure):
    """Mirror of aatc_calibration (include/aatc.h)."""

    _fields_ = [
        ("d", ctypes.c_int32),
        ("budget_bits", ctypes.c_int32),
        ("record_bytes", ctypes.c_int32),
        ("d_active", ctypes.c_int32),
        ("quantizer", ctypes.c_int32),
        ("transform", ctypes.c_float * (HEAD_DIM * HEAD_DIM)),
        ("bits", ctypes.c_uint8 * HEAD_DIM),
        ("scale_f16", ctypes.c_uint16 * HEAD_DIM),
        ("perm", ctypes.c_int32 * HEAD_DIM),
        ("sigma2", ctypes.c_double * HEAD_DIM),
        ("weight", ctypes.c_double * HEAD_DIM),
        ("bits_eig", ctypes.c_uint8 * HEAD_DIM),
    ]

    # numpy views (copies) for convenience
    @property
    def T(self) -> np.ndarray:
        return np.ctypeslib.as_array(self.transform).reshape(HEAD_DIM, HEAD_DIM).copy()

    @property
    def bits_np(self) -> np.ndarray:
        return np.ctypeslib.as_array(self.bits).astype(np.int64)

    @property
    def s16(self) -> np.ndarray:
        return np.ctypeslib.as_array(self.scale_f16).copy().view(np.float16)


LIB_PATH = os.environ.get("AATC_LIBRARY", LIB)   # optional override of the built library
if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; call __graft_entry__.build() first")
_L = ctypes.CDLL(LIB_PATH)

_vp, _i32, _i64, _sz, _f32, _f64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                    ctypes.c_size_t, ctypes.c_float, ctypes.c_double)
_L.aatc_status_string.restype = ctypes.c_char_p
_L.aatc_status_string.argtypes = [ctypes.c_int]
_L.aatc_calibrate.restype = ctypes.c_int
_L.aatc_calibrate.argtypes = [_vp, _i64, _i32, _vp, _i64, _i32, _vp, _i32, _f64, _i32, _f64,
                              ctypes.POINTER(Calibration)]
_L.aatc_calibrate_whitened.restype = ctypes.c_int
_L.aatc_calibrate_whitened.argtypes = [_vp, _i64, _i32, _vp, _i32, _vp, _i64, _i32, _vp, _i32,
                                       _f64, _i32, _f64, ctypes.POINTER(Calibration)]
_L.aatc_calibrate_bits.restype = ctypes.c_int
_L.aatc_calibrate_bits.argtypes = [_vp, _i64, _i32, _vp, _i64, _i32, _vp, _i32, _vp, _i32, _f64,
                                   ctypes.POINTER(Calibration)]
_L.aatc_params_bytes.restype = _sz
_L.aatc_params_bytes.argtypes = [_i32]
_L.aatc_params_pack.restype = ctypes.c_int
_L.aatc_params_pack.argtypes = [ctypes.POINTER(Calibration), _i32, _vp, _sz]
_L.aatc_encode.restype = ctypes.c_int
_L.aatc_encode.argtypes = [_vp, _i32, _i32, _vp, ctypes.c_int, _i64, _i64, ctypes.c_int, _vp,
                           _vp, _i64, _i64, _vp]
_L.aatc_decode_workspace_bytes.restype = _sz
_L.aatc_decode_workspace_bytes.argtypes = [_i32, _i32, _i32, _i64]
_L.aatc_decode_attention.restype = ctypes.c_int
_L.aatc_decode_attention.argtypes = [_vp, _vp, _i32, _i32, _i32, _i32, _vp, ctypes.c_int,
                                     _vp, _vp, _vp, _vp, _vp, _i64, _i32, _i32, _f32, _vp, _vp,
                                     _sz, _vp]
_L.aatc_append_decode_attention.restype = ctypes.c_int
_L.aatc_append_decode_attention.argtypes = [_vp, _vp, _i32, _i32, _i32, _i32, _vp,
                                            ctypes.c_int, _vp, _vp, ctypes.c_int, _vp, _vp, _vp,
                                            _vp, _vp, _i64, _i32, _i32, _f32, _vp, _vp, _sz, _vp]

_L.aatc_append_decode_attention_noalloc.restype = ctypes.c_int
_L.aatc_append_decode_attention_noalloc.argtypes = [_vp, _vp, _i32, _i32, _i32, _i32, _vp,
                                                    ctypes.c_int, _vp, _vp, ctypes.c_int, _vp,
                                                    _vp, _vp, _vp, _vp, _i64, _i32, _i32, _f32,
                                                    _vp, _vp]
_L.aatc_decode_attention_segmented.restype = ctypes.c_int
_L.aatc_decode_attention_segmented.argtypes = [_vp, _vp, _i32, _i32, _i32, _i32, _vp,
                                               ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _i64,
                                               _i32, _i32, _f32, _vp, _vp, ctypes.c_int, _vp,
                                               _i32, _vp, _vp, _sz, _vp]
_L.aatc_segment_counts.restype = ctypes.c_int
_L.aatc_segment_counts.argtypes = [_i64, _i32, _i32, _i32, ctypes.POINTER(ctypes.c_int64),
                                   ctypes.POINTER(ctypes.c_int32)]


def library() -> ctypes.CDLL:
    return _L


def exported_symbols_declared_in_header(header_path: str):
    """Names of the functions include/aatc.h declares."""
    text = open(header_path).read()
    return sorted(set(re.findall(r"\b(aatc_[a-z_0-9]+)\s*\(", text)))


def _status_string(status: int) -> str:
    return _L.aatc_status_string(int(status)).decode()


aatc_status_string = _status_string


def _check(func: str, status: int):
    if status != OK:
        raise AatcError(func, status)


def _np_ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def aatc_calibrate(x_calib, avg_bits: float, b_max: int = 8, percentile: float = 0.99,
                   q_calib=None, q_group: int = 1, w_o=None) -> Calibration:
    """Host calibration of one (KV head, tensor); arrays are float32 numpy arrays."""
    x = np.ascontiguousarray(x_calib, dtype=np.float32)
    q = None if q_calib is None else np.ascontiguousarray(q_calib, dtype=np.float32)
    wo = None if w_o is None else np.ascontiguousarray(w_o, dtype=np.float32)
    out = Calibration()
    st = _L.aatc_calibrate(_np_ptr(x), x.shape[0], x.shape[1] if x.ndim == 2 else 0,
                           _np_ptr(q), 0 if q is None else q.shape[0], int(q_group),
                           _np_ptr(wo), 0 if wo is None else wo.shape[1],
                           float(avg_bits), int(b_max), float(percentile), ctypes.byref(out))
    _check("aatc_calibrate", st)
    return out


def aatc_calibrate_whitened(x_in, w_proj, avg_bits: float, b_max: int = 8,
                            percentile: float = 0.99, q_calib=None, q_group: int = 1,
                            w_o=None) -> Calibration:
    """Host calibration from layer inputs [T, d_model] and a projection [d_model, d]."""
    x = np.ascontiguousarray(x_in, dtype=np.float32)
    w = np.ascontiguousarray(w_proj, dtype=np.float32)
    if x.ndim != 2 or w.ndim != 2 or w.shape[0] != x.shape[1]:
        raise ValueError("x_in must be [T, d_model] and w_proj [d_model, d]")
    q = None if q_calib is None else np.ascontiguousarray(q_calib, dtype=np.float32)
    wo = None if w_o is None else np.ascontiguousarray(w_o, dtype=np.float32)
    out = Calibration()
    st = _L.aatc_calibrate_whitened(_np_ptr(x), x.shape[0], x.shape[1], _np_ptr(w), w.shape[1],
                                    _np_ptr(q), 0 if q is None else q.shape[0], int(q_group),
                                    _np_ptr(wo), 0 if wo is None else wo.shape[1],
                                    float(avg_bits), int(b_max), float(percentile),
                                    ctypes.byref(out))
    _check("aatc_calibrate_whitened", st)
    return out


_L.aatc_allocate_global.restype = ctypes.c_int
_L.aatc_allocate_global.argtypes = [_vp, _vp, _i32, _i32, _f64, _i32, _i32, _i32, _i32, _vp]


def aatc_allocate_global(sigma2, weight, avg_bits: float, b_max: int = 8, n_protect: int = 3,
                         protect_extra: int = 0, normalize_weight: bool = False) -> np.ndarray:
    """Widths [L][m] of one tensor over all layers under one budget (host only)."""
    s2 = np.ascontiguousarray(sigma2, dtype=np.float64)
    if s2.ndim != 2:
        raise ValueError("sigma2 must be [layers][channels]")
    w = None if weight is None else np.ascontiguousarray(weight, dtype=np.float64)
    if w is not None and w.shape != s2.shape:
        raise ValueError("weight and sigma2 differ in shape")
    bits = np.zeros(s2.shape, dtype=np.uint8)
    st = _L.aatc_allocate_global(_np_ptr(s2), None if w is None else _np_ptr(w), s2.shape[0],
                                 s2.shape[1], float(avg_bits), b_max, n_protect, protect_extra,
                                 int(bool(normalize_weight)), _np_ptr(bits))
    _check("aatc_allocate_global", st)
    return bits


def aatc_params_bytes(n_kv_heads: int) -> int:
    return int(_L.aatc_params_bytes(int(n_kv_heads)))


def aatc_params_pack(calibrations) -> np.ndarray:
    """Host parameter block (uint8 numpy array) for a list of per-head Calibration."""
    n = len(calibrations)
    arr = (Calibration * n)(*calibrations)
    buf = np.zeros(aatc_params_bytes(n), dtype=np.uint8)
    _check("aatc_params_pack", _L.aatc_params_pack(arr, n, _np_ptr(buf), buf.nbytes))
    return buf


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(int(stream))
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dptr(t):
    return ctypes.c_void_p(t.data_ptr())


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def aatc_encode(dev_params, n_kv_heads: int, x, n_tok: int, x_tok_stride: int, layout: int,
                codes, alpha, cap: int, pos: int, stream=None):
    """Append n_tok tokens of x ([n_tok, n_kv_heads, 128] view) to a sequence's cache."""
    st = _L.aatc_encode(_dptr(dev_params), int(n_kv_heads), HEAD_DIM, _dptr(x), _dtype_code(x),
                        int(n_tok), int(x_tok_stride), int(layout), _dptr(codes), _dptr(alpha),
                        int(cap), int(pos), _stream(stream))
    _check("aatc_encode", st)


def aatc_decode_workspace_bytes(batch: int, n_q_heads: int, n_kv_heads: int, cap: int) -> int:
    return int(_L.aatc_decode_workspace_bytes(int(batch), int(n_q_heads), int(n_kv_heads),
                                              int(cap)))


def aatc_decode_attention(dev_params_k, dev_params_v, batch: int, n_q_heads: int,
                          n_kv_heads: int, q, k_codes, k_alpha, v_codes, v_alpha, seq_len,
                          cap: int, k_record_bytes: int, v_record_bytes: int,
                          softmax_scale: float, out, workspace, stream=None):
    st = _L.aatc_decode_attention(
        _dptr(dev_params_k), _dptr(dev_params_v), int(batch), int(n_q_heads), int(n_kv_heads),
        HEAD_DIM, _dptr(q), _dtype_code(q), _dptr(k_codes), _dptr(k_alpha), _dptr(v_codes),
        _dptr(v_alpha), _dptr(seq_len), int(cap), int(k_record_bytes), int(v_record_bytes),
        float(softmax_scale), _dptr(out), _dptr(workspace),
        int(workspace.numel() * workspace.element_size()), _stream(stream))
    _check("aatc_decode_attention", st)


def aatc_append_decode_attention(dev_params_k, dev_params_v, batch: int, n_q_heads: int,
                                 n_kv_heads: int, q, x_k, x_v, k_codes, k_alpha, v_codes,
                                 v_alpha, seq_len, cap: int, k_record_bytes: int,
                                 v_record_bytes: int, softmax_scale: float, out, workspace,
                                 stream=None):
    """Appends token seq_len[b] - 1 (x_k[b], x_v[b]: [n_kv_heads][128]) to the caches and
    runs the decode step over the updated caches, in one launch."""
    if _dtype_code(x_k) != _dtype_code(x_v):
        raise AatcError("aatc_append_decode_attention (x_k and x_v dtypes differ)", E_INVALID)
    st = _L.aatc_append_decode_attention(
        _dptr(dev_params_k), _dptr(dev_params_v), int(batch), int(n_q_heads), int(n_kv_heads),
        HEAD_DIM, _dptr(q), _dtype_code(q), _dptr(x_k), _dptr(x_v), _dtype_code(x_k),
        _dptr(k_codes), _dptr(k_alpha), _dptr(v_codes), _dptr(v_alpha), _dptr(seq_len),
        int(cap), int(k_record_bytes), int(v_record_bytes), float(softmax_scale), _dptr(out),
        _dptr(workspace), int(workspace.numel() * workspace.element_size()), _stream(stream))
    _check("aatc_append_decode_attention", st)


def aatc_append_decode_attention_noalloc(dev_params_k, dev_params_v, batch: int, n_q_heads: int,
                                         n_kv_heads: int, q, x_k, x_v, k_codes, k_alpha,
                                         v_codes, v_alpha, seq_len, cap: int,
                                         k_record_bytes: int, v_record_bytes: int,
                                         softmax_scale: float, out, stream=None):
    """aatc_append_decode_attention with the library's static workspace (no allocation)."""
    if _dtype_code(x_k) != _dtype_code(x_v):
        raise AatcError("aatc_append_decode_attention_noalloc (x_k and x_v dtypes differ)",
                        E_INVALID)
    st = _L.aatc_append_decode_attention_noalloc(
        _dptr(dev_params_k), _dptr(dev_params_v), int(batch), int(n_q_heads), int(n_kv_heads),
        HEAD_DIM, _dptr(q), _dtype_code(q), _dptr(x_k), _dptr(x_v), _dtype_code(x_k),
        _dptr(k_codes), _dptr(k_alpha), _dptr(v_codes), _dptr(v_alpha), _dptr(seq_len),
        int(cap), int(k_record_bytes), int(v_record_bytes), float(softmax_scale), _dptr(out),
        _stream(stream))
    _check("aatc_append_decode_attention_noalloc", st)


def aatc_decode_attention_segmented(dev_params_k, dev_params_v, batch: int, n_q_heads: int,
                                    n_kv_heads: int, q, k_codes, k_alpha, v_codes, v_alpha,
                                    seq_len, cap: int, k_record_bytes: int, v_record_bytes: int,
                                    softmax_scale: float, seg_k, seg_v, seg_len, seg_cap: int,
                                    out, workspace, stream=None):
    """Decode attention over the compressed caches plus the full-precision segment
    (seg_k / seg_v: [batch][n_kv_heads][seg_cap][128])."""
    if _dtype_code(seg_k) != _dtype_code(seg_v):
        raise AatcError("aatc_decode_attention_segmented (seg_k and seg_v dtypes differ)",
                        E_INVALID)
    st = _L.aatc_decode_attention_segmented(
        _dptr(dev_params_k), _dptr(dev_params_v), int(batch), int(n_q_heads), int(n_kv_heads),
        HEAD_DIM, _dptr(q), _dtype_code(q), _dptr(k_codes), _dptr(k_alpha), _dptr(v_codes),
        _dptr(v_alpha), _dptr(seq_len), int(cap), int(k_record_bytes), int(v_record_bytes),
        float(softmax_scale), _dptr(seg_k), _dptr(seg_v), _dtype_code(seg_k), _dptr(seg_len),
        int(seg_cap), _dptr(out), _dptr(workspace),
        int(workspace.numel() * workspace.element_size()), _stream(stream))
    _check("aatc_decode_attention_segmented", st)


def aatc_segment_counts(n_tokens: int, sink: int = 4, window: int = 128, step: int = 16):
    """(n_compressed, n_segment) of a sequence under the full-precision sink/window policy."""
    c = ctypes.c_int64()
    g = ctypes.c_int32()
    _check("aatc_segment_counts",
           _L.aatc_segment_counts(int(n_tokens), int(sink), int(window), int(step),
                                  ctypes.byref(c), ctypes.byref(g)))
    return int(c.value), int(g.value)


def aatc_calibrate_bits(x_calib, bits_eig, record_bytes: int = 0, percentile: float = 0.99,
                        q_calib=None, q_group: int = 1, w_o=None) -> Calibration:
    """aatc_calibrate with the widths (eigen order) given, e.g. from aatc_allocate_global."""
    x = np.ascontiguousarray(x_calib, dtype=np.float32)
    b = np.ascontiguousarray(bits_eig, dtype=np.uint8)
    q = None if q_calib is None else np.ascontiguousarray(q_calib, dtype=np.float32)
    wo = None if w_o is None else np.ascontiguousarray(w_o, dtype=np.float32)
    out = Calibration()
    st = _L.aatc_calibrate_bits(_np_ptr(x), x.shape[0], x.shape[1], _np_ptr(q),
                                0 if q is None else q.shape[0], int(q_group), _np_ptr(wo),
                                0 if wo is None else wo.shape[1], _np_ptr(b), int(record_bytes),
                                float(percentile), ctypes.byref(out))
    _check("aatc_calibrate_bits", st)
    return out


# --------------------------------------------------------------------------------------
# Head groups
# --------------------------------------------------------------------------------------
GROUP_MAX_DIM = 512


class GroupCalibration(ctypes.Structure):
    """Mirror of aatc_group_calibration (include/aatc.h); transform rows have stride d."""

    _fields_ = [
        ("d", ctypes.c_int32),
        ("budget_bits", ctypes.c_int32),
        ("record_bytes", ctypes.c_int32),
        ("d_active", ctypes.c_int32),
        ("quantizer", ctypes.c_int32),
        ("transform", ctypes.c_float * (GROUP_MAX_DIM * GROUP_MAX_DIM)),
        ("bits", ctypes.c_uint8 * GROUP_MAX_DIM),
        ("scale_f16", ctypes.c_uint16 * GROUP_MAX_DIM),
        ("perm", ctypes.c_int32 * GROUP_MAX_DIM),
        ("sigma2", ctypes.c_double * GROUP_MAX_DIM),
        ("weight", ctypes.c_double * GROUP_MAX_DIM),
        ("bits_eig", ctypes.c_uint8 * GROUP_MAX_DIM),
    ]

    @property
    def T(self) -> np.ndarray:
        d = self.d
        return np.ctypeslib.as_array(self.transform)[:d * d].reshape(d, d).copy()

    @property
    def bits_np(self) -> np.ndarray:
        return np.ctypeslib.as_array(self.bits)[:self.d].astype(np.int64)

    @property
    def s16(self) -> np.ndarray:
        return np.ctypeslib.as_array(self.scale_f16)[:self.d].copy().view(np.float16)


_L.aatc_calibrate_group.restype = ctypes.c_int
_L.aatc_calibrate_group.argtypes = [_vp, _i64, _i32, _vp, _i64, _i32, _vp, _i32, _f64, _i32,
                                    _f64, ctypes.POINTER(GroupCalibration)]
_L.aatc_group_params_bytes.restype = _sz
_L.aatc_group_params_bytes.argtypes = [_i32]
_L.aatc_group_params_pack.restype = ctypes.c_int
_L.aatc_group_params_pack.argtypes = [ctypes.POINTER(GroupCalibration), _i32, _vp, _sz]
_L.aatc_group_encode.restype = ctypes.c_int
_L.aatc_group_encode.argtypes = [_vp, _i32, _i32, _vp, ctypes.c_int, _i64, _i64, _vp, _vp,
                                 _i64, _i64, _vp]
_L.aatc_group_decode_workspace_bytes.restype = _sz
_L.aatc_group_decode_workspace_bytes.argtypes = [_i32, _i32, _i32, _i32, _i64]
_L.aatc_group_decode_attention.restype = ctypes.c_int
_L.aatc_group_decode_attention.argtypes = [_vp, _vp, _i32, _i32, _i32, _i32, _vp, ctypes.c_int,
                                           _vp, _vp, _vp, _vp, _vp, _i64, _i32, _i32, _f32,
                                           _vp, _vp, _sz, _vp]


def aatc_calibrate_group(x_calib, avg_bits: float, b_max: int = 8, percentile: float = 0.99,
                         q_calib=None, q_group: int = 1, w_o=None) -> GroupCalibration:
    """Host calibration of one (head group, tensor) from its concatenated tokens [n, d]."""
    x = np.ascontiguousarray(x_calib, dtype=np.float32)
    q = None if q_calib is None else np.ascontiguousarray(q_calib, dtype=np.float32)
    wo = None if w_o is None else np.ascontiguousarray(w_o, dtype=np.float32)
    out = GroupCalibration()
    st = _L.aatc_calibrate_group(_np_ptr(x), x.shape[0], x.shape[1] if x.ndim == 2 else 0,
                                 _np_ptr(q), 0 if q is None else q.shape[0], int(q_group),
                                 _np_ptr(wo), 0 if wo is None else wo.shape[1],
                                 float(avg_bits), int(b_max), float(percentile),
                                 ctypes.byref(out))
    _check("aatc_calibrate_group", st)
    return out


def aatc_group_params_bytes(n_groups: int) -> int:
    return int(_L.aatc_group_params_bytes(int(n_groups)))


def aatc_group_params_pack(calibrations) -> np.ndarray:
    """Host parameter block (uint8 numpy array) for a list of per-group GroupCalibration."""
    n = len(calibrations)
    arr = (GroupCalibration * n)(*calibrations)
    buf = np.zeros(aatc_group_params_bytes(n), dtype=np.uint8)
    _check("aatc_group_params_pack", _L.aatc_group_params_pack(arr, n, _np_ptr(buf), buf.nbytes))
    return buf


def aatc_group_encode(dev_params, n_groups: int, gkv: int, x, n_tok: int, x_tok_stride: int,
                      codes, alpha, cap: int, pos: int, stream=None):
    """Append n_tok tokens of x ([n_tok, n_groups * gkv, 128] view) to a sequence's
    group-compressed cache (codes [n_groups][cap][R], alpha [n_groups][cap])."""
    st = _L.aatc_group_encode(_dptr(dev_params), int(n_groups), int(gkv), _dptr(x),
                              _dtype_code(x), int(n_tok), int(x_tok_stride), _dptr(codes),
                              _dptr(alpha), int(cap), int(pos), _stream(stream))
    _check("aatc_group_encode", st)


def aatc_group_decode_workspace_bytes(batch: int, n_q_heads: int, n_kv_heads: int, gkv: int,
                                      cap: int) -> int:
    return int(_L.aatc_group_decode_workspace_bytes(int(batch), int(n_q_heads),
                                                    int(n_kv_heads), int(gkv), int(cap)))


def aatc_group_decode_attention(dev_params_k, dev_params_v, batch: int, n_q_heads: int,
                                n_kv_heads: int, gkv: int, q, k_codes, k_alpha, v_codes,
                                v_alpha, seq_len, cap: int, k_record_bytes: int,
                                v_record_bytes: int, softmax_scale: float, out, workspace,
                                stream=None):
    st = _L.aatc_group_decode_attention(
        _dptr(dev_params_k), _dptr(dev_params_v), int(batch), int(n_q_heads), int(n_kv_heads),
        int(gkv), _dptr(q), _dtype_code(q), _dptr(k_codes), _dptr(k_alpha), _dptr(v_codes),
        _dptr(v_alpha), _dptr(seq_len), int(cap), int(k_record_bytes), int(v_record_bytes),
        float(softmax_scale), _dptr(out), _dptr(workspace),
        int(workspace.numel() * workspace.element_size()), _stream(stream))
    _check("aatc_group_decode_attention", st)
