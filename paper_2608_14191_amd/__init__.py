"""AATC (Attention-Aware Transform Coding) KV-cache compression on MI355X.

The compute path lives in libaatc.so (host C++ calibration + HIP kernels for gfx950)
behind the C ABI of include/aatc.h; ``_lib`` binds it with the same function names.
"""
from ._lib import (  # noqa: F401
    BF16, F32, HEAD_DIM, LAYOUT_RECORDS, LAYOUT_TILES, MAX_BITS, QUANT_MIDRISE,
    QUANT_MIDTREAD, TILE_TOKENS,
    AatcError, Calibration,
    aatc_allocate_global, aatc_append_decode_attention, aatc_append_decode_attention_noalloc,
    aatc_calibrate, aatc_calibrate_bits, aatc_calibrate_whitened, aatc_decode_attention, aatc_decode_attention_segmented,
    aatc_decode_workspace_bytes, aatc_encode, aatc_segment_counts,
    aatc_params_bytes, aatc_params_pack, aatc_status_string, library,
    GroupCalibration, aatc_calibrate_group, aatc_group_decode_attention,
    aatc_group_decode_workspace_bytes, aatc_group_encode, aatc_group_params_bytes,
    aatc_group_params_pack,
)
