// Host launchers of the head-group kernels (group.hip).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "aatc.h"

namespace aatc {

aatc_status launch_group_encode(const void* params, int n_groups, int gkv, const void* x,
                                aatc_dtype x_dtype, int64_t n_tok, int64_t x_tok_stride,
                                void* codes, uint16_t* alpha, int64_t cap, int64_t pos,
                                void* stream);

size_t group_decode_workspace_bytes(int batch, int n_q_heads, int n_kv_heads, int gkv,
                                    int64_t cap);

aatc_status launch_group_decode(const void* params_k, const void* params_v, int batch,
                                int n_q_heads, int n_kv_heads, int gkv, const void* q,
                                aatc_dtype q_dtype, const void* k_codes,
                                const uint16_t* k_alpha, const void* v_codes,
                                const uint16_t* v_alpha, const int32_t* seq_len, int64_t cap,
                                int k_record_bytes, int v_record_bytes, float softmax_scale,
                                float* out, void* workspace, void* stream);

}  // namespace aatc
