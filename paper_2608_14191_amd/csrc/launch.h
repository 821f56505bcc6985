// Host launchers implemented next to their kernels (encode.hip, decode.hip).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "aatc.h"

namespace aatc {

constexpr int kMaxGroup = 16;     // query heads per KV head handled by one workgroup

uint16_t f64_to_f16_bits(double v);
double f16_bits_to_f64(uint16_t h);

aatc_status launch_encode(const void* params, int n_heads, const void* x, aatc_dtype x_dtype,
                          int64_t n_tok, int64_t x_tok_stride, aatc_layout layout,
                          void* codes, uint16_t* alpha, int64_t cap, int64_t pos,
                          void* stream);

// Encodes token seq_len[b] - 1 of every sequence b (caches [batch][n_heads][cap] ...).
aatc_status launch_encode_last(const void* params, int n_heads, int batch, const void* x,
                               aatc_dtype x_dtype, aatc_layout layout, void* codes,
                               uint16_t* alpha, int64_t cap, int record_bytes,
                               const int32_t* seq_len, void* stream);

// counter_rows: see ws_layout (0: the call's own rows).
size_t decode_workspace_bytes(int batch, int n_q_heads, int n_kv_heads, int64_t cap,
                              int counter_rows = 0);

aatc_status launch_decode(const void* params_k, const void* params_v, int batch,
                          int n_q_heads, int n_kv_heads, const void* q, aatc_dtype q_dtype,
                          const void* k_codes, const uint16_t* k_alpha, const void* v_codes,
                          const uint16_t* v_alpha, const int32_t* seq_len, int64_t cap,
                          int k_record_bytes, int v_record_bytes, float softmax_scale,
                          float* out, void* workspace, void* stream,
                          const void* x_k = nullptr, const void* x_v = nullptr,
                          aatc_dtype x_dtype = AATC_BF16, int counter_rows = 0,
                          const void* seg_k = nullptr, const void* seg_v = nullptr,
                          aatc_dtype seg_dtype = AATC_BF16, const int32_t* seg_len = nullptr,
                          int seg_cap = 0);

// The static workspace of aatc_append_decode_attention_noalloc (noalloc.hip).
constexpr size_t kScratchBytes = (size_t)32 << 20;
constexpr int kScratchRows = 256;      // (sequence, KV head) rows with a fixed counter slot
// This device's static workspace: its address (hipGetSymbolAddress, once per device, with
// the counters region cleared by a kernel on `stream` at that first call).
aatc_status noalloc_scratch(void** ptr, void* stream);

}  // namespace aatc
