// C ABI entry points: argument validation, parameter-block packing and dispatch to
// the HIP launchers.  No exception crosses the boundary.
#include <algorithm>
#include <cmath>
#include <cstring>

#include "aatc.h"
#include "launch.h"
#include "params.h"

using namespace aatc;

namespace {

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// bf16 of a finite fp32 value, round to nearest even, and back (exact).
uint16_t f32_to_bf16_rne(float x) {
  uint32_t u;
  std::memcpy(&u, &x, 4);
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}
float bf16_to_f32(uint16_t h) {
  const uint32_t u = (uint32_t)h << 16;
  float x;
  std::memcpy(&x, &u, 4);
  return x;
}

bool calibration_ok(const aatc_calibration& c) {
  if (c.d != kD) return false;
  if (c.quantizer != AATC_QUANT_MIDTREAD && c.quantizer != AATC_QUANT_MIDRISE) return false;
  int sum = 0, active = 0, prev = kMaxBits;
  for (int i = 0; i < kD; ++i) {
    if (c.bits[i] > kMaxBits || c.bits[i] > prev) return false;   // non-increasing
    prev = c.bits[i];
    sum += c.bits[i];
    if (c.bits[i]) ++active;
  }
  // Records hold at least the budget, in whole dwords (more when the heads of one tensor
  // share the record size of the widest).
  if (!(sum == c.budget_bits && active == c.d_active && sum > 0 &&
        c.record_bytes >= 4 * ((sum + 31) / 32) && c.record_bytes % 4 == 0 &&
        c.record_bytes <= kMaxBudget / 8))
    return false;
  // The stored transform: every entry a multiple of 2^-22 with magnitude at most 1.
  for (int i = 0; i < kD * kD; ++i) {
    const double q = std::ldexp((double)c.transform[i], kTFrac);
    if (!(std::fabs(q) <= (double)(1 << kTFrac)) || q != std::nearbyint(q)) return false;
  }
  return true;
}

}  // namespace

extern "C" const char* aatc_status_string(aatc_status s) {
  switch (s) {
    case AATC_OK: return "ok";
    case AATC_E_INVALID: return "invalid argument";
    case AATC_E_UNSUPPORTED: return "unsupported configuration";
    case AATC_E_NUMERIC: return "numerical failure";
    case AATC_E_DEVICE: return "device error";
    case AATC_E_WORKSPACE: return "workspace too small";
  }
  return "unknown status";
}

extern "C" size_t aatc_params_bytes(int32_t n_kv_heads) {
  if (n_kv_heads < 1) return 0;
  return params_bytes(n_kv_heads);
}

extern "C" aatc_status aatc_params_pack(const aatc_calibration* per_head, int32_t n_kv_heads,
                                        void* host_buf, size_t bytes) {
  try {
    if (!per_head || !host_buf || n_kv_heads < 1) return AATC_E_INVALID;
    if (bytes < params_bytes(n_kv_heads)) return AATC_E_INVALID;
    for (int h = 0; h < n_kv_heads; ++h) {
      if (!calibration_ok(per_head[h])) return AATC_E_INVALID;
      if (per_head[h].record_bytes != per_head[0].record_bytes) return AATC_E_INVALID;
      if (per_head[h].quantizer != per_head[0].quantizer) return AATC_E_INVALID;
    }
    std::memset(host_buf, 0, params_bytes(n_kv_heads));
    auto* hdr = static_cast<TensorHeader*>(host_buf);
    hdr->magic = kMagic;
    hdr->n_heads = n_kv_heads;
    hdr->budget = per_head[0].budget_bits;
    hdr->record_bytes = per_head[0].record_bytes;
    for (int h = 0; h < n_kv_heads; ++h) {
      const aatc_calibration& c = per_head[h];
      auto* hp = const_cast<HeadParams*>(head_params(host_buf, h));
      std::memcpy(hp->T, c.transform, sizeof(hp->T));
      for (int w = 0; w < 8; ++w)
        for (int kk = 0; kk < 4; ++kk)
          for (int l = 0; l < 64; ++l)
            for (int e = 0; e < 8; ++e) {
              const float x = c.transform[(16 * w + l % 16) * kD + 32 * kk + 8 * (l / 16) + e];
              const uint16_t hi = f32_to_bf16_rne(x);
              const uint16_t lo = f32_to_bf16_rne(x - bf16_to_f32(hi));
              hp->Tm[(((w * 4 + kk) * 2 + 0) * 64 + l) * 8 + e] = hi;
              hp->Tm[(((w * 4 + kk) * 2 + 1) * 64 + l) * 8 + e] = lo;
            }
      for (int j = 0; j < kD; ++j)
        for (int ch = 0; ch < kD; ++ch)
          hp->Tqt[ch * kD + j] =
              (int32_t)std::ldexp((double)c.transform[j * kD + ch], kTFrac);   // exact
      float inv_s_max = 0.f;
      int off = 0, max_bits = 0;
      for (int ch = 0; ch < kD; ++ch) {
        const int b = c.bits[ch];
        hp->bits[ch] = (uint8_t)b;
        hp->bit_off[ch] = (uint16_t)off;
        hp->s16[ch] = c.scale_f16[ch];
        const double s = b ? f16_bits_to_f64(c.scale_f16[ch]) : 0.0;
        hp->s[ch] = (float)s;
        // fp32 1/s correctly rounded: the fp64 quotient of an 11-bit divisor rounds
        // to fp32 without a double-rounding error.
        hp->inv_s[ch] = (b && s > 0.0) ? (float)(1.0 / s) : 0.0f;
        hp->half_step[ch] = (b && c.quantizer == AATC_QUANT_MIDRISE) ? std::ldexp(1.0f, -b) : 0.0f;
        max_bits = std::max(max_bits, b);
        inv_s_max = std::fmax(inv_s_max, hp->inv_s[ch]);
        for (int k = 0; k < b; ++k) {
          const int v = off + k;
          hp->virt_chan[v] = (uint8_t)ch;
          hp->virt_bit[v] = (uint8_t)k;
          hp->bit_desc[((v >> 5) * 8 + (v & 7)) * 4 + ((v >> 3) & 3)] =
              (uint16_t)(0x8000 | (k == b - 1 ? 0x4000 : 0) | ((kDescBias + k + 1 - b) << 8) | ch);
        }
        off += b;
      }
      hp->d_active = c.d_active;
      hp->budget = c.budget_bits;
      hp->record_bytes = c.record_bytes;
      hp->inv_s_max = inv_s_max;
      hp->quantizer = c.quantizer;
      hp->max_bits = max_bits;
    }
    return AATC_OK;
  } catch (...) {
    return AATC_E_INVALID;
  }
}

extern "C" aatc_status aatc_encode(const void* dev_params, int32_t n_kv_heads, int32_t d,
                                   const void* x, aatc_dtype x_dtype, int64_t n_tok,
                                   int64_t x_tok_stride, aatc_layout layout, void* codes,
                                   uint16_t* alpha, int64_t cap, int64_t pos, void* stream) {
  try {
    if (d != kD) return AATC_E_UNSUPPORTED;
    if (!dev_params || !x || !codes || !alpha) return AATC_E_INVALID;
    if (n_kv_heads < 1 || n_tok < 0 || cap < 1 || pos < 0 || pos + n_tok > cap)
      return AATC_E_INVALID;
    if (x_dtype != AATC_F32 && x_dtype != AATC_BF16) return AATC_E_INVALID;
    if (layout != AATC_LAYOUT_RECORDS && layout != AATC_LAYOUT_TILES) return AATC_E_INVALID;
    if (layout == AATC_LAYOUT_TILES && cap % kTile != 0) return AATC_E_INVALID;
    if (x_tok_stride < (int64_t)n_kv_heads * d) return AATC_E_INVALID;
    if (!aligned(dev_params, 16) || !aligned(codes, 16) || !aligned(alpha, 2) ||
        !aligned(x, x_dtype == AATC_F32 ? 4 : 2))
      return AATC_E_INVALID;
    if (n_tok == 0) return AATC_OK;
    return launch_encode(dev_params, n_kv_heads, x, x_dtype, n_tok, x_tok_stride, layout,
                         codes, alpha, cap, pos, stream);
  } catch (...) {
    return AATC_E_INVALID;
  }
}

extern "C" size_t aatc_decode_workspace_bytes(int32_t batch, int32_t n_q_heads,
                                              int32_t n_kv_heads, int64_t cap) {
  if (batch < 1 || n_q_heads < 1 || n_kv_heads < 1 || cap < 0) return 0;
  return decode_workspace_bytes(batch, n_q_heads, n_kv_heads, cap);
}

namespace {

aatc_status check_decode(const void* dev_params_k, const void* dev_params_v, int32_t batch,
                         int32_t n_q_heads, int32_t n_kv_heads, int32_t d, const void* q,
                         aatc_dtype q_dtype, const void* k_codes, const uint16_t* k_alpha,
                         const void* v_codes, const uint16_t* v_alpha, const int32_t* seq_len,
                         int64_t cap, int32_t k_record_bytes, int32_t v_record_bytes,
                         float softmax_scale, const float* out, const void* workspace,
                         size_t ws_bytes, bool static_ws = false) {
  if (d != kD) return AATC_E_UNSUPPORTED;
  if (!dev_params_k || !dev_params_v || !q || !k_codes || !k_alpha || !v_codes || !v_alpha ||
      !seq_len || !out || (!workspace && !static_ws))
    return AATC_E_INVALID;
  if (batch < 1 || n_q_heads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads != 0)
    return AATC_E_INVALID;
  if (n_q_heads / n_kv_heads > kMaxGroup) return AATC_E_UNSUPPORTED;
  if (cap < kTile || cap % kTile != 0) return AATC_E_INVALID;
  if (k_record_bytes < 4 || k_record_bytes > kMaxBudget / 8 || k_record_bytes % 4 != 0 ||
      v_record_bytes < 4 || v_record_bytes > kMaxBudget / 8 || v_record_bytes % 4 != 0)
    return AATC_E_INVALID;
  if (q_dtype != AATC_F32 && q_dtype != AATC_BF16) return AATC_E_INVALID;
  if (!std::isfinite(softmax_scale)) return AATC_E_INVALID;
  if (!aligned(dev_params_k, 16) || !aligned(dev_params_v, 16) || !aligned(k_codes, 16) ||
      !aligned(v_codes, 16) || !aligned(k_alpha, 16) || !aligned(v_alpha, 16) ||
      !aligned(seq_len, 4) || !aligned(out, 16) || !aligned(workspace, 256) ||
      !aligned(q, q_dtype == AATC_F32 ? 4 : 2))
    return AATC_E_INVALID;
  if (static_ws) {
    if ((int64_t)batch * n_kv_heads > kScratchRows ||
        decode_workspace_bytes(batch, n_q_heads, n_kv_heads, cap, kScratchRows) > kScratchBytes)
      return AATC_E_WORKSPACE;
  } else if (ws_bytes < decode_workspace_bytes(batch, n_q_heads, n_kv_heads, cap)) {
    return AATC_E_WORKSPACE;
  }
  return AATC_OK;
}

aatc_status check_new_tokens(const void* x_k, const void* x_v, aatc_dtype x_dtype) {
  if (!x_k || !x_v) return AATC_E_INVALID;
  if (x_dtype != AATC_F32 && x_dtype != AATC_BF16) return AATC_E_INVALID;
  const size_t xa = x_dtype == AATC_F32 ? 4 : 2;
  if (!aligned(x_k, xa) || !aligned(x_v, xa)) return AATC_E_INVALID;
  return AATC_OK;
}

}  // namespace

extern "C" aatc_status aatc_decode_attention(
    const void* dev_params_k, const void* dev_params_v, int32_t batch, int32_t n_q_heads,
    int32_t n_kv_heads, int32_t d, const void* q, aatc_dtype q_dtype, const void* k_codes,
    const uint16_t* k_alpha, const void* v_codes, const uint16_t* v_alpha,
    const int32_t* seq_len, int64_t cap, int32_t k_record_bytes, int32_t v_record_bytes,
    float softmax_scale, float* out, void* workspace, size_t ws_bytes, void* stream) {
  try {
    const aatc_status e = check_decode(dev_params_k, dev_params_v, batch, n_q_heads, n_kv_heads,
                                       d, q, q_dtype, k_codes, k_alpha, v_codes, v_alpha,
                                       seq_len, cap, k_record_bytes, v_record_bytes,
                                       softmax_scale, out, workspace, ws_bytes);
    if (e != AATC_OK) return e;
    return launch_decode(dev_params_k, dev_params_v, batch, n_q_heads, n_kv_heads, q, q_dtype,
                         k_codes, k_alpha, v_codes, v_alpha, seq_len, cap, k_record_bytes,
                         v_record_bytes, softmax_scale, out, workspace, stream);
  } catch (...) {
    return AATC_E_INVALID;
  }
}

extern "C" aatc_status aatc_append_decode_attention(
    const void* dev_params_k, const void* dev_params_v, int32_t batch, int32_t n_q_heads,
    int32_t n_kv_heads, int32_t d, const void* q, aatc_dtype q_dtype, const void* x_k,
    const void* x_v, aatc_dtype x_dtype, void* k_codes, uint16_t* k_alpha, void* v_codes,
    uint16_t* v_alpha, const int32_t* seq_len, int64_t cap, int32_t k_record_bytes,
    int32_t v_record_bytes, float softmax_scale, float* out, void* workspace, size_t ws_bytes,
    void* stream) {
  try {
    const aatc_status e = check_decode(dev_params_k, dev_params_v, batch, n_q_heads, n_kv_heads,
                                       d, q, q_dtype, k_codes, k_alpha, v_codes, v_alpha,
                                       seq_len, cap, k_record_bytes, v_record_bytes,
                                       softmax_scale, out, workspace, ws_bytes);
    if (e != AATC_OK) return e;
    const aatc_status ex = check_new_tokens(x_k, x_v, x_dtype);
    if (ex != AATC_OK) return ex;
    return launch_decode(dev_params_k, dev_params_v, batch, n_q_heads, n_kv_heads, q, q_dtype,
                         k_codes, k_alpha, v_codes, v_alpha, seq_len, cap, k_record_bytes,
                         v_record_bytes, softmax_scale, out, workspace, stream, x_k, x_v,
                         x_dtype);
  } catch (...) {
    return AATC_E_INVALID;
  }
}

extern "C" aatc_status aatc_decode_attention_segmented(
    const void* dev_params_k, const void* dev_params_v, int32_t batch, int32_t n_q_heads,
    int32_t n_kv_heads, int32_t d, const void* q, aatc_dtype q_dtype, const void* k_codes,
    const uint16_t* k_alpha, const void* v_codes, const uint16_t* v_alpha,
    const int32_t* seq_len, int64_t cap, int32_t k_record_bytes, int32_t v_record_bytes,
    float softmax_scale, const void* seg_k, const void* seg_v, aatc_dtype seg_dtype,
    const int32_t* seg_len, int32_t seg_cap, float* out, void* workspace, size_t ws_bytes,
    void* stream) {
  try {
    const aatc_status e = check_decode(dev_params_k, dev_params_v, batch, n_q_heads, n_kv_heads,
                                       d, q, q_dtype, k_codes, k_alpha, v_codes, v_alpha,
                                       seq_len, cap, k_record_bytes, v_record_bytes,
                                       softmax_scale, out, workspace, ws_bytes);
    if (e != AATC_OK) return e;
    if (!seg_k || !seg_v || !seg_len) return AATC_E_INVALID;
    if (seg_dtype != AATC_F32 && seg_dtype != AATC_BF16) return AATC_E_INVALID;
    if (seg_cap < 1 || seg_cap > 256) return AATC_E_INVALID;
    const size_t sa = seg_dtype == AATC_F32 ? 4 : 2;
    if (!aligned(seg_k, sa) || !aligned(seg_v, sa) || !aligned(seg_len, 4)) return AATC_E_INVALID;
    return launch_decode(dev_params_k, dev_params_v, batch, n_q_heads, n_kv_heads, q, q_dtype,
                         k_codes, k_alpha, v_codes, v_alpha, seq_len, cap, k_record_bytes,
                         v_record_bytes, softmax_scale, out, workspace, stream, nullptr, nullptr,
                         AATC_BF16, 0, seg_k, seg_v, seg_dtype, seg_len, seg_cap);
  } catch (...) {
    return AATC_E_INVALID;
  }
}

extern "C" aatc_status aatc_segment_counts(int64_t n_tokens, int32_t sink, int32_t window,
                                           int32_t step, int64_t* n_compressed,
                                           int32_t* n_segment) {
  if (!n_compressed || !n_segment) return AATC_E_INVALID;
  if (n_tokens < 0 || sink < 0 || window < 1 || step < 1 || step > window)
    return AATC_E_INVALID;
  const int64_t m = n_tokens > sink ? n_tokens - sink : 0;    // tokens after the sink
  const int64_t c = m < window ? 0 : (int64_t)step * ((m - window) / step + 1);
  *n_compressed = c;
  *n_segment = (int32_t)(n_tokens - c);
  return AATC_OK;
}

extern "C" aatc_status aatc_append_decode_attention_noalloc(
    const void* dev_params_k, const void* dev_params_v, int32_t batch, int32_t n_q_heads,
    int32_t n_kv_heads, int32_t d, const void* q, aatc_dtype q_dtype, const void* x_k,
    const void* x_v, aatc_dtype x_dtype, void* k_codes, uint16_t* k_alpha, void* v_codes,
    uint16_t* v_alpha, const int32_t* seq_len, int64_t cap, int32_t k_record_bytes,
    int32_t v_record_bytes, float softmax_scale, float* out, void* stream) {
  try {
    const aatc_status e = check_decode(dev_params_k, dev_params_v, batch, n_q_heads, n_kv_heads,
                                       d, q, q_dtype, k_codes, k_alpha, v_codes, v_alpha,
                                       seq_len, cap, k_record_bytes, v_record_bytes,
                                       softmax_scale, out, nullptr, 0, true);
    if (e != AATC_OK) return e;
    const aatc_status ex = check_new_tokens(x_k, x_v, x_dtype);
    if (ex != AATC_OK) return ex;
    void* ws = nullptr;
    const aatc_status es = noalloc_scratch(&ws, stream);
    if (es != AATC_OK) return es;
    return launch_decode(dev_params_k, dev_params_v, batch, n_q_heads, n_kv_heads, q, q_dtype,
                         k_codes, k_alpha, v_codes, v_alpha, seq_len, cap, k_record_bytes,
                         v_record_bytes, softmax_scale, out, ws, stream, x_k, x_v, x_dtype,
                         kScratchRows);
  } catch (...) {
    return AATC_E_INVALID;
  }
}
