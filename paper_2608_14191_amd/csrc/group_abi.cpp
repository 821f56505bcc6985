// C ABI of the head-group path: parameter packing, argument validation and dispatch to the
// launchers in group.hip.  No exception crosses the boundary.
#include <algorithm>
#include <cmath>
#include <cstring>

#include "aatc.h"
#include "group.h"
#include "group_launch.h"
#include "launch.h"

using namespace aatc;

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool group_dim_ok(int d) { return d >= 128 && d <= kGMax && d % 128 == 0; }

bool group_calibration_ok(const aatc_group_calibration& c) {
  const int d = c.d;
  if (!group_dim_ok(d)) return false;
  if (c.quantizer != AATC_QUANT_MIDTREAD && c.quantizer != AATC_QUANT_MIDRISE) return false;
  int sum = 0, active = 0, prev = kMaxBits;
  for (int i = 0; i < d; ++i) {
    if (c.bits[i] > kMaxBits || c.bits[i] > prev) return false;   // non-increasing
    prev = c.bits[i];
    sum += c.bits[i];
    if (c.bits[i]) ++active;
  }
  if (!(sum == c.budget_bits && active == c.d_active && sum > 0 &&
        c.record_bytes >= 4 * ((sum + 31) / 32) && c.record_bytes % 4 == 0 &&
        c.record_bytes <= d * kMaxBits / 8))
    return false;
  for (int i = 0; i < d * d; ++i) {
    const double q = std::ldexp((double)c.transform[i], kTFrac);
    if (!(std::fabs(q) <= (double)(1 << kTFrac)) || q != std::nearbyint(q)) return false;
  }
  return true;
}

}  // namespace

extern "C" size_t aatc_group_params_bytes(int32_t n_groups) {
  if (n_groups < 1) return 0;
  return group_params_bytes(n_groups);
}

extern "C" aatc_status aatc_group_params_pack(const aatc_group_calibration* per_group,
                                              int32_t n_groups, void* host_buf, size_t bytes) {
  try {
    if (!per_group || !host_buf || n_groups < 1) return AATC_E_INVALID;
    if (bytes < group_params_bytes(n_groups)) return AATC_E_INVALID;
    for (int g = 0; g < n_groups; ++g) {
      if (!group_calibration_ok(per_group[g])) return AATC_E_INVALID;
      if (per_group[g].d != per_group[0].d ||
          per_group[g].record_bytes != per_group[0].record_bytes ||
          per_group[g].quantizer != per_group[0].quantizer)
        return AATC_E_INVALID;
    }
    std::memset(host_buf, 0, group_params_bytes(n_groups));
    auto* hdr = static_cast<GroupHeader*>(host_buf);
    hdr->magic = kGroupMagic;
    hdr->n_groups = n_groups;
    hdr->d = per_group[0].d;
    hdr->record_bytes = per_group[0].record_bytes;
    for (int g = 0; g < n_groups; ++g) {
      const aatc_group_calibration& c = per_group[g];
      const int d = c.d;
      auto* gp = const_cast<GroupParams*>(group_params(host_buf, g));
      std::memcpy(gp->T, c.transform, sizeof(float) * (size_t)d * d);
      for (int j = 0; j < d; ++j)
        for (int ch = 0; ch < d; ++ch)
          gp->Tqt[(size_t)ch * d + j] =
              (int32_t)std::ldexp((double)c.transform[(size_t)j * d + ch], kTFrac);   // exact
      int off = 0, max_bits = 0;
      for (int ch = 0; ch < d; ++ch) {
        const int b = c.bits[ch];
        gp->bits[ch] = (uint8_t)b;
        gp->bit_off[ch] = (uint16_t)off;
        gp->s16[ch] = b ? c.scale_f16[ch] : 0;
        const double s = b ? f16_bits_to_f64(c.scale_f16[ch]) : 0.0;
        gp->s[ch] = (float)s;
        // fp32 1/s correctly rounded (the fp64 quotient of an 11-bit divisor rounds to
        // fp32 without a double-rounding error)
        gp->inv_s[ch] = (b && s > 0.0) ? (float)(1.0 / s) : 0.0f;
        off += b;
        max_bits = std::max(max_bits, b);
      }
      gp->d = d;
      gp->gkv = d / 128;
      gp->budget = c.budget_bits;
      gp->record_bytes = c.record_bytes;
      gp->d_active = c.d_active;
      gp->quantizer = c.quantizer;
      gp->max_bits = max_bits;
    }
    return AATC_OK;
  } catch (...) {
    return AATC_E_INVALID;
  }
}

extern "C" aatc_status aatc_group_encode(const void* dev_params, int32_t n_groups, int32_t gkv,
                                         const void* x, aatc_dtype x_dtype, int64_t n_tok,
                                         int64_t x_tok_stride, void* codes, uint16_t* alpha,
                                         int64_t cap, int64_t pos, void* stream) {
  if (!dev_params || !x || !codes || !alpha) return AATC_E_INVALID;
  if (n_groups < 1 || gkv < 1 || gkv > 4 || n_tok < 0 || cap < 1 || pos < 0 ||
      pos > cap || n_tok > cap - pos)
    return AATC_E_INVALID;
  if (x_dtype != AATC_F32 && x_dtype != AATC_BF16) return AATC_E_INVALID;
  if (x_tok_stride < (int64_t)n_groups * 128 * gkv) return AATC_E_INVALID;
  if (!aligned16(dev_params) || !aligned16(codes) || !aligned16(alpha)) return AATC_E_INVALID;
  if (!aligned16(x)) return AATC_E_INVALID;
  if (n_tok == 0) return AATC_OK;
  return launch_group_encode(dev_params, n_groups, gkv, x, x_dtype, n_tok, x_tok_stride,
                             codes, alpha, cap, pos, stream);
}

extern "C" size_t aatc_group_decode_workspace_bytes(int32_t batch, int32_t n_q_heads,
                                                    int32_t n_kv_heads, int32_t gkv,
                                                    int64_t cap) {
  if (batch < 1 || n_q_heads < 1 || n_kv_heads < 1 || gkv < 1 || gkv > 4 || cap < 1 ||
      n_kv_heads % gkv || n_q_heads % n_kv_heads)
    return 0;
  return group_decode_workspace_bytes(batch, n_q_heads, n_kv_heads, gkv, cap);
}

extern "C" aatc_status aatc_group_decode_attention(
    const void* dev_params_k, const void* dev_params_v, int32_t batch, int32_t n_q_heads,
    int32_t n_kv_heads, int32_t gkv, const void* q, aatc_dtype q_dtype, const void* k_codes,
    const uint16_t* k_alpha, const void* v_codes, const uint16_t* v_alpha,
    const int32_t* seq_len, int64_t cap, int32_t k_record_bytes, int32_t v_record_bytes,
    float softmax_scale, float* out, void* workspace, size_t ws_bytes, void* stream) {
  if (!dev_params_k || !dev_params_v || !q || !k_codes || !k_alpha || !v_codes || !v_alpha ||
      !seq_len || !out || !workspace)
    return AATC_E_INVALID;
  if (batch < 1 || n_q_heads < 1 || n_kv_heads < 1 || gkv < 1 || gkv > 4 || cap < 1 ||
      n_kv_heads % gkv || n_q_heads % n_kv_heads)
    return AATC_E_INVALID;
  if (q_dtype != AATC_F32 && q_dtype != AATC_BF16) return AATC_E_INVALID;
  if (!std::isfinite(softmax_scale)) return AATC_E_INVALID;
  for (int32_t rb : {k_record_bytes, v_record_bytes})
    if (rb < 4 || rb % 4) return AATC_E_INVALID;
  if (k_record_bytes > kGMaxRecord || v_record_bytes > kGMaxRecord) return AATC_E_UNSUPPORTED;
  const int n_groups = n_kv_heads / gkv;
  if (n_q_heads / n_groups > kGMaxHeads) return AATC_E_UNSUPPORTED;
  for (const void* p : {dev_params_k, dev_params_v, k_codes, v_codes, (const void*)out,
                        (const void*)workspace})
    if (!aligned16(p)) return AATC_E_INVALID;
  if (ws_bytes < group_decode_workspace_bytes(batch, n_q_heads, n_kv_heads, gkv, cap))
    return AATC_E_WORKSPACE;
  return launch_group_decode(dev_params_k, dev_params_v, batch, n_q_heads, n_kv_heads, gkv, q,
                             q_dtype, k_codes, k_alpha, v_codes, v_alpha, seq_len, cap,
                             k_record_bytes, v_record_bytes, softmax_scale, out, workspace,
                             stream);
}
