// Per-token encode arithmetic shared by the encode kernels and the decode kernel's fused
// append (Sec. 5.2 quantizer, fixed-point transform of the canonical encode).  Device
// code only.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "aatc.h"
#include "params.h"

namespace aatc {

__device__ inline float load_elem(const void* x, int dtype, int64_t idx) {
  if (dtype == AATC_BF16) {
    uint32_t b = static_cast<const uint16_t*>(x)[idx];
    return __uint_as_float(b << 16);
  }
  return static_cast<const float*>(x)[idx];
}

// Fixed-point shift of a token: max |x_j| 2^shift lies in [2^13, 2^14) (0 for a zero token).
__device__ inline int token_shift(float max_abs) {
  int e = 0;
  frexpf(max_abs, &e);                             // max_abs = f 2^e, f in [0.5, 1)
  return (max_abs > 0.f) ? (kXLead - (e - 1)) : 0;
}

// h_c from the exact integer sum of X_j Tq_jc: one rounding to fp32.
__device__ inline float fixed_point_result(long long acc, int shift) {
  return (float)ldexp((double)acc, -(shift + kTFrac));
}

// Token scale alpha = fp16(max |r_c| over stored channels) and fp32 1/alpha, correctly
// rounded (an 11-bit divisor: the fp64 quotient rounds to fp32 without double rounding).
__device__ inline __half token_alpha(float max_abs_r) {
  return __float2half_rn(fminf(max_abs_r, 65504.f));
}
__device__ inline float inverse_alpha(__half a16) {
  const float a32 = __half2float(a16);
  return (a32 > 0.f) ? (float)(1.0 / (double)a32) : 0.f;
}

// Quantize one transformed coefficient (canonical fp32 sequence); returns the b-bit two's
// complement pattern of the code.
__device__ inline uint32_t quantize_code(float r, float inv_a, int b) {
  float y = r * inv_a;
  float xq = ldexpf(y, b - 1);
  float f = floorf(xq);
  int code = (int)f + ((xq - f) >= 0.5f ? 1 : 0);
  const int half = 1 << (b - 1);
  code = min(max(code, -half), half - 1);
  return (uint32_t)code & ((1u << b) - 1u);
}

// Position of a token of a 64-token value tile: word 2 v + tile_word(p) of the tile holds
// record bit v of token p at bit tile_bit(p).
__device__ inline int tile_word(int p) { return (p >> 4) >> 1; }
__device__ inline int tile_bit(int p) { return 8 * (p & 3) + 2 * ((p >> 2) & 3) + ((p >> 4) & 1); }

}  // namespace aatc
