// Per-token encode arithmetic shared by the encode kernels and the decode kernel's fused
// append (Sec. 5.2 quantizer; the transform of Alg. 1 "project", h = T^T x, rounded once
// to fp32 from its exact value).  Device code only.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "aatc.h"
#include "exact_dot.h"
#include "params.h"

namespace aatc {

__device__ inline float load_elem(const void* x, int dtype, int64_t idx) {
  if (dtype == AATC_BF16) {
    uint32_t b = static_cast<const uint16_t*>(x)[idx];
    return __uint_as_float(b << 16);
  }
  return static_cast<const float*>(x)[idx];
}

// Fixed-point shift of a token for the integer transform: max |x_j| 2^shift lies in
// [2^21, 2^22), so X_j = rint(x_j 2^shift) splits into three balanced int8 limbs (0 for a
// zero token).  X_j equals x_j 2^shift exactly unless |x_j| is below about 2^-14 max |x|
// (bf16) or carries more bits (fp32).
__device__ inline int token_shift(float max_abs) {
  int e = 0;
  frexpf(max_abs, &e);                             // max_abs = f 2^e, f in [0.5, 1)
  return (max_abs > 0.f) ? (kXLead - (e - 1)) : 0;
}

// h = fl32(H 2^-(shift + 22)) for the exact integer H = sum_j X_j Tq_j (|H| < 2^51, exact
// in fp64): when every X_j is exact this is the canonical h.
__device__ inline float integer_result(double H, int shift) {
  return (float)ldexp(H, -(shift + kTFrac));
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
// complement pattern of the code.  Midtread: floor(x + 1/2) taken exactly; midrise:
// floor(x) (its level is (code + 1/2) Delta).
__device__ inline uint32_t quantize_code(float r, float inv_a, int b, bool midrise) {
  float y = r * inv_a;
  float xq = ldexpf(y, b - 1);
  float f = floorf(xq);
  int code = (int)f + ((!midrise && (xq - f) >= 0.5f) ? 1 : 0);
  const int half = 1 << (b - 1);
  code = min(max(code, -half), half - 1);
  return (uint32_t)code & ((1u << b) - 1u);
}

// Distance of a quantizer input x to the nearest decision boundary of its reading:
// half-integers for midtread (round half up), integers for midrise (floor).
__device__ inline float boundary_distance(float x, bool midrise) {
  const float f = floorf(x);
  const float frac = x - f;                         // exact, in [0, 1)
  return midrise ? fminf(frac, 1.f - frac) : fabsf(frac - 0.5f);
}

// Position of a token of a 64-token value tile: word 2 v + tile_word(p) of the tile holds
// record bit v of token p at bit tile_bit(p).
__device__ inline int tile_word(int p) { return (p >> 4) >> 1; }
__device__ inline int tile_bit(int p) { return 8 * (p & 3) + 2 * ((p >> 2) & 3) + ((p >> 4) & 1); }

__device__ inline float wave_max64(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// The exact fallback for one channel: h_c from the token (element j held by lane j % 64
// of the wave, in xl[j / 64]) and column c of the integer transform, read 16 entries per
// round trip.
__device__ inline float exact_h_channel(const float (&xl)[2], const int32_t* tcol) {
  // (j is uniform; the register is chosen by j, not per lane: the caller may run this with
  // some lanes inactive, and readlane reads the chosen register of any lane)
  return exact_dot_q22_batched(
      [&](int j) {
        const int a = __builtin_amdgcn_readlane(__float_as_int(xl[0]), j & 63);
        const int b = __builtin_amdgcn_readlane(__float_as_int(xl[1]), j & 63);
        return __int_as_float(j < 64 ? a : b);
      },
      reinterpret_cast<const int4*>(tcol), kD);
}

// The same with the token's elements and the column read one entry at a time from memory:
// fewer registers (for kernels that call it with much else live), one round trip per entry.
__device__ inline float exact_h_channel_lean(const void* xrow, int dtype, const int32_t* tcol) {
  return exact_dot_q22([&](int j) { return load_elem(xrow, dtype, j); },
                       [&](int j) { return tcol[j]; }, kD);
}

// The exponent of the lowest set bit over a token's nonzero elements (element j held by lane
// j % 64 of the wave, in xl[j / 64]): every x_j is a multiple of 2^g.  4096 for a zero token.
__device__ inline int token_lsb(const float (&xl)[2]) {
  int g = 4096;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const uint32_t b = __float_as_uint(xl[i]) & 0x7fffffffu;
    if (b != 0u) {
      const int ef = (int)(b >> 23), m = (int)(b & 0x7fffffu);
      g = min(g, ef ? ef - 150 + __builtin_ctz((uint32_t)m | 0x800000u) : -149 + __builtin_ctz((uint32_t)m));
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) g = min(g, __shfl_xor(g, o, 64));
  return g;
}

// r_c = fl32(h_c (1/s_c)) for channels c = lane and lane + 64 of one token, from the fp64
// sums s_i = sum_j x_j Tq_jc and a_i = sum_j |x_j Tq_jc| (every product exact: at most
// 24 + 23 bits).  Every product, hence every partial sum, is a multiple of 2^g (g from
// token_lsb); while a_i stays below 2^(53 + g) each of them is an fp64 number, s_i is exact
// and one rounding gives h_c (ties included).  Otherwise s_i is within 128 2^-53 (1 + tiny)
// a_i of its exact value: where that interval, scaled by 2^-22, rounds to one fp32 number
// it is h_c, elsewhere the exact accumulator of exact_dot.h decides (xl / xrow / dtype: the
// token, as below).
template <bool LEAN = false>
__device__ inline void exact_r_finish(const HeadParams* hp, const double (&s)[2],
                                      const double (&a)[2], int g, const float (&xl)[2],
                                      const void* xrow, int dtype, float (&r)[2]) {
  const int lane = threadIdx.x & 63;
  // (a_i itself is within 128 2^-53 of the exact sum of |products|)
  const double lim = ldexp(1.0 - 0x1p-40, 53 + min(g, 900));
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = lane + 64 * i;
    const double sv = ldexp(s[i], -kTFrac), av = ldexp(a[i], -kTFrac);
    float h;
    if (a[i] < lim) {
      h = (float)sv;
    } else {
      const double b = av * (kD * 0x1p-52);
      const double bb = b * (1.0 + 0x1p-48) + fabs(sv) * 0x1p-51 + 0x1p-1060;
      const float lo = (float)(sv - bb), hi = (float)(sv + bb);
      h = lo;
      // (a dropped channel's r is 0 whatever h is)
      if (lo != hi && hp->bits[c] > 0)
        h = LEAN ? exact_h_channel_lean(xrow, dtype, hp->Tqt + c * kD)
                 : exact_h_channel(xl, hp->Tqt + c * kD);
    }
    r[i] = h * hp->inv_s[c];
  }
}

// The same for one wave holding the token: xl holds this lane's elements lane and
// lane + 64 (as fp32), xrow / dtype address the token in memory for the exact fallback;
// the transform is read from the parameter block, 16 entries per round trip.
// LEAN selects the exact routine's register-light form.
template <bool LEAN = false>
__device__ inline void exact_r_wave(const HeadParams* hp, const float (&xl)[2],
                                    const void* xrow, int dtype, float (&r)[2]) {
  const int lane = threadIdx.x & 63;
  double s[2] = {0.0, 0.0}, a[2] = {0.0, 0.0};
  const int4* tc[2] = {reinterpret_cast<const int4*>(hp->Tqt + lane * kD),
                       reinterpret_cast<const int4*>(hp->Tqt + (lane + 64) * kD)};
#pragma unroll 1
  for (int jb = 0; jb < kD; jb += 16) {
    int4 tv[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) tv[i][q] = tc[i][jb / 4 + q];
    const float xw = (jb < 64) ? xl[0] : xl[1];
#pragma unroll
    for (int jj = 0; jj < 16; ++jj) {
      const double xd =
          (double)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(xw), (jb + jj) & 63));
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int4 t4 = tv[i][jj >> 2];
        const int ti = (jj & 3) == 0 ? t4.x : (jj & 3) == 1 ? t4.y : (jj & 3) == 2 ? t4.z : t4.w;
        const double t = (double)ti;
        s[i] = fma(xd, t, s[i]);
        a[i] = fma(fabs(xd), fabs(t), a[i]);
      }
    }
  }
  exact_r_finish<LEAN>(hp, s, a, token_lsb(xl), xl, xrow, dtype, r);
}

// Certificate of a token encoded from the fixed-point transform (one wave, lane l:
// channels l and l + 64): r holds fl32(fl32(h~) / s) with |h - h~| <= eh for the exact h.
// True if the fp16 scale and every code are certainly those of the exact transform: the
// fp16 rounding of the largest |r| cannot change within the bound, and no code's
// quantizer input lies within the bound (in its units, plus the fp32 roundings of both
// evaluations) of a rounding boundary.
__device__ inline bool wave_certify(const HeadParams* hp, const float (&r)[2], float eh) {
  const int lane = threadIdx.x & 63;
  int b[2];
  float m = 0.f;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    b[i] = hp->bits[lane + 64 * i];
    m = fmaxf(m, b[i] > 0 ? fabsf(r[i]) : 0.f);
  }
  const float amax = wave_max64(m);
  const __half a16 = token_alpha(amax);
  const float inv = inverse_alpha(a16);
  // The range of the exact max |r_c|: each r_c within eh / s_c of its computed value (plus
  // the fp32 roundings, the 2^-21 amax slack).
  float lo = 0.f, hi = 0.f;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float er = eh * hp->inv_s[lane + 64 * i] * (1.f + 0x1p-20f);
    const float ar = b[i] > 0 ? fabsf(r[i]) : 0.f;
    lo = fmaxf(lo, ar - er);
    hi = fmaxf(hi, ar + er);
  }
  lo = wave_max64(lo) - 0x1p-21f * amax;
  hi = wave_max64(hi) + 0x1p-21f * amax + 0x1p-140f;
  bool ok = __half_as_ushort(token_alpha(fmaxf(lo, 0.f))) ==
            __half_as_ushort(token_alpha(hi));
  const float ea = eh * inv;
  const bool midrise = hp->quantizer == AATC_QUANT_MIDRISE;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    if (b[i] > 0) {
      const float xq = ldexpf(r[i] * inv, b[i] - 1);
      const float k = ldexpf(hp->inv_s[lane + 64 * i], b[i] - 1) * (1.f + 0x1p-20f);
      const float mg = fmaf(k, ea, fmaf(0x1p-21f, fabsf(xq), 0x1p-22f));
      ok = ok && (boundary_distance(xq, midrise) > mg);
    }
  }
  return __builtin_amdgcn_ballot_w64(!ok) == 0ull;
}

// One token's codes from r (lane l: channels l and l + 64, one wave), OR-ed into its
// record row `rec` (zero on entry; LDS); returns the fp16 token scale.
__device__ inline __half wave_quantize_into(const HeadParams* hp, const float (&r)[2],
                                            uint32_t* rec) {
  const int lane = threadIdx.x & 63;
  int b[2], off[2];
  float m = 0.f;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    b[i] = hp->bits[lane + 64 * i];
    off[i] = hp->bit_off[lane + 64 * i];
    m = fmaxf(m, b[i] > 0 ? fabsf(r[i]) : 0.f);
  }
  const __half a16 = token_alpha(wave_max64(m));
  const float inv = inverse_alpha(a16);
  const bool midrise = hp->quantizer == AATC_QUANT_MIDRISE;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    if (b[i] > 0) {
      const uint32_t u = quantize_code(r[i], inv, b[i], midrise);
      atomicOr(&rec[off[i] >> 5], u << (off[i] & 31));
      if ((off[i] & 31) + b[i] > 32) atomicOr(&rec[(off[i] >> 5) + 1], u >> (32 - (off[i] & 31)));
    }
  }
  return a16;
}

}  // namespace aatc
