// Exact fp32 rounding of a dot product with the stored transform, for the rare tokens whose
// fast-path result cannot be certified.  Plain C++ usable on the host and the device: a
// fixed-point accumulator wide enough to hold any sum of 128 products of a finite fp32
// number and a multiple of 2^-22 of magnitude at most 1, with no rounding at all, then
// one rounding to fp32 (nearest, ties to even, with subnormals), as IEEE 754 defines it.
#pragma once

#include <math.h>
#include <stdint.h>

#if defined(__HIPCC__)
#define AATC_HD __host__ __device__
#else
#define AATC_HD
#endif

namespace aatc {

// Accumulator value = sum_i word_i 2^(32 i - kAccLsb).  A product x Tq 2^-22 with
// x = m 2^e (m < 2^24, e >= -149) and |Tq| <= 2^22 is an integer < 2^46 times 2^(e - 22),
// and e - 22 >= -171; the sum of 128 of them is below 2^(46 + 104 - 22 + 7) = 2^135, so
// bits -171 .. 135 (307 bits with the sign) fit in ten words.
constexpr int kAccWords = 10;
constexpr int kAccLsb = 171;

// Word i (0 <= i < kAccWords, i known at the call) of a 320-bit little-endian integer held
// as ten words, without indexing the array by a run-time value.
AATC_HD inline uint32_t acc_word(const uint32_t (&u)[kAccWords], int i) {
  uint32_t r = 0u;
#pragma unroll
  for (int k = 0; k < kAccWords; ++k) r = (k == i) ? u[k] : r;
  return r;
}

// Adds x Tq 2^-22 (x any finite fp32 value, |Tq| <= 2^22) to the accumulator, exactly.
AATC_HD inline void acc_add(int64_t (&w)[kAccWords], float xv, int32_t t) {
  uint32_t bits;
  __builtin_memcpy(&bits, &xv, 4);
  const uint32_t ef = (bits >> 23) & 255u;
  const uint64_t m = ef ? ((bits & 0x7fffffu) | 0x800000u) : (bits & 0x7fffffu);
  const int e = ef ? (int)ef - 150 : -149;            // x = +-m 2^e
  const uint64_t p = m * (uint64_t)(t < 0 ? -(int64_t)t : (int64_t)t);   // < 2^46
  const bool neg = ((bits >> 31) != 0u) != (t < 0);
  const int k = e - 22 + kAccLsb;                     // bit position of p's lsb, 0 .. 253
#pragma unroll
  for (int i = 0; i < kAccWords; ++i) {
    const int sh = k - 32 * i;
    uint64_t s = 0;
    if (sh >= 0 && sh < 32) s = (p << sh) & 0xffffffffull;
    else if (sh < 0 && sh > -64) s = (p >> (-sh)) & 0xffffffffull;
    w[i] += neg ? -(int64_t)s : (int64_t)s;           // |w_i| < 2^39
  }
}

// The accumulator's value rounded once to fp32 (nearest, ties to even, with subnormals).
AATC_HD inline float acc_round(int64_t (&w)[kAccWords]) {
  // Carries: words 0..8 into [0, 2^32), the sign in the top word.
#pragma unroll
  for (int i = 0; i < kAccWords - 1; ++i) {
    const int64_t c = w[i] >> 32;                     // floor(w_i / 2^32)
    w[i] -= c * 4294967296ll;
    w[i + 1] += c;
  }
  const bool neg = w[kAccWords - 1] < 0;
  uint32_t u[kAccWords];
#pragma unroll
  for (int i = 0; i < kAccWords; ++i) u[i] = (uint32_t)w[i];
  if (neg) {                                          // magnitude: two's complement negation
    uint32_t carry = 1u;
#pragma unroll
    for (int i = 0; i < kAccWords; ++i) {
      const uint64_t v = (uint64_t)(~u[i]) + carry;
      u[i] = (uint32_t)v;
      carry = (uint32_t)(v >> 32);
    }
  }
  int top = -1;                                       // highest set bit
#pragma unroll
  for (int i = 0; i < kAccWords; ++i)
    if (u[i]) top = 32 * i + 31 - __builtin_clz(u[i]);
  if (top < 0) return 0.f;
  // Keep 24 bits from the top, or the bits at and above 2^-149 (lsb position
  // 22 = -149 + kAccLsb) below 2^-126; the kept lsb position L is at least 22.
  const int L = (top - 23 > 22) ? top - 23 : 22;
  const int wi = L >> 5, off = L & 31;
  const uint64_t win = (uint64_t)acc_word(u, wi) | ((uint64_t)acc_word(u, wi + 1) << 32);
  uint32_t mant = (uint32_t)((win >> off) & 0x1ffffffull);   // <= 24 bits set
  const int rb = L - 1;                               // round bit position (>= 21)
  const bool round_bit = (acc_word(u, rb >> 5) >> (rb & 31)) & 1u;
  bool sticky = (acc_word(u, rb >> 5) & ((1u << (rb & 31)) - 1u)) != 0u;
#pragma unroll
  for (int i = 0; i < kAccWords; ++i)
    if (32 * i + 31 < rb && u[i]) sticky = true;
  if (round_bit && (sticky || (mant & 1u))) ++mant;   // may carry to 2^24: still exact
  const float r = ldexpf((float)mant, L - kAccLsb);   // inf beyond the fp32 range
  return neg ? -r : r;
}

// fl32(sum_{j < n} x_j Tq_j 2^-22) exactly rounded.  x_j = xf(j) (any finite fp32 value),
// Tq_j = tq(j) (integers, |Tq_j| <= 2^22), n <= 128.
template <typename XF, typename TQ>
AATC_HD inline float exact_dot_q22(XF xf, TQ tq, int n) {
  int64_t w[kAccWords];
#pragma unroll
  for (int i = 0; i < kAccWords; ++i) w[i] = 0;
#pragma unroll 1
  for (int j = 0; j < n; ++j) acc_add(w, xf(j), tq(j));
  return acc_round(w);
}

#if defined(__HIPCC__)
// The same sum with Tq read from 16-byte-aligned memory, 16 entries per round trip (the
// four loads of a group are issued together), n a multiple of 16.
template <typename XF>
__device__ inline float exact_dot_q22_batched(XF xf, const int4* tq, int n) {
  int64_t w[kAccWords];
#pragma unroll
  for (int i = 0; i < kAccWords; ++i) w[i] = 0;
#pragma unroll 1
  for (int j0 = 0; j0 < n; j0 += 16) {
    int4 v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = tq[j0 / 4 + q];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      acc_add(w, xf(j0 + 4 * q), v[q].x);
      acc_add(w, xf(j0 + 4 * q + 1), v[q].y);
      acc_add(w, xf(j0 + 4 * q + 2), v[q].z);
      acc_add(w, xf(j0 + 4 * q + 3), v[q].w);
    }
  }
  return acc_round(w);
}
#endif

}  // namespace aatc
