// Device parameter block of one tensor (keys or values): a header followed by one
// HeadParams per KV head.  Built on the host by aatc_params_pack, read by the
// encode and decode kernels.  Shared between host and device code.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace aatc {

constexpr int kD = 128;                   // head dimension
constexpr int kMaxBits = 16;              // widest channel code
constexpr int kMaxBudget = kD * kMaxBits; // most bits per token record
constexpr int kTile = 64;                 // tokens per value-cache tile
constexpr int kTFrac = 22;                // the stored transform: multiples of 2^-22
constexpr int kXLead = 21;                // encoder: per-token x scaled into [2^21, 2^22)
constexpr uint32_t kMagic = 0x43544141u;  // "AATC"

struct alignas(256) HeadParams {
  float T[kD * kD];               // [j][c] stored transform (multiples of 2^-22, exact fp32)
  // The same transform as two bf16 terms, Th = bf16(T) and Tl = bf16(T - Th), laid out as
  // the decode merge's matrix-core A operands: 16-byte unit ((4 w + kk) 2 + t) 64 + l holds
  // term t (0: Th, 1: Tl) of T[16 w + l % 16][32 kk + 8 (l / 16) .. + 7], w < 8, kk < 4,
  // l < 64 (8 KiB per block of 16 rows).
  uint16_t Tm[2 * kD * kD];
  int32_t Tqt[kD * kD];           // [c][j] T * 2^22 (integers, |Tq| <= 2^22), transposed
  float inv_s[kD];                // fp32 1/s_c (0 for dropped or zero-scale channels)
  float s[kD];                    // s_c as fp32 (exact value of the fp16 scale)
  uint16_t s16[kD];               // s_c fp16 bits
  uint8_t bits[kD];               // width of storage channel c
  uint16_t bit_off[kD];           // first record bit of channel c
  uint8_t virt_chan[kMaxBudget];  // record bit v -> storage channel
  uint8_t virt_bit[kMaxBudget];   // record bit v -> bit index inside that channel's code
  // Record bit v = 32 D + 8 j + d described at [(8 D + d) * 4 + j]: storage channel c
  // (bits 0-6), kDescBias + k + 1 - b_c for bit k of a b_c-bit code (bits 8-11), sign
  // bit of the code (bit 14), bit in use (bit 15).
  uint16_t bit_desc[kMaxBudget];
  int32_t d_active;
  int32_t budget;
  int32_t record_bytes;
  float inv_s_max;                // largest 1/s_c over the stored channels
  int32_t quantizer;              // aatc_quantizer (0 midtread, 1 midrise)
  int32_t max_bits;               // widest channel
  int32_t pad_[2];
  // Midrise: 2^(-b_c) for stored channels (0 for dropped ones and for midtread), the
  // extra half step of every level in units of alpha s_c.
  float half_step[kD];
};
// bit_desc exponent field offset: k + 1 - b_c lies in [1 - kMaxBits, 0].
constexpr int kDescBias = kMaxBits - 1;

// The decode kernel reads these fields with 16-, 8- and 4-byte vector loads.
static_assert(offsetof(HeadParams, T) % 16 == 0, "T alignment");
static_assert(offsetof(HeadParams, Tm) % 16 == 0, "Tm alignment");
static_assert(offsetof(HeadParams, Tqt) % 16 == 0, "Tqt alignment");
static_assert(offsetof(HeadParams, s) % 16 == 0, "s alignment");
static_assert(offsetof(HeadParams, bit_off) % 8 == 0, "bit_off alignment");
static_assert(offsetof(HeadParams, bits) % 4 == 0, "bits alignment");
static_assert(offsetof(HeadParams, bit_desc) % 8 == 0, "bit_desc alignment");
static_assert(offsetof(HeadParams, half_step) % 16 == 0, "half_step alignment");

struct alignas(256) TensorHeader {
  uint32_t magic;
  int32_t n_heads;
  int32_t budget;
  int32_t record_bytes;
};

inline constexpr size_t params_bytes(int n_heads) {
  return sizeof(TensorHeader) + sizeof(HeadParams) * (size_t)n_heads;
}

#if defined(__HIPCC__)
__host__ __device__
#endif
inline const HeadParams* head_params(const void* block, int head) {
  return reinterpret_cast<const HeadParams*>(static_cast<const char*>(block) +
                                             sizeof(TensorHeader)) + head;
}

}  // namespace aatc
