// Device parameter block of one tensor under head-group transforms: a header followed by
// one GroupParams per group.  A group is gkv consecutive KV heads whose vectors are
// concatenated into d = 128 gkv elements (Sec. 5.1, the remark on head groups); it has one
// transform, one allocation and one token scale (Sec. 5.2).  Built on the host by
// aatc_group_params_pack, read by the group kernels.  Shared between host and device code.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "params.h"

namespace aatc {

constexpr int kGMax = 512;                   // widest group (four KV heads)
constexpr int kGMaxRecord = 512;             // largest record the group decode stages (bytes)
constexpr int kGMaxHeads = 32;               // query heads per group the decode handles
constexpr uint32_t kGroupMagic = 0x47544141u;   // "AATG"

struct alignas(256) GroupParams {
  int32_t Tqt[kGMax * kGMax];   // [c][j] at c d + j: T_jc 2^22 (integers, |Tq| <= 2^22)
  float T[kGMax * kGMax];       // [j][c] at j d + c: the stored transform
  float inv_s[kGMax];           // fp32 1/s_c (0 for dropped channels)
  float s[kGMax];               // s_c as fp32 (the exact value of the fp16 scale)
  uint16_t s16[kGMax];          // s_c fp16 bits
  uint16_t bit_off[kGMax];      // first record bit of storage channel c
  uint8_t bits[kGMax];          // width of storage channel c (non-increasing)
  int32_t d;                    // 128 gkv
  int32_t gkv;
  int32_t budget;
  int32_t record_bytes;
  int32_t d_active;             // stored channels: 0 .. d_active - 1
  int32_t quantizer;            // aatc_quantizer
  int32_t max_bits;
  int32_t pad_;
};
static_assert(offsetof(GroupParams, T) % 16 == 0, "T alignment");
static_assert(offsetof(GroupParams, inv_s) % 16 == 0, "inv_s alignment");

struct alignas(256) GroupHeader {
  uint32_t magic;
  int32_t n_groups;
  int32_t d;
  int32_t record_bytes;
};

inline constexpr size_t group_params_bytes(int n_groups) {
  return sizeof(GroupHeader) + sizeof(GroupParams) * (size_t)n_groups;
}

#if defined(__HIPCC__)
__host__ __device__
#endif
inline const GroupParams* group_params(const void* block, int g) {
  return reinterpret_cast<const GroupParams*>(static_cast<const char*>(block) +
                                              sizeof(GroupHeader)) + g;
}

// Decode workspace under head groups, per call: the query weights W [batch][n_groups]
// [heads][d], the midrise constants [batch][n_groups][heads], the split partials
// [batch][n_groups][n_splits][heads][kGPH + d] (m, l, unused to a 128-byte header, o~[d]:
// every o~ row starts on a 128-byte line), then for the
// matrix-core split the weights as fp16 operands [batch][n_groups][d / 32][hi, lo][64 lanes]
// [8] (16 head slots) and their per-head power-of-two exponents [batch][n_groups][16], then
// the merged transformed-domain outputs o~ [batch][n_groups * heads][d].
constexpr int kGSplit = 256;                 // tokens per decode split
constexpr int kGPH = 32;                     // header floats of a split partial row

struct GroupWs {
  size_t w, c, partials, wop, wexp, ot, total;
  int n_splits;
};

inline GroupWs group_ws_layout(int batch, int n_groups, int heads, int d, int64_t cap) {
  auto r256 = [](size_t x) { return (x + 255) / 256 * 256; };
  GroupWs l;
  l.n_splits = (int)((cap + kGSplit - 1) / kGSplit);
  const size_t rows = (size_t)batch * n_groups * heads;
  const size_t gsets = (size_t)batch * n_groups;
  l.w = 0;
  l.c = r256(rows * d * sizeof(float));
  l.partials = r256(l.c + rows * sizeof(float));
  l.wop = r256(l.partials + rows * (size_t)l.n_splits * (d + kGPH) * sizeof(float));
  l.wexp = r256(l.wop + gsets * (size_t)(d / 32) * 2 * 64 * 16);
  l.ot = r256(l.wexp + gsets * 16 * sizeof(int32_t));
  l.total = l.ot + rows * d * sizeof(float);
  return l;
}

}  // namespace aatc
