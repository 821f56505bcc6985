// Layout of the decode workspace: arrival counters per (sequence, KV head), the split
// partials, the appended token's transformed coefficients (key then value, per (sequence,
// KV head)) and the full-precision segment's partials.  Plain C++ shared by the decode
// kernels and host code.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <algorithm>

#include "params.h"

namespace aatc {

constexpr int kMinSplit = 256;                   // smallest split of either decode kernel

struct alignas(16) Partial {   // per (sequence, KV head, split, head-in-group)
  float m;                     // split max of the log2-domain logits
  float l;                     // sum of 2^(z - m)
  float pad_[2];
  float o[kD];                 // sum of 2^(z - m) h^V (transformed domain, storage channels)
};

// Arrival counters sit 256 bytes apart: the device-scope atomics on one cache line
// serialize, and every split of every (sequence, KV head) arrives at nearly once.
constexpr int kCtrStride = 64;

// Fused append, per (sequence, KV head): r_c of the key then the value token (2 x 128),
// then each token's fixed-point error bound eh (0 when exact), padded to 16 bytes.
constexpr int kAppStride = 2 * kD + 4;

struct WsLayout {
  size_t counters, partials, append_r, seg, total;
};

#if defined(__HIPCC__)
__host__ __device__
#endif
inline size_t round256(size_t x) { return (x + 255) / 256 * 256; }

// counter_rows > rows reserves the counters of that many rows, so that the counters keep
// one place whatever the shape of the call (the static workspace of the no-allocation entry
// point: counters left at zero by one call are where the next call looks for them).
inline WsLayout ws_layout(int batch, int n_q_heads, int n_kv_heads, int64_t cap,
                          int counter_rows = 0) {
  const size_t rows = (size_t)batch * n_kv_heads;
  const size_t crows = std::max(rows, (size_t)std::max(counter_rows, 0));
  const size_t n_splits = (size_t)((cap + kMinSplit - 1) / kMinSplit);
  WsLayout w;
  w.counters = 0;
  w.partials = round256(crows * kCtrStride * sizeof(unsigned));
  w.append_r = round256(w.partials + (size_t)batch * n_q_heads * n_splits * sizeof(Partial));
  // the full-precision segment's partial per (sequence, query head)
  w.seg = round256(w.append_r + rows * kAppStride * sizeof(float));
  w.total = w.seg + (size_t)batch * n_q_heads * sizeof(Partial);
  return w;
}

}  // namespace aatc
