// AATC encode on gfx950: transform, per-token scale, quantize, pack (Algorithm 1,
// inference part; Sec. 5.2).
//
// The transform of a token is h_c = fl32(sum_j x_j T_jc): the exact product of the token
// with the stored transform (entries multiples of 2^-22), rounded once.  Three kernels
// produce it bit for bit:
//   - encode_mfma_kernel (bulk, 16-byte aligned token rows): the integer product of the
//     token in 22-bit fixed point with the integer transform on the matrix cores, which is
//     the exact h whenever the token's fixed-point form is exact (every element above
//     about 2^-14 of the token's largest, for bf16 input); other tokens are certified from
//     a bound on the fixed-point error, and the few it cannot certify are redone exactly;
//   - encode_exact_kernel (any layout): every token by the exact one-wave routine;
//   - encode_token_kernel (a few tokens): the same, one wave per (token, KV head).
#include <algorithm>

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "encode_core.h"
#include "launch.h"
#include "params.h"

namespace aatc {
namespace {

constexpr int kEncThreads = 256;                 // four waves
constexpr int kRecWords = kMaxBudget / 32;       // words of the largest record
// LDS record rows are one word longer than the largest record, so that one word of many
// rows (the tile transpose, the per-token bit fields) falls into different banks.
constexpr int kRecStride = kRecWords + 1;
constexpr int kSmallBatch = 16;                  // appends up to this many tokens: per-token kernel
constexpr uint16_t kRedo = 0xFFFFu;              // scale mark of a token left to the exact routine
                                                 // (an fp16 NaN: no token scale has it)

// This lane's two elements (lane, lane + 64) of a token.
__device__ inline void load_token_pair(const void* xrow, int dtype, float (&xl)[2]) {
  const int lane = threadIdx.x & 63;
  xl[0] = load_elem(xrow, dtype, lane);
  xl[1] = load_elem(xrow, dtype, lane + 64);
}

// Writes the records [lo, hi) of a 64-token tile from LDS rows (`rec`, rows of kRecStride
// words) into the cache in `layout`, and clears every LDS word it reads.  Tile bits of
// tokens outside [lo, hi) keep their value in memory.
__device__ inline void write_tile(uint32_t (*rec)[kRecStride], int lo, int hi, int rwords,
                                  int layout, uint8_t* codes, int64_t head, int64_t cap,
                                  int64_t tile, int nthreads) {
  const int tid = threadIdx.x;
  if (layout == AATC_LAYOUT_RECORDS) {
    uint32_t* out = reinterpret_cast<uint32_t*>(codes) + (head * cap + tile * kTile) * rwords;
    for (int i = lo * rwords + tid; i < hi * rwords; i += nthreads) {
      out[i] = rec[i / rwords][i % rwords];
      rec[i / rwords][i % rwords] = 0u;
    }
  } else {
    // Bit-transposed tile: word 2 v + W holds record bit v of the tile's tokens
    // t = 16 d + 4 g + i with d / 2 = W, at bit 8 i + 2 g + d % 2.
    uint32_t* out = reinterpret_cast<uint32_t*>(codes) + (head * (cap / kTile) + tile) * (16 * rwords * 4);
    for (int wi = tid; wi < 64 * rwords; wi += nthreads) {
      const int v = wi >> 1, W = wi & 1;
      uint32_t mask = 0, nw = 0;
      for (int p = 0; p < 32; ++p) {
        const int t = 16 * (2 * W + (p & 1)) + 4 * ((p >> 1) & 3) + (p >> 3);
        if (t >= lo && t < hi) {
          mask |= 1u << p;
          nw |= ((rec[t][v >> 5] >> (v & 31)) & 1u) << p;
        }
      }
      if (!mask) continue;
      const uint32_t old = (mask == 0xffffffffu) ? 0u : out[wi];
      out[wi] = (old & ~mask) | nw;
    }
    __syncthreads();                             // every bit read before the rows clear
    for (int i = tid; i < kTile * rwords; i += nthreads) rec[i / rwords][i % rwords] = 0u;
  }
}

// One 64-token tile by a workgroup of kEncThreads threads: wave w encodes the tile's
// tokens w, w + 4, ... with the exact one-wave routine into the LDS rows `rec` (zero on
// entry, zero again on return), which are then written out.
__device__ void exact_tile(const HeadParams* hp, const void* __restrict__ x, int dtype,
                           int64_t n_tok, int64_t x_stride, int layout,
                           uint8_t* __restrict__ codes, uint16_t* __restrict__ alpha,
                           int64_t cap, int64_t pos, int64_t tile, int head,
                           uint32_t (*rec)[kRecStride]) {
  const int rwords = hp->record_bytes / 4;
  const int64_t tile_base = tile * kTile;
  const int64_t t_begin = max(tile_base, pos);
  const int64_t t_end = min(tile_base + kTile, pos + n_tok);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  for (int64_t t = t_begin + wave; t < t_end; t += kEncThreads / 64) {
    const void* xrow = static_cast<const char*>(x) +
                       ((t - pos) * x_stride + (int64_t)head * kD) * (dtype == AATC_BF16 ? 2 : 4);
    float xl[2], r[2];
    load_token_pair(xrow, dtype, xl);
    exact_r_wave<true>(hp, xl, xrow, dtype, r);
    const __half a16 = wave_quantize_into(hp, r, rec[t - tile_base]);
    if (lane == 0) alpha[(int64_t)head * cap + t] = __half_as_ushort(a16);
  }
  __syncthreads();
  write_tile(rec, (int)(t_begin - tile_base), (int)(t_end - tile_base), rwords, layout, codes,
             head, cap, tile, kEncThreads);
  __syncthreads();                               // (the cleared rows before their next use)
}

// Any layout, any token count: one workgroup per (64-token tile, KV head).
__global__ __launch_bounds__(kEncThreads) void encode_exact_kernel(
    const void* __restrict__ params, const void* __restrict__ x, int dtype, int64_t n_tok,
    int64_t x_stride, int layout, uint8_t* __restrict__ codes, uint16_t* __restrict__ alpha,
    int64_t cap, int64_t pos) {
  __shared__ uint32_t rec[kTile][kRecStride];
  const int head = blockIdx.y;
  for (int i = threadIdx.x; i < kTile * kRecStride; i += kEncThreads) (&rec[0][0])[i] = 0u;
  __syncthreads();
  exact_tile(head_params(params, head), x, dtype, n_tok, x_stride, layout, codes, alpha, cap,
             pos, pos / kTile + blockIdx.x, head, rec);
}

// ---------------------------------------------------------------------------------------
// The bulk encode on the matrix cores.
//
// Per token, S is chosen with max |x_j| 2^S in [2^21, 2^22) and X_j is x_j 2^S rounded to
// an integer; the integer transform is Tq = T 2^22 (|Tq| <= 2^22).  Both split into int8
// limbs, X = 2^16 X2 + 2^8 X1 + X0 and Tq = 2^16 T2 + 2^8 T1 + T0 (X0, X1, T0, T1 in
// [-128, 127], |X2|, |T2| <= 64), and the nine limb products go to
// v_mfma_i32_16x16x64_i8 in five int32 sums by weight, S_k = sum over a + b = k of
// sum_j X_a T_b (each below 2^23, exact).  H = sum_k 2^(8k) S_k = sum_j X_j Tq_jc is below
// 2^51 and is formed exactly in fp64.
//   - If every X_j equals x_j 2^S (the token is exact in fixed point), H 2^-(S+22) is the
//     exact h.  With k = S + 22 in [0, 100] every intermediate below is a normal fp32
//     number (or zero), so the power of two leaves the roundings: u_c = fl32(fl32(H) / s_c)
//     is r_c 2^k, alpha is the fp16 rounding of max |u| 2^-k and the quantizer input is
//     fl32(u_c (2^-k / alpha)), bit for bit the canonical sequence.
//   - Otherwise |H - H_exact| <= E 2^22 with E = sum_j |x_j 2^S - X_j|.  The token's scale
//     and codes are certified against that bound: alpha if the fp16 rounding of the largest
//     |r| cannot change within it, each code if its fp32 quantizer input lies farther than
//     the bound (plus the fp32 roundings of both evaluations) from a rounding boundary.
// Tokens that fail, and tokens whose k is out of range, get the scale mark kRedo;
// encode_fixup_kernel, launched next on the stream, encodes them exactly.
//
// A workgroup of twelve waves shares the limb tables of one KV head's transform (48 KiB of
// LDS, built once).  After that each wave works alone, with no workgroup barrier, on
// 32-token units (half a 64-token tile): two groups of 16 tokens against all 128 channels,
// codes OR-ed into the wave's own LDS record rows, then the unit's records, or its half of
// the tile's bit-transposed words, written out.  Lane 16 kg + n holds token n's elements
// j = 64 kc + 16 kg .. + 15 (kc = 0, 1): the B operand columns; the A operand lane
// (channel 16 ct + n) reads the same j of row c of the limb tables.  The products leave
// lane 16 kg + n with channels 16 ct + 4 kg + i, i < 4, of its own token: four consecutive
// codes, one bit field of the record.
// Needs 16-byte aligned token rows (checked by the launcher).
// ---------------------------------------------------------------------------------------
// Limb tables in matrix-core operand order: the 16 bytes lane l of a wave feeds for
// channel tile ct and k half kc sit at ((2 ct + kc) 64 + l) 16, so every operand read is one
// contiguous 1 KiB per wave (no bank conflicts).
constexpr int kTbBytes = 8 * 2 * 64 * 16;        // one limb of the 128 x 128 transform
constexpr int kMW = 12;                           // waves per matrix-core workgroup
constexpr int kMThreads = 64 * kMW;
constexpr int kUnit = 32;                         // tokens per wave work unit
constexpr int kNarrowWords = kD * 8 / 32;         // largest record of codes up to 8 bits
constexpr int kStage = kNarrowWords + 1;          // LDS record row stride (one word of padding)
// X + kXBias (2^15 + 2^7) carries the limbs as bytes: X0 = byte 0 - 128, X1 = byte 1 - 128,
// X2 = byte 2 (signed).
constexpr int kXBias = 32896;

typedef int ev4i __attribute__((ext_vector_type(4)));
typedef unsigned short eu2 __attribute__((ext_vector_type(2)));

// Maximum / sum over lanes l, l ^ 16, l ^ 32 and l ^ 48 (the gfx950 row swaps): the four
// lanes of one token.
__device__ inline float enc_cross_row_max(float v) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float enc_cross_row_sum(float v) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ inline uint32_t enc_cross_row_umax(uint32_t v) {
  auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = max((uint32_t)r[0], (uint32_t)r[1]);
  r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return max((uint32_t)r[0], (uint32_t)r[1]);
}
__device__ inline uint32_t enc_cross_row_umin(uint32_t v) {
  auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = min((uint32_t)r[0], (uint32_t)r[1]);
  r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return min((uint32_t)r[0], (uint32_t)r[1]);
}

// Orders one wave's LDS accesses across its lanes (a wave's LDS instructions execute in
// issue order; this keeps the compiler from moving accesses across the point).
__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// One stage of a 32 x 32 bit-matrix transpose over the 32 lanes of each half wave (lane i
// holds row i): blocks of S bits are exchanged with lane i ^ S.
template <int S, uint32_t M>
__device__ inline uint32_t bit_transpose_stage(uint32_t x, int lane) {
  const uint32_t y = (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, 0x1f | (S << 10));
  return (lane & S) ? ((x & ~M) | ((y >> S) & M)) : ((x & M) | ((y & M) << S));
}

// This lane's 32 elements of a token: the 16 at j = 64 kc + 16 kg .. + 15 for kc = 0, 1.
template <bool BF16> struct Chunk;
template <> struct Chunk<true> {
  uint4 w[2][2];                                   // [kc][half]: bf16 pairs, low half first
  __device__ void load(const void* x, int64_t base, int kg) {
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      const uint4* p = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(x) + base +
                                                      64 * kc + 16 * kg);
      w[kc][0] = p[0];
      w[kc][1] = p[1];
    }
  }
  __device__ void clear() {
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) w[kc][0] = w[kc][1] = make_uint4(0u, 0u, 0u, 0u);
  }
  __device__ uint32_t word(int kc, int i) const {  // elements 2 i, 2 i + 1
    const uint4& u = w[kc][i >> 2];
    const int q = i & 3;
    return q == 0 ? u.x : q == 1 ? u.y : q == 2 ? u.z : u.w;
  }
  __device__ float elem(int kc, int e) const {
    const uint32_t v = word(kc, e >> 1);
    return __uint_as_float((e & 1) ? (v & 0xffff0000u) : (v << 16));
  }
};
template <> struct Chunk<false> {
  float4 w[2][4];
  __device__ void load(const void* x, int64_t base, int kg) {
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(x) + base +
                                                        64 * kc + 16 * kg);
#pragma unroll
      for (int q = 0; q < 4; ++q) w[kc][q] = p[q];
    }
  }
  __device__ void clear() {
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int q = 0; q < 4; ++q) w[kc][q] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  __device__ float elem(int kc, int e) const {
    const float4& f = w[kc][e >> 2];
    const int q = e & 3;
    return q == 0 ? f.x : q == 1 ? f.y : q == 2 ? f.z : f.w;
  }
};

// The token's largest |x_j| (over its four lanes), and whether its fixed-point form may be
// inexact.  bf16: X_j = x_j 2^S exactly whenever x_j's exponent is at least the largest
// one's minus 14 (8 significant bits, 22 bits of fixed point), so only tokens with a
// smaller (or zero, or subnormal) element are flagged.  fp32: always flagged.
template <bool BF16>
__device__ inline float chunk_stats(const Chunk<BF16>& c, bool& maybe_inexact) {
  if constexpr (BF16) {
    eu2 mx = {0, 0}, mn = {0xffff, 0xffff};
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const eu2 v = __builtin_bit_cast(eu2, c.word(kc, i) & 0x7fff7fffu);
        mx = __builtin_elementwise_max(mx, v);
        mn = __builtin_elementwise_min(mn, v);
      }
    const uint32_t hi = enc_cross_row_umax(max((uint32_t)mx.x, (uint32_t)mx.y));
    const uint32_t lo = enc_cross_row_umin(min((uint32_t)mn.x, (uint32_t)mn.y));
    maybe_inexact = hi != 0u && (lo >> 7) + 14u < (hi >> 7);
    return __uint_as_float(hi << 16);
  } else {
    float m = 0.f;
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int e = 0; e < 16; ++e) m = fmaxf(m, fabsf(c.elem(kc, e)));
    maybe_inexact = true;
    return enc_cross_row_max(m);
  }
}

// The scale of one token for chunk_y: 2^S.
struct XScale {
  float f;
  __device__ explicit XScale(int S) : f(ldexpf(1.f, S)) {}
};

// y = X + kXBias for elements 4 q .. 4 q + 3 of k half kc, X = x 2^S rounded to an integer
// (x 2^S + kXBias rounded to fp32, then toward zero: any rounding would do, since E below is
// taken against these very integers).  Elements with x 2^S an integer give exactly that
// integer.  -22 <= S <= 78.
template <bool BF16>
__device__ inline void chunk_y(const Chunk<BF16>& c, int kc, int q, const XScale& sc,
                               uint32_t (&y)[4]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) y[e] = (uint32_t)(int)fmaf(c.elem(kc, 4 * q + e), sc.f, (float)kXBias);
}

// The int8 limbs of X as B operands (byte e of word q: element 4 q + e): X0 = byte 0 of y
// - 128, X1 = byte 1 of y - 128, X2 = byte 2 of y (signed), for y = X + kXBias.
template <bool BF16>
__device__ inline void chunk_limbs(const Chunk<BF16>& c, const XScale& sc, ev4i (&A)[3][2]) {
#pragma unroll
  for (int kc = 0; kc < 2; ++kc)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t y[4];
      chunk_y<BF16>(c, kc, q, sc, y);
      // v_perm_b32(a, b, sel): byte k of the result is byte sel_k of {a: 4..7, b: 0..3}
      const uint32_t p01 = __builtin_amdgcn_perm(y[1], y[0], 0x05010400u);
      const uint32_t p23 = __builtin_amdgcn_perm(y[3], y[2], 0x05010400u);
      A[0][kc][q] = (int)(__builtin_amdgcn_perm(p23, p01, 0x05040100u) ^ 0x80808080u);
      A[1][kc][q] = (int)(__builtin_amdgcn_perm(p23, p01, 0x07060302u) ^ 0x80808080u);
      A[2][kc][q] = (int)(__builtin_amdgcn_perm(y[1], y[0], 0x0c0c0602u) |
                          __builtin_amdgcn_perm(y[3], y[2], 0x06020c0cu));
    }
}

// This lane's part of E = sum_j |x_j 2^S - X_j| for the X_j of chunk_limbs (each term
// exact: x_j 2^S - X_j has at most 8 (bf16) or 24 (fp32) significant bits; a product
// below the fp32 range rounds by under 2^-150, which the caller's slack covers).
template <bool BF16>
__device__ inline float chunk_err(const Chunk<BF16>& c, const XScale& sc) {
  float E = 0.f;
#pragma unroll
  for (int kc = 0; kc < 2; ++kc)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t y[4];
      chunk_y<BF16>(c, kc, q, sc, y);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        E += fabsf(fmaf(c.elem(kc, 4 * q + e), sc.f, (float)(kXBias - (int)y[e])));
    }
  return E;
}

// A value the compiler cannot see through (keeps work that depends on it inside its branch).
__device__ inline float opaque(float v) {
  asm volatile("" : "+v"(v));
  return v;
}

// The int8 limb bytes of four integers |v| <= 2^22 (the transform): limb 0 = byte 0 of v,
// limb 1 = byte 1 of v + 128, limb 2 = byte 2 of v + 32896 (the balanced digits:
// v = 65536 l2 + 256 l1 + l0 with l0, l1 in [-128, 127]).
__device__ inline void limb_bytes4(const int (&v)[4], uint32_t (&out)[3]) {
  uint32_t y1[4], y2[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    y1[e] = (uint32_t)(v[e] + 128);
    y2[e] = (uint32_t)(v[e] + 32896);
  }
  out[0] = __builtin_amdgcn_perm((uint32_t)v[1], (uint32_t)v[0], 0x0c0c0400u) |
           __builtin_amdgcn_perm((uint32_t)v[3], (uint32_t)v[2], 0x04000c0cu);
  out[1] = __builtin_amdgcn_perm(y1[1], y1[0], 0x0c0c0501u) |
           __builtin_amdgcn_perm(y1[3], y1[2], 0x05010c0cu);
  out[2] = __builtin_amdgcn_perm(y2[1], y2[0], 0x0c0c0602u) |
           __builtin_amdgcn_perm(y2[3], y2[2], 0x06020c0cu);
}

template <bool BF16>
__global__ __launch_bounds__(kMThreads) void encode_mfma_kernel(
    const void* __restrict__ params, const void* __restrict__ x, int64_t n_tok,
    int64_t x_stride, int layout, uint8_t* __restrict__ codes, uint16_t* __restrict__ alpha,
    int64_t cap, int64_t pos) {
  __shared__ __align__(16) int8_t tb[3][kTbBytes];         // [limb][ct][kc][lane][16]
  __shared__ uint32_t stage[kMW][kUnit][kStage];           // each wave's record rows
  // Channel tables, read by the lanes that hold channels 16 ct + 4 kg + i.
  __shared__ __align__(16) float tab_is[kD];               // 1 / s_c
  __shared__ __align__(16) float tab_p2[kD];               // 2^(b_c - 1) (1 for b_c = 0)
  __shared__ __align__(16) float tab_hi[kD];               // 2^(b_c - 1) - 1: largest code
  __shared__ __align__(16) float tab_k[kD];                // 2^(b_c - 1) / s_c (1 + 2^-20)
  __shared__ __align__(16) uint32_t tab_sh[kD];            // bit of c in its group's field
  __shared__ uint32_t tab_bias[kD / 4];                    // sum of 2^(b - 1) << sh
  __shared__ uint32_t tab_msb[kD / 4];                     // sum of 1 << (sh + b - 1)
  __shared__ uint16_t tab_o[kD];                           // first record bits

  const int head = blockIdx.y;
  const HeadParams* hp = head_params(params, head);
  const int tid = threadIdx.x, lane = tid & 63, n = lane & 15, kg = lane >> 4;
  // (the wave index as a scalar: the unit and tile indices and addresses derived from it
  // stay in scalar registers)
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t first = pos / kTile, last = (pos + n_tok - 1) / kTile;
  const int64_t n_units = 2 * (last - first + 1);
  if (hp->max_bits > 8) {
    // Codes wider than 8 bits need not fit a four-channel field: every token goes to the
    // exact routine of encode_fixup_kernel (uniform over the grid).
    for (int64_t i = (int64_t)blockIdx.x * kMThreads + tid; i < n_tok;
         i += (int64_t)gridDim.x * kMThreads)
      alpha[(int64_t)head * cap + pos + i] = kRedo;
    return;
  }
  const bool midrise = hp->quantizer == AATC_QUANT_MIDRISE;
  const int rwords = hp->record_bytes / 4;
  // i / rwords = (i rmagic) >> 16 for i < 1024 and rwords <= 32
  const uint32_t rmagic = rwords ? (65536u + rwords - 1) / rwords : 0u;

  // Limb tables of the transposed integer transform: operand slot u = (2 ct + kc) 64 + l
  // (l = 16 kg + n) holds Tq^T[16 ct + n][64 kc + 16 kg .. + 15].
  for (int u = tid; u < 1024; u += kMThreads) {
    const int l = u & 63, ct = u >> 7, kc = (u >> 6) & 1;
    const int4* src = reinterpret_cast<const int4*>(hp->Tqt + (16 * ct + (l & 15)) * kD +
                                                    64 * kc + 16 * (l >> 4));
    uint32_t w[3][4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int4 t4 = src[q];
      const int v[4] = {t4.x, t4.y, t4.z, t4.w};
      uint32_t lb[3];
      limb_bytes4(v, lb);
#pragma unroll
      for (int li = 0; li < 3; ++li) w[li][q] = lb[li];
    }
#pragma unroll
    for (int li = 0; li < 3; ++li)
      *reinterpret_cast<uint4*>(&tb[li][16 * u]) = make_uint4(w[li][0], w[li][1], w[li][2], w[li][3]);
  }
  if (tid < kD) {
    const int b = hp->bits[tid];
    tab_is[tid] = hp->inv_s[tid];
    tab_k[tid] = ldexpf(hp->inv_s[tid], max(b, 1) - 1) * (1.f + 0x1p-20f);
    tab_p2[tid] = ldexpf(1.f, max(b, 1) - 1);
    tab_hi[tid] = ldexpf(1.f, max(b, 1) - 1) - 1.f;
    int sh = 0;
    for (int c = tid & ~3; c < tid; ++c) sh += hp->bits[c];
    tab_sh[tid] = (uint32_t)sh;
    tab_o[tid] = hp->bit_off[tid];
  }
  if (tid < kD / 4) {
    uint32_t w = 0u, bias = 0u, msb = 0u;
    for (int i = 0; i < 4; ++i) {
      const int b = hp->bits[4 * tid + i];
      if (b > 0) {
        bias += (1u << (b - 1)) << w;
        msb |= 1u << (w + b - 1);
      }
      w += b;
    }
    tab_bias[tid] = bias;
    tab_msb[tid] = msb;
  }
  for (int i = tid; i < kMW * kUnit * kStage; i += kMThreads) (&stage[0][0][0])[i] = 0u;
  __syncthreads();                                 // (the last workgroup barrier)

  const int64_t ustep = (int64_t)gridDim.x * kMW;
  int64_t u = (int64_t)blockIdx.x * kMW + wave;
  if (u >= n_units) return;
  uint32_t (*rows)[kStage] = stage[wave];
  // Where this lane's eight fields go in a record row: byte offset of the first word (bits
  // 0-7) and bit within it (bits 8-12); a field spills into the next word at most (the
  // row's padding word takes a zero OR at the end).
  uint32_t place[8];
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) {
    const int off = tab_o[16 * ct + 4 * kg];
    place[ct] = (uint32_t)(4 * (off >> 5)) | ((uint32_t)(off & 31) << 8);
  }
  // Token t = 64 first + 32 v + 16 g + n of unit v (32 v + 16 g + n past the first tile);
  // the loads run one group ahead.
  const int64_t t0 = first * kTile + n;
  Chunk<BF16> nxt;
  auto fetch = [&](int64_t v, int g) {
    const int64_t t = t0 + 32 * v + 16 * g;
    if (v < n_units && t >= pos && t < pos + n_tok)
      nxt.load(x, (t - pos) * x_stride + (int64_t)head * kD, kg);
    else
      nxt.clear();
  };
  fetch(u, 0);
  for (; u < n_units; u += ustep) {
    const int64_t tile = first + (u >> 1);
    const int W = (int)(u & 1);
    const int64_t ubase = tile * kTile + 32 * W;
    const int lo = (int)max<int64_t>(pos - ubase, 0);
    const int hi = (int)min<int64_t>(pos + n_tok - ubase, kUnit);
#pragma unroll 1
    for (int g = 0; g < 2; ++g) {
      const Chunk<BF16> cur = nxt;
      if (g == 0) fetch(u, 1);
      else fetch(u + ustep, 0);
      const int tu = 16 * g + n;
      const bool valid = tu >= lo && tu < hi;
      // (1) The token's fixed-point shift and exactness flag.
      bool maybe = false;
      const int S = token_shift(chunk_stats<BF16>(cur, maybe));
      const int k = S + kTFrac;
      const bool k_ok = k >= 0 && k <= 100;
      const XScale sc(min(max(S, -kTFrac), 100 - kTFrac));
      const bool cert = __builtin_amdgcn_ballot_w64(maybe) != 0ull;
      // (2) The limbs of X as B operands, and in waves with a flagged token the fixed-point
      //     error sum E of each token (over its four lanes).
      ev4i A[3][2];
      chunk_limbs<BF16>(cur, sc, A);
      float Et = 0.f;
      if (cert) Et = opaque(enc_cross_row_sum(chunk_err<BF16>(cur, sc)));
      // (3) Channel tile by channel tile: the five limb-product sums (18 products), H exactly,
      //     then u_c = fl32(fl32(H) / s_c) for channels 16 ct + 4 kg + i of this token.  The
      //     operands of the next k half are read while the products of this one run, and
      //     the sums of tile ct - 1 are turned into u while those of tile ct accumulate.
      float uv[8][4], am = 0.f;
      // (an opaque zero in the operand addresses: the tables are the same for every group,
      // and loads hoisted out of the loop would hold 192 registers)
      int tb0;
      asm volatile("s_mov_b32 %0, 0" : "=s"(tb0));
      auto load_b = [&](int q, ev4i (&bq)[3]) {
        const int o = 16 * ((2 * (q >> 1) + (q & 1)) * 64 + lane) + tb0;
#pragma unroll
        for (int l = 0; l < 3; ++l) bq[l] = *reinterpret_cast<const ev4i*>(&tb[l][o]);
      };
      auto products = [&](const ev4i (&bq)[3], int kc, ev4i (&sa)[5]) {
        sa[4] = __builtin_amdgcn_mfma_i32_16x16x64_i8(bq[2], A[2][kc], sa[4], 0, 0, 0);
        sa[3] = __builtin_amdgcn_mfma_i32_16x16x64_i8(bq[2], A[1][kc], sa[3], 0, 0, 0);
        sa[2] = __builtin_amdgcn_mfma_i32_16x16x64_i8(bq[2], A[0][kc], sa[2], 0, 0, 0);
        sa[1] = __builtin_amdgcn_mfma_i32_16x16x64_i8(bq[1], A[0][kc], sa[1], 0, 0, 0);
        sa[0] = __builtin_amdgcn_mfma_i32_16x16x64_i8(bq[0], A[0][kc], sa[0], 0, 0, 0);
        sa[3] = __builtin_amdgcn_mfma_i32_16x16x64_i8(bq[1], A[2][kc], sa[3], 0, 0, 0);
        sa[2] = __builtin_amdgcn_mfma_i32_16x16x64_i8(bq[1], A[1][kc], sa[2], 0, 0, 0);
        sa[1] = __builtin_amdgcn_mfma_i32_16x16x64_i8(bq[0], A[1][kc], sa[1], 0, 0, 0);
        sa[2] = __builtin_amdgcn_mfma_i32_16x16x64_i8(bq[0], A[2][kc], sa[2], 0, 0, 0);
      };
      auto to_u = [&](const ev4i (&sa)[5], int ct) {
        const float4 is4 = *reinterpret_cast<const float4*>(&tab_is[16 * ct + 4 * kg]);
        const float isv[4] = {is4.x, is4.y, is4.z, is4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // H = 2^24 (2^8 S4 + S3) + 2^16 S2 + (2^8 S1 + S0): exact in fp64 (< 2^51)
          const int hi8 = sa[4][i] * 256 + sa[3][i];
          const int lo8 = sa[1][i] * 256 + sa[0][i];
          const double H = fma(fma((double)hi8, 256.0, (double)sa[2][i]), 65536.0, (double)lo8);
          uv[ct][i] = (float)H * isv[i];
          am = fmaxf(am, fabsf(uv[ct][i]));          // (u = 0 on dropped channels)
        }
      };
      {
        ev4i bq[2][3], sa[2][5];
        load_b(0, bq[0]);
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int ct = q >> 1, kc = q & 1;
          if (q + 1 < 16) load_b(q + 1, bq[(q + 1) & 1]);
          __builtin_amdgcn_sched_barrier(0);            // (the reads stay ahead of the products)
          if (kc == 0) {
#pragma unroll
            for (int kk = 0; kk < 5; ++kk) sa[ct & 1][kk] = (ev4i){0, 0, 0, 0};
          }
          products(bq[q & 1], kc, sa[ct & 1]);
          if (kc == 1 && ct > 0) to_u(sa[(ct - 1) & 1], ct - 1);
        }
        to_u(sa[1], 7);
      }
      // (4) The token's scale (its 128 channels: 4 lanes), then its codes: channels
      //     16 ct + 4 kg .. + 3 are consecutive in the record, one bit field of <= 32 bits.
      const float amax_r = ldexpf(enc_cross_row_max(am), -k);
      const __half a16 = token_alpha(amax_r);
      const float inv_ak = ldexpf(inverse_alpha(a16), -k);
      bool bad = !k_ok;
      float ea = 0.f;
      if (cert) {
        // |H - H_exact| <= eH (with the (1 + 2^-20) of the fp32 products below); the range of
        // the exact max |r| widened by the fp32 roundings must round to one fp16 scale.
        // Only tokens with E > 0 need the certificate.
        const float eH = opaque((Et + 0x1p-143f) * (1.f + 0x1p-16f) * 0x1p22f * (1.f + 0x1p-20f));
        float alo = 0.f, ahi = 0.f;
#pragma unroll
        for (int ct = 0; ct < 8; ++ct) {
          const float4 is4 = *reinterpret_cast<const float4*>(&tab_is[16 * ct + 4 * kg]);
          const float isv[4] = {is4.x, is4.y, is4.z, is4.w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            ahi = fmaxf(ahi, fmaf(eH, isv[i], fabsf(uv[ct][i])));
            alo = fmaxf(alo, fmaf(-eH, isv[i], fabsf(uv[ct][i])));
          }
        }
        const float lo_r = ldexpf(enc_cross_row_max(alo), -k) - 0x1p-21f * amax_r;
        const float hi_r = ldexpf(enc_cross_row_max(ahi), -k) + 0x1p-21f * amax_r + 0x1p-140f;
        const bool a_unc = __half_as_ushort(token_alpha(fmaxf(lo_r, 0.f))) !=
                           __half_as_ushort(token_alpha(hi_r));
        ea = Et > 0.f ? eH * inv_ak : -1.f;
        bad |= Et > 0.f && a_unc;
      }
      uint32_t field[8];
      auto codes_of = [&](auto certify, auto mid_rise) {
        constexpr bool CERT = decltype(certify)::value;
        constexpr bool MR = decltype(mid_rise)::value;
#pragma unroll
        for (int ct = 0; ct < 8; ++ct) {
          const int c0 = 16 * ct + 4 * kg;
          const float4 p4 = *reinterpret_cast<const float4*>(&tab_p2[c0]);
          const float4 h4 = *reinterpret_cast<const float4*>(&tab_hi[c0]);
          const uint4 s4 = *reinterpret_cast<const uint4*>(&tab_sh[c0]);
          const float p2[4] = {p4.x, p4.y, p4.z, p4.w}, hv[4] = {h4.x, h4.y, h4.z, h4.w};
          const uint32_t sh[4] = {s4.x, s4.y, s4.z, s4.w};
          float4 k4;
          if constexpr (CERT) k4 = *reinterpret_cast<const float4*>(&tab_k[c0]);
          // Offset binary (code + 2^(b-1)) summed into the field, the sign bits flipped at
          // the end: b-bit two's complement codes.
          uint32_t f = tab_bias[c0 >> 2];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            // The canonical quantizer: xq = fl32(r / alpha) 2^(b-1) (the power of two is
            // exact), code = floor(xq + 1/2) (midtread) or floor(xq) (midrise) clamped to
            // [-2^(b-1), 2^(b-1) - 1].  Clamping xq first (the bounds are integers) and then
            // rounding gives the same code; for midtread the rounding half up is one
            // v_cvt_rpi_i32_f32 (checked on the hardware against floor(xq) + (frac >= 1/2):
            // boundary values within 64 ulps of k and k + 1/2 for |k| <= 130, 2^24 values in
            // all).  Dropped channels have u = 0 and contribute code 0.
            const float xq = (uv[ct][i] * inv_ak) * p2[i];
            const float xc = __builtin_amdgcn_fmed3f(xq, -p2[i], hv[i]);
            int code;
            if constexpr (MR)
              asm("v_cvt_flr_i32_f32 %0, %1" : "=v"(code) : "v"(xc));
            else
              asm("v_cvt_rpi_i32_f32 %0, %1" : "=v"(code) : "v"(xc));
            f += (uint32_t)code << sh[i];
            if constexpr (CERT) {
              const float kf = i == 0 ? k4.x : i == 1 ? k4.y : i == 2 ? k4.z : k4.w;
              // the bound in x units, plus both evaluations' fp32 roundings and that of
              // xq + 1/2; the distance to the nearest boundary from the fraction
              const float mg = fmaf(kf, ea, fmaf(0x1p-21f, fabsf(xq), 0x1p-22f));
              const float d = fabsf(__builtin_amdgcn_fractf(xq) - 0.5f);
              bad |= MR ? (d >= 0.5f - mg) : (d <= mg);
            }
          }
          field[ct] = f ^ tab_msb[c0 >> 2];
        }
      };
      if (midrise) {
        if (cert) codes_of(std::true_type{}, std::true_type{});
        else codes_of(std::false_type{}, std::true_type{});
      } else {
        if (cert) codes_of(std::true_type{}, std::false_type{});
        else codes_of(std::false_type{}, std::false_type{});
      }
      // A token is redone exactly if any of its four lanes could not certify it.
      const bool redo = enc_cross_row_max(bad ? 1.f : 0.f) > 0.f;
      if (valid && !redo) {
        char* row = reinterpret_cast<char*>(rows[tu]);
#pragma unroll
        for (int ct = 0; ct < 8; ++ct) {
          uint32_t* w0 = reinterpret_cast<uint32_t*>(row + (place[ct] & 0xffu));
          const uint64_t v = (uint64_t)field[ct] << ((place[ct] >> 8) & 31u);
          atomicOr(w0, (uint32_t)v);
          atomicOr(w0 + 1, (uint32_t)(v >> 32));
        }
      }
      if (valid && kg == 0)
        alpha[(int64_t)head * cap + ubase + tu] = redo ? kRedo : __half_as_ushort(a16);
    }
    // (5) The unit out of the wave's rows, each word cleared once read.
    wave_lds_sync();
    if (layout == AATC_LAYOUT_RECORDS) {
      uint32_t* out = reinterpret_cast<uint32_t*>(codes) + ((int64_t)head * cap + ubase) * rwords;
      for (int i = lo * rwords + lane; i < hi * rwords; i += 64) {
        const int q = (int)(((uint32_t)i * rmagic) >> 16), r = i - q * rwords;
        out[i] = rows[q][r];
        rows[q][r] = 0u;
      }
    } else {
      // Record word w of the unit's tokens -> tile words 64 w + 2 b + W.  Lane q (and
      // q + 32, one word further) holds the word of the token at half-tile position q,
      // i.e. token 16 (q % 2) + 4 ((q / 2) % 4) + q / 8 of the unit; a 32 x 32 bit transpose
      // within each half of the wave leaves lane q with bit q over the 32 positions.
      uint32_t* out = reinterpret_cast<uint32_t*>(codes) +
                      ((int64_t)head * (cap / kTile) + tile) * (16 * rwords * 4);
      const int q = lane & 31, hs = lane >> 5;
      const int ptok = 16 * (q & 1) + 4 * ((q >> 1) & 3) + (q >> 3);
      const uint32_t keep = ~(uint32_t)__builtin_amdgcn_ballot_w64(ptok >= lo && ptok < hi);
      for (int w = 0; w < rwords; w += 2) {
        const int ww = w + hs;
        uint32_t xw = 0u;
        if (ww < rwords) {
          xw = rows[ptok][ww];
          rows[ptok][ww] = 0u;
        }
        xw = bit_transpose_stage<16, 0x0000ffffu>(xw, lane);
        xw = bit_transpose_stage<8, 0x00ff00ffu>(xw, lane);
        xw = bit_transpose_stage<4, 0x0f0f0f0fu>(xw, lane);
        xw = bit_transpose_stage<2, 0x33333333u>(xw, lane);
        xw = bit_transpose_stage<1, 0x55555555u>(xw, lane);
        if (ww < rwords) {
          uint32_t* o = out + 64 * ww + 2 * q + W;
          *o = keep ? ((*o & keep) | (xw & ~keep)) : xw;
        }
      }
    }
    wave_lds_sync();                                // (the cleared rows before the next unit)
  }
}

// exact_r_wave (the same sums in the same order, hence the same r) with the transform
// entries for j + 16 .. j + 31 in flight while those for j .. j + 15 are summed: four round
// trips to the parameter block in sequence instead of eight, for more registers.  For the
// kernels that encode a token or a few per wave, where that latency is the time.
template <bool LEAN = false>
__device__ inline void exact_r_wave_pipelined(const HeadParams* hp, const float (&xl)[2],
                                              const void* xrow, int dtype, float (&r)[2]) {
  const int lane = threadIdx.x & 63;
  double s[2] = {0.0, 0.0}, a[2] = {0.0, 0.0};
  const int4* tc[2] = {reinterpret_cast<const int4*>(hp->Tqt + lane * kD),
                       reinterpret_cast<const int4*>(hp->Tqt + (lane + 64) * kD)};
  auto load = [&](int jb, int4 (&tv)[2][4]) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) tv[i][q] = tc[i][jb / 4 + q];
  };
  auto sum = [&](int jb, const int4 (&tv)[2][4]) {
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
  };
  int4 ta[2][4], tb[2][4];
  load(0, ta);
#pragma unroll 1
  for (int jb = 0; jb < kD; jb += 32) {
    load(jb + 16, tb);
    sum(jb, ta);
    if (jb + 32 < kD) load(jb + 32, ta);
    sum(jb + 16, tb);
  }
  exact_r_finish<LEAN>(hp, s, a, token_lsb(xl), xl, xrow, dtype, r);
}

// Codes and scale of one token from r (lane l: channels l and l + 64, one wave) into the
// LDS row `rec` (zero on entry, zero again on return), then into the cache.  Tile bits are
// set and cleared with device atomics, so tokens that share a tile word may be encoded by
// other waves at the same time.
__device__ inline void store_token_wave(const HeadParams* hp, const float (&r)[2], int layout,
                                        uint8_t* codes, uint16_t* alpha, int64_t cap,
                                        int64_t t, int head, uint32_t* rec) {
  const int lane = threadIdx.x & 63;
  const int rbytes = hp->record_bytes;
  const __half a16 = wave_quantize_into(hp, r, rec);
  if (lane == 0) alpha[(int64_t)head * cap + t] = __half_as_ushort(a16);
  wave_lds_sync();
  if (layout == AATC_LAYOUT_RECORDS) {
    uint32_t* out = reinterpret_cast<uint32_t*>(codes + ((int64_t)head * cap + t) * rbytes);
    for (int i = lane; i < rbytes / 4; i += 64) out[i] = rec[i];
  } else {
    const int p = (int)(t % kTile);
    const uint32_t bit = 1u << tile_bit(p);
    uint32_t* tw = reinterpret_cast<uint32_t*>(codes) +
                   ((int64_t)head * (cap / kTile) + t / kTile) * (16 * rbytes) + tile_word(p);
    for (int v = lane; v < 8 * rbytes; v += 64) {
      if ((rec[v >> 5] >> (v & 31)) & 1u)
        __hip_atomic_fetch_or(tw + 2 * v, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      else
        __hip_atomic_fetch_and(tw + 2 * v, ~bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  wave_lds_sync();
  for (int i = lane; i < kRecWords; i += 64) rec[i] = 0u;
  wave_lds_sync();
}

// One wave per (token, KV head), for appends of a few tokens.
// With `seq_len` set, block x is a sequence instead: it encodes token seq_len[b] - 1 of
// sequence b (nothing for an empty sequence) into caches `codes_bstride` bytes and
// `alpha_bstride` scales apart.
__global__ __launch_bounds__(64) void encode_token_kernel(
    const void* __restrict__ params, const void* __restrict__ x, int dtype, int64_t x_stride,
    int layout, uint8_t* __restrict__ codes, uint16_t* __restrict__ alpha, int64_t cap,
    int64_t pos, const int32_t* __restrict__ seq_len, int64_t codes_bstride,
    int64_t alpha_bstride) {
  __shared__ uint32_t rec[kRecWords];
  int64_t t = pos + blockIdx.x;
  if (seq_len) {
    t = min<int64_t>(max(seq_len[blockIdx.x], 0), cap) - 1;
    if (t < 0) return;
    codes += blockIdx.x * codes_bstride;
    alpha += blockIdx.x * alpha_bstride;
  }
  const int head = blockIdx.y;
  for (int i = threadIdx.x; i < kRecWords; i += 64) rec[i] = 0u;
  wave_lds_sync();
  const void* xrow = static_cast<const char*>(x) +
                     ((int64_t)blockIdx.x * x_stride + (int64_t)head * kD) * (dtype == AATC_BF16 ? 2 : 4);
  const HeadParams* hp = head_params(params, head);
  float xl[2], r[2];
  load_token_pair(xrow, dtype, xl);
  exact_r_wave_pipelined(hp, xl, xrow, dtype, r);
  store_token_wave(hp, r, layout, codes, alpha, cap, t, head, rec);
}

// The tokens the matrix-core kernel left with the mark kRedo.  A workgroup scans the marks
// of kFixTokens tokens of one KV head (eight per thread, read together) and its four waves
// encode the marked tokens exactly, one token per wave at a time, each reading the
// transform columns from the parameter block (a few tokens per workgroup: a copy of the
// transform into LDS would move as many bytes as the reads it saves).
constexpr int kFixThreads = 256;
constexpr int kFixWaves = kFixThreads / 64;
constexpr int kFixTokens = 2048;
__global__ __launch_bounds__(kFixThreads) void encode_fixup_kernel(
    const void* __restrict__ params, const void* __restrict__ x, int dtype, int64_t n_tok,
    int64_t x_stride, int layout, uint8_t* __restrict__ codes, uint16_t* __restrict__ alpha,
    int64_t cap, int64_t pos) {
  __shared__ uint16_t list[kFixTokens];
  __shared__ int n_list;
  __shared__ uint32_t rec[kFixWaves][kRecStride];
  const int head = blockIdx.y, tid = threadIdx.x, wave = tid >> 6;
  const HeadParams* hp = head_params(params, head);
  const int64_t base = (int64_t)blockIdx.x * kFixTokens;
  if (tid == 0) n_list = 0;
  __syncthreads();
  {
    // (all marks of a thread read before any is tested, past the end clamped to the last
    // token: one round trip)
    const uint16_t* am = alpha + (int64_t)head * cap + pos;
    uint16_t mv[kFixTokens / kFixThreads];
#pragma unroll
    for (int m = 0; m < kFixTokens / kFixThreads; ++m)
      mv[m] = am[min<int64_t>(base + tid + kFixThreads * m, n_tok - 1)];
#pragma unroll
    for (int m = 0; m < kFixTokens / kFixThreads; ++m) {
      const int i = tid + kFixThreads * m;
      if (mv[m] == kRedo && base + i < n_tok) list[atomicAdd(&n_list, 1)] = (uint16_t)i;
    }
  }
  __syncthreads();
  const int cnt = n_list;
  if (cnt == 0) return;
  const size_t esize = dtype == AATC_BF16 ? 2 : 4;
  for (int i = tid; i < kFixWaves * kRecStride; i += kFixThreads) (&rec[0][0])[i] = 0u;
  __syncthreads();
  for (int k = wave; k < cnt; k += kFixWaves) {
    const int64_t t = pos + base + list[k];
    const void* xrow = static_cast<const char*>(x) +
                       ((t - pos) * x_stride + (int64_t)head * kD) * esize;
    float xl[2], r[2];
    load_token_pair(xrow, dtype, xl);
    exact_r_wave_pipelined<true>(hp, xl, xrow, dtype, r);
    store_token_wave(hp, r, layout, codes, alpha, cap, t, head, rec[wave]);
  }
}

}  // namespace

aatc_status launch_encode(const void* params, int n_heads, const void* x, aatc_dtype x_dtype,
                          int64_t n_tok, int64_t x_tok_stride, aatc_layout layout,
                          void* codes, uint16_t* alpha, int64_t cap, int64_t pos,
                          void* stream) {
  if (n_tok <= kSmallBatch) {
    hipLaunchKernelGGL(encode_token_kernel, dim3((unsigned)n_tok, (unsigned)n_heads), dim3(64),
                       0, (hipStream_t)stream, params, x, (int)x_dtype, x_tok_stride,
                       (int)layout, static_cast<uint8_t*>(codes), alpha, cap, pos, nullptr,
                       (int64_t)0, (int64_t)0);
    return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
  }
  const int64_t first = pos / kTile, last = (pos + n_tok - 1) / kTile;
  const int64_t n_tiles = last - first + 1;
  const size_t esize = x_dtype == AATC_BF16 ? 2 : 4;
  const bool aligned = (reinterpret_cast<uintptr_t>(x) % 16 == 0) &&
                       ((size_t)x_tok_stride * esize) % 16 == 0;
  if (aligned) {
    // About one workgroup of twelve waves per compute unit over all KV heads.
    const int64_t per_head = std::min<int64_t>(std::max(1, 256 / n_heads),
                                               (2 * n_tiles + kMW - 1) / kMW);
    dim3 grid((unsigned)per_head, (unsigned)n_heads);
    if (x_dtype == AATC_BF16)
      hipLaunchKernelGGL(encode_mfma_kernel<true>, grid, dim3(kMThreads), 0,
                         (hipStream_t)stream, params, x, n_tok, x_tok_stride, (int)layout,
                         static_cast<uint8_t*>(codes), alpha, cap, pos);
    else
      hipLaunchKernelGGL(encode_mfma_kernel<false>, grid, dim3(kMThreads), 0,
                         (hipStream_t)stream, params, x, n_tok, x_tok_stride, (int)layout,
                         static_cast<uint8_t*>(codes), alpha, cap, pos);
    if (hipGetLastError() != hipSuccess) return AATC_E_DEVICE;
    // The tokens whose certificate failed, exactly (stream order: after the kernel above).
    const dim3 fgrid((unsigned)((n_tok + kFixTokens - 1) / kFixTokens), (unsigned)n_heads);
    hipLaunchKernelGGL(encode_fixup_kernel, fgrid, dim3(kFixThreads), 0, (hipStream_t)stream, params, x,
                       (int)x_dtype, n_tok, x_tok_stride, (int)layout,
                       static_cast<uint8_t*>(codes), alpha, cap, pos);
    return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
  }
  dim3 grid((unsigned)n_tiles, (unsigned)n_heads);
  hipLaunchKernelGGL(encode_exact_kernel, grid, dim3(kEncThreads), 0, (hipStream_t)stream,
                     params, x, (int)x_dtype, n_tok, x_tok_stride, (int)layout,
                     static_cast<uint8_t*>(codes), alpha, cap, pos);
  return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
}

aatc_status launch_encode_last(const void* params, int n_heads, int batch, const void* x,
                               aatc_dtype x_dtype, aatc_layout layout, void* codes,
                               uint16_t* alpha, int64_t cap, int record_bytes,
                               const int32_t* seq_len, void* stream) {
  hipLaunchKernelGGL(encode_token_kernel, dim3((unsigned)batch, (unsigned)n_heads), dim3(64), 0,
                     (hipStream_t)stream, params, x, (int)x_dtype, (int64_t)n_heads * kD,
                     (int)layout, static_cast<uint8_t*>(codes), alpha, cap, (int64_t)0, seq_len,
                     (int64_t)n_heads * cap * record_bytes, (int64_t)n_heads * cap);
  return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
}

}  // namespace aatc
