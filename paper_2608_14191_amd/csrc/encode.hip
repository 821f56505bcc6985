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
// Per token, X_j = rint(x_j 2^S) with S such that max |X| lies in [2^21, 2^22), and the
// integer transform Tq = T 2^22 (|Tq| <= 2^22).  Both split into balanced int8 limbs,
// X = 2^16 X2 + 2^8 X1 + X0 and Tq = 2^16 T2 + 2^8 T1 + T0 (|X2|, |T2| <= 64, the others
// in [-128, 127]), and the nine limb products go to v_mfma_i32_16x16x64_i8 in five int32
// sums by weight, S_k = sum over a + b = k of sum_j X_a T_b (each below 2^23, exact).
// H = sum_k 2^(8k) S_k = sum_j X_j Tq_jc is below 2^51 and is formed exactly in fp64.
//   - If every X_j equals x_j 2^S (the token is exact in fixed point), H 2^-(S+22) is the
//     exact h and one rounding gives the canonical result.
//   - Otherwise |h - H 2^-(S+22)| <= E 2^-S with E = sum_j |x_j 2^S - X_j|.  The token's
//     scale and codes are certified against that bound: alpha if the fp16 rounding of the
//     largest |r| cannot change within it, each code if its fp32 quantizer input lies
//     farther than the bound (plus the fp32 roundings of both evaluations) from a rounding
//     boundary.  A token that fails is encoded again by the exact one-wave routine.
// One workgroup of four waves takes 64-token tiles of one KV head in a grid-stride loop
// (the limb tables of the head's transform are built once per workgroup); wave w takes
// tokens 16 w .. 16 w + 15 against all 128 channels.  Lane 16 kg + n reads token n's
// elements j = 64 kc + 16 kg .. + 15 (kc = 0, 1): the B operand columns; the A operand lane
// (channel 16 ct + n) reads the same j of row c of the limb tables.  The products leave
// lane 16 kg + n with channels 16 ct + 4 kg + i, i < 4, of its own token, so a lane's four
// consecutive codes go into the record as one bit field.
// Needs 16-byte aligned token rows (checked by the launcher).
// ---------------------------------------------------------------------------------------
// Limb tables in matrix-core operand order: the 16 bytes lane l of a wave feeds for
// channel tile ct and k half kc sit at ((2 ct + kc) 64 + l) 16, so every operand read is one
// contiguous 1 KiB per wave (no bank conflicts).
constexpr int kTbBytes = 8 * 2 * 64 * 16;       // one limb of the 128 x 128 transform

typedef int ev4i __attribute__((ext_vector_type(4)));

template <int CTRL>
__device__ inline float enc_dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
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

// One stage of a 32 x 32 bit-matrix transpose over the 32 lanes of each half wave (lane i
// holds row i): blocks of S bits are exchanged with lane i ^ S.
template <int S, uint32_t M>
__device__ inline uint32_t bit_transpose_stage(uint32_t x, int lane) {
  const uint32_t y = (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, 0x1f | (S << 10));
  return (lane & S) ? ((x & ~M) | ((y >> S) & M)) : ((x & M) | ((y & M) << S));
}

template <bool BF16>
__device__ inline void load_token_elems(const void* x, int64_t base, int kg, float (&xv)[2][16]) {
#pragma unroll
  for (int kc = 0; kc < 2; ++kc) {
    if constexpr (BF16) {
      const uint4* p = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(x) + base +
                                                      64 * kc + 16 * kg);
      const uint4 u[2] = {p[0], p[1]};
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const uint32_t wv[4] = {u[q].x, u[q].y, u[q].z, u[q].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          xv[kc][8 * q + 2 * e] = __uint_as_float(wv[e] << 16);
          xv[kc][8 * q + 2 * e + 1] = __uint_as_float(wv[e] & 0xffff0000u);
        }
      }
    } else {
      const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(x) + base +
                                                        64 * kc + 16 * kg);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 f = p[q];
        xv[kc][4 * q] = f.x, xv[kc][4 * q + 1] = f.y, xv[kc][4 * q + 2] = f.z,
        xv[kc][4 * q + 3] = f.w;
      }
    }
  }
}

// The int8 limb bytes of four integers |v| < 2^22 (or |v| <= 2^22 for the transform):
// limb 0 = byte 0 of v, limb 1 = byte 1 of v + 128, limb 2 = byte 2 of v + 32896 (the
// balanced digits: v = 65536 l2 + 256 l1 + l0 with l0, l1 in [-128, 127]).
__device__ inline void limb_bytes4(const int (&v)[4], uint32_t (&out)[3]) {
  uint32_t y1[4], y2[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    y1[e] = (uint32_t)(v[e] + 128);
    y2[e] = (uint32_t)(v[e] + 32896);
  }
  // v_perm_b32(a, b, sel): byte k of the result is byte sel_k of the pair {a: 4..7, b: 0..3}
  out[0] = __builtin_amdgcn_perm((uint32_t)v[1], (uint32_t)v[0], 0x0c0c0400u) |
           __builtin_amdgcn_perm((uint32_t)v[3], (uint32_t)v[2], 0x04000c0cu);
  out[1] = __builtin_amdgcn_perm(y1[1], y1[0], 0x0c0c0501u) |
           __builtin_amdgcn_perm(y1[3], y1[2], 0x05010c0cu);
  out[2] = __builtin_amdgcn_perm(y2[1], y2[0], 0x0c0c0602u) |
           __builtin_amdgcn_perm(y2[3], y2[2], 0x06020c0cu);
}

template <bool BF16>
__global__ __attribute__((amdgpu_flat_work_group_size(kEncThreads, kEncThreads),
                          amdgpu_waves_per_eu(2, 2))) void encode_mfma_kernel(
    const void* __restrict__ params, const void* __restrict__ x, int64_t n_tok,
    int64_t x_stride, int layout, uint8_t* __restrict__ codes, uint16_t* __restrict__ alpha,
    int64_t cap, int64_t pos) {
  static_assert(kEncThreads == 256, "four waves of 16 tokens per 64-token tile");
  __shared__ __align__(16) int8_t tb[3][kTbBytes];       // [limb][ct][kc][lane][16]
  __shared__ uint32_t rec[kTile][kRecStride];              // records of the tile's tokens
  // Channel tables, read per tile by the lanes that hold channels 16 ct + 4 kg + i.
  __shared__ __align__(16) float tab_is[kD];              // 1 / s_c
  __shared__ __align__(16) float tab_k[kD];               // 2^(b_c - 1) / s_c (1 + 2^-20)
  __shared__ __align__(16) float tab_p2[kD];              // 2^(b_c - 1) (1 for b_c = 0)
  __shared__ __align__(16) float tab_hi[kD];              // 2^(b_c - 1) - 1: largest code
  __shared__ __align__(16) uint32_t tab_msk[kD];          // 2^b_c - 1
  __shared__ __align__(16) uint32_t tab_sh[kD];           // bit of c in its group's field
  __shared__ __align__(16) uint32_t tab_w[kD / 4];        // width of each group of four
  __shared__ __align__(16) uint16_t tab_o[kD];            // first record bits

  const int head = blockIdx.y;
  const HeadParams* hp = head_params(params, head);
  const int rwords = hp->record_bytes / 4;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, n = lane & 15, kg = lane >> 4;
  const int dtype = BF16 ? AATC_BF16 : AATC_F32;
  // Channels wider than 8 bits: four consecutive codes may not fit one 32-bit field, so
  // such tensors take the exact one-wave routine per token (uniform over the grid).
  if (hp->max_bits > 8) {
    for (int i = tid; i < kTile * kRecStride; i += kEncThreads) (&rec[0][0])[i] = 0u;
    __syncthreads();
    for (int64_t tile = pos / kTile + blockIdx.x; tile <= (pos + n_tok - 1) / kTile;
         tile += gridDim.x)
      exact_tile(hp, x, dtype, n_tok, x_stride, layout, codes, alpha, cap, pos, tile, head, rec);
    return;
  }
  const bool midrise = hp->quantizer == AATC_QUANT_MIDRISE;

  // Limb tables of the transposed integer transform: operand slot u = (2 ct + kc) 64 + l
  // (l = 16 kg + n) holds Tq^T[16 ct + n][64 kc + 16 kg .. + 15]; thread tid fills slots
  // tid + 256 k.
  for (int k = 0; k < 4; ++k) {
    const int u = tid + kEncThreads * k, l = u & 63, ct = u >> 7, kc = (u >> 6) & 1;
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
    tab_msk[tid] = (1u << b) - 1u;
    int sh = 0;
    for (int c = tid & ~3; c < tid; ++c) sh += hp->bits[c];
    tab_sh[tid] = (uint32_t)sh;
    tab_o[tid] = hp->bit_off[tid];
  }
  if (tid < kD / 4)
    tab_w[tid] = hp->bits[4 * tid] + hp->bits[4 * tid + 1] + hp->bits[4 * tid + 2] + hp->bits[4 * tid + 3];
  for (int i = tid; i < kTile * kRecStride; i += kEncThreads) (&rec[0][0])[i] = 0u;
  // Value tiles: lane p of a wave stands for tile bit position p (word p / 32, bit p % 32),
  // i.e. token 16 (2 (p / 32) + p % 2) + 4 ((p / 2) % 4) + (p % 32) / 8.
  const int ptok = 16 * (2 * (lane >> 5) + (lane & 1)) + 4 * ((lane >> 1) & 3) + ((lane & 31) >> 3);

  const int64_t first = pos / kTile, last = (pos + n_tok - 1) / kTile;
  // Token 16 wave + n of the tile: the element loads run one tile ahead.
  const int tl = 16 * wave + n;
  float xv[2][16];
  auto fetch = [&](int64_t tile) {
    const int64_t t = tile * kTile + tl;
    if (tile <= last && t >= pos && t < pos + n_tok) {
      load_token_elems<BF16>(x, (t - pos) * x_stride + (int64_t)head * kD, kg, xv);
    } else {
#pragma unroll
      for (int kc = 0; kc < 2; ++kc)
#pragma unroll
        for (int e = 0; e < 16; ++e) xv[kc][e] = 0.f;
    }
  };
  fetch(first + blockIdx.x);
  for (int64_t tile = first + blockIdx.x; tile <= last; tile += gridDim.x) {
    const int64_t tile_base = tile * kTile;
    const int64_t t_begin = max(tile_base, pos);
    const int64_t t_end = min(tile_base + kTile, pos + n_tok);
    const bool valid = tile_base + tl >= t_begin && tile_base + tl < t_end;
    // (1) The token's fixed-point shift (max over its 128 elements: 4 lanes).
    float m = 0.f;
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int e = 0; e < 16; ++e) m = fmaxf(m, fabsf(xv[kc][e]));
    const int shift = token_shift(enc_cross_row_max(m));
    // (2) The limbs of X = rint(x 2^shift) as B operands (byte e: element e), and this
    //     lane's part of E = sum_j |x_j 2^shift - X_j| (exact: each term is).
    ev4i A[3][2];
    float E = 0.f;
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int X[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float v = ldexpf(xv[kc][4 * q + e], shift);
          const float vr = rintf(v);
          X[e] = (int)vr;
          E += fabsf(v - vr);
        }
        uint32_t lb[3];
        limb_bytes4(X, lb);
#pragma unroll
        for (int l = 0; l < 3; ++l) A[l][kc][q] = (int)lb[l];
      }
    fetch(tile + gridDim.x);                      // the next tile's elements, in flight
    if (tile == first + blockIdx.x) __syncthreads();   // (the limb and channel tables)
    // The token's fixed-point error bound: |h_c - h~_c| <= eh for every channel (|T| <= 1).
    // Waves with an inexact token certify their codes (below).
    const float Et = enc_cross_row_sum(E);
    const bool cert = __builtin_amdgcn_ballot_w64(Et > 0.f) != 0ull;
    const float eh = ldexpf(Et * (1.f + 0x1p-16f), -shift);
    // (3) Four channel tiles at a time: the five limb-product sums, H exactly, then
    //     r_c = fl32(fl32(H 2^-(S+22)) / s_c) for channels 16 ct + 4 kg + i of this token.
    //     With a certificate, also the range of the exact max |r_c|: each r_c is within
    //     eh / s_c (plus fp32 roundings) of its computed value.
    float r[8][4], am = 0.f, alo = 0.f, ahi = 0.f;
#pragma unroll
    for (int c4 = 0; c4 < 8; c4 += 4) {
      ev4i s[5][4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int k = 0; k < 5; ++k) s[k][u] = (ev4i){0, 0, 0, 0};
#pragma unroll
      for (int kc = 0; kc < 2; ++kc)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int o = 16 * ((2 * (c4 + u) + kc) * 64 + lane);
          const ev4i b0 = *reinterpret_cast<const ev4i*>(&tb[0][o]);
          const ev4i b1 = *reinterpret_cast<const ev4i*>(&tb[1][o]);
          const ev4i b2 = *reinterpret_cast<const ev4i*>(&tb[2][o]);
          s[4][u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b2, A[2][kc], s[4][u], 0, 0, 0);
          s[3][u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b2, A[1][kc], s[3][u], 0, 0, 0);
          s[2][u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b2, A[0][kc], s[2][u], 0, 0, 0);
          s[1][u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b1, A[0][kc], s[1][u], 0, 0, 0);
          s[0][u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b0, A[0][kc], s[0][u], 0, 0, 0);
          s[3][u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b1, A[2][kc], s[3][u], 0, 0, 0);
          s[2][u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b1, A[1][kc], s[2][u], 0, 0, 0);
          s[1][u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b0, A[1][kc], s[1][u], 0, 0, 0);
          s[2][u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b0, A[2][kc], s[2][u], 0, 0, 0);
        }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int ct = c4 + u, c0 = 16 * ct + 4 * kg;
        const float4 is4 = *reinterpret_cast<const float4*>(&tab_is[c0]);
        const float isv[4] = {is4.x, is4.y, is4.z, is4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // H = 2^16 (2^8 (2^8 S4 + S3) + S2) + (2^8 S1 + S0): exact in fp64 (< 2^51).
          const int hi = s[4][u][i] * 256 + s[3][u][i];
          const int lo = s[1][u][i] * 256 + s[0][u][i];
          const double H = fma(fma((double)hi, 256.0, (double)s[2][u][i]), 65536.0, (double)lo);
          r[ct][i] = integer_result(H, shift) * isv[i];
          am = fmaxf(am, fabsf(r[ct][i]));          // (r = 0 on dropped channels)
          if (cert) {
            const float er = eh * isv[i] * (1.f + 0x1p-20f);
            alo = fmaxf(alo, fabsf(r[ct][i]) - er);
            ahi = fmaxf(ahi, fabsf(r[ct][i]) + er);
          }
        }
      }
      // (one half's accumulators at a time)
      __builtin_amdgcn_sched_barrier(0);
    }
    // (4) The token's scale (its 128 channels: 4 lanes), its codes and record: channels
    //     16 ct + 4 kg .. + 3 are consecutive in the record, one bit field of <= 32 bits.
    const float amax = enc_cross_row_max(am);
    const __half a16 = token_alpha(amax);
    const float inv_a = inverse_alpha(a16);
    uint32_t field[8];
    bool uncertain = false;
    auto codes_of = [&](auto certify, auto mid_rise) {
      constexpr bool CERT = decltype(certify)::value;
      constexpr bool MR = decltype(mid_rise)::value;
      float ea = 0.f;
      if constexpr (CERT) {
        // The fp16 scale is certain when both ends of the range of the exact max |r_c|
        // (over the token's four lanes), widened by the fp32 roundings, round alike.
        // eh = E 2^-S (1 + 2^-16) covers the fp32 sum of E; ldexpf may underflow to 0
        // only below the absolute slack.
        const float lo = enc_cross_row_max(alo) - 0x1p-21f * amax;
        const float hi = enc_cross_row_max(ahi) + 0x1p-21f * amax + 0x1p-140f;
        uncertain = __half_as_ushort(token_alpha(fmaxf(lo, 0.f))) !=
                    __half_as_ushort(token_alpha(hi));
        ea = eh * inv_a;
      }
#pragma unroll
      for (int ct = 0; ct < 8; ++ct) {
        const int c0 = 16 * ct + 4 * kg;
        const float4 p4 = *reinterpret_cast<const float4*>(&tab_p2[c0]);
        const float4 h4 = *reinterpret_cast<const float4*>(&tab_hi[c0]);
        const uint4 m4 = *reinterpret_cast<const uint4*>(&tab_msk[c0]);
        const uint4 s4 = *reinterpret_cast<const uint4*>(&tab_sh[c0]);
        const float p2[4] = {p4.x, p4.y, p4.z, p4.w}, hv[4] = {h4.x, h4.y, h4.z, h4.w};
        const uint32_t mk[4] = {m4.x, m4.y, m4.z, m4.w}, sh[4] = {s4.x, s4.y, s4.z, s4.w};
        float4 k4;
        if constexpr (CERT) k4 = *reinterpret_cast<const float4*>(&tab_k[c0]);
        uint32_t f = 0u;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // The canonical quantizer: xq = fl32(r / alpha) 2^(b-1) (the power of two is
          // exact), code = floor(xq + 1/2) (midtread) or floor(xq) (midrise) clamped to
          // [-2^(b-1), 2^(b-1) - 1], b-bit two's complement.  Clamping xq first (the bounds
          // are integers) and then rounding gives the same code; for midtread the rounding
          // half up is one v_cvt_rpi_i32_f32 (checked on the hardware against floor(xq) +
          // (frac >= 1/2): boundary values within 64 ulps of k and k + 1/2 for |k| <= 130,
          // 2^24 values in all).  Dropped channels have r = 0 and mask 0.
          const float xq = (r[ct][i] * inv_a) * p2[i];
          const float xc = __builtin_amdgcn_fmed3f(xq, -p2[i], hv[i]);
          int code;
          if constexpr (MR)
            code = (int)floorf(xc);
          else
            asm("v_cvt_rpi_i32_f32 %0, %1" : "=v"(code) : "v"(xc));
          if constexpr (CERT) {
            const float kf = i == 0 ? k4.x : i == 1 ? k4.y : i == 2 ? k4.z : k4.w;
            // the bound in x units, plus both evaluations' fp32 roundings and that of
            // xq + 1/2
            const float mg = fmaf(kf, ea, fmaf(0x1p-21f, fabsf(xq), 0x1p-22f));
            uncertain |= boundary_distance(xq, MR) <= mg;
          }
          f |= ((uint32_t)code & mk[i]) << sh[i];
        }
        field[ct] = f;
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
    const bool redo = enc_cross_row_max(uncertain ? 1.f : 0.f) > 0.f;
    if (valid && !redo) {
#pragma unroll
      for (int ct = 0; ct < 8; ++ct) {
        const int c0 = 16 * ct + 4 * kg;
        const int width = (int)tab_w[c0 >> 2];
        const int off = tab_o[c0];
        if (width > 0) {
          atomicOr(&rec[tl][off >> 5], field[ct] << (off & 31));
          if ((off & 31) + width > 32) atomicOr(&rec[tl][(off >> 5) + 1], field[ct] >> (32 - (off & 31)));
        }
      }
      if (kg == 0) alpha[(int64_t)head * cap + tile_base + tl] = __half_as_ushort(a16);
    }
    // (5) A token that failed the certificate keeps a zero record row here and the mark
    //     kRedo as its scale; encode_fixup_kernel, launched next on the stream, encodes it
    //     with the exact one-wave routine (a few in ten thousand tokens; done here, each
    //     would stall the whole workgroup for several dependent memory round trips).
    if (valid && redo && kg == 0) alpha[(int64_t)head * cap + tile_base + tl] = kRedo;
    __syncthreads();
    const int lo = (int)(t_begin - tile_base), hi = (int)(t_end - tile_base);
    if (layout == AATC_LAYOUT_RECORDS) {
      uint32_t* out = reinterpret_cast<uint32_t*>(codes) + ((int64_t)head * cap + tile_base) * rwords;
      for (int i = lo * rwords + tid; i < hi * rwords; i += kEncThreads) {
        out[i] = rec[i / rwords][i % rwords];
        rec[i / rwords][i % rwords] = 0u;          // (each word read and cleared by one thread)
      }
    } else {
      // Record word w of the tile's tokens -> tile words 64 w .. 64 w + 63.  Lane p holds
      // the word of the token at position p; a 32 x 32 bit transpose within each half of
      // the wave (five butterfly stages on lane-xor swizzles) leaves lane 32 W + b with bit
      // 32 w + b over the positions of half W: tile word 2 (32 w + b) + W.
      uint32_t* out = reinterpret_cast<uint32_t*>(codes) +
                      ((int64_t)head * (cap / kTile) + tile) * (16 * rwords * 4);
      const uint64_t vmask = __builtin_amdgcn_ballot_w64(ptok >= lo && ptok < hi);
      const uint32_t keep = ~(uint32_t)((lane >> 5) ? (vmask >> 32) : vmask);
      for (int w = wave; w < rwords; w += kEncThreads / 64) {
        uint32_t xw = rec[ptok][w];
        rec[ptok][w] = 0u;                          // (each word read and cleared by one lane)
        xw = bit_transpose_stage<16, 0x0000ffffu>(xw, lane);
        xw = bit_transpose_stage<8, 0x00ff00ffu>(xw, lane);
        xw = bit_transpose_stage<4, 0x0f0f0f0fu>(xw, lane);
        xw = bit_transpose_stage<2, 0x33333333u>(xw, lane);
        xw = bit_transpose_stage<1, 0x55555555u>(xw, lane);
        uint32_t* o = out + 64 * w + 2 * (lane & 31) + (lane >> 5);
        *o = keep ? ((*o & keep) | (xw & ~keep)) : xw;
      }
    }
    __syncthreads();                                // (the cleared rows before the next tile's bits)
  }
}

// One token of one KV head by one wave (the exact one-wave routine): codes into the LDS
// row `rec` (zero on entry), then into the cache.  Tile bits are set and cleared with
// device atomics, so tokens that share a tile word may be encoded by other workgroups.
__device__ __forceinline__ void encode_token_wave(const HeadParams* hp, const void* xrow,
                                                  int dtype, int layout, uint8_t* codes,
                                                  uint16_t* alpha, int64_t cap, int64_t t,
                                                  int head, uint32_t* rec) {
  const int lane = threadIdx.x & 63;
  const int rbytes = hp->record_bytes;
  float xl[2], r[2];
  load_token_pair(xrow, dtype, xl);
  exact_r_wave(hp, xl, xrow, dtype, r);
  const __half a16 = wave_quantize_into(hp, r, rec);
  if (lane == 0) alpha[(int64_t)head * cap + t] = __half_as_ushort(a16);
  __syncthreads();                                  // (the record, one wave)
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
  if (threadIdx.x < kRecWords) rec[threadIdx.x] = 0u;
  __syncthreads();
  const void* xrow = static_cast<const char*>(x) +
                     ((int64_t)blockIdx.x * x_stride + (int64_t)head * kD) * (dtype == AATC_BF16 ? 2 : 4);
  encode_token_wave(head_params(params, head), xrow, dtype, layout, codes, alpha, cap, t, head,
                    rec);
}

// The tokens the matrix-core kernel left with the mark kRedo (failed certificates): one
// wave per workgroup scans 64 tokens at a time of each KV head and encodes the marked ones
// exactly.
__global__ __launch_bounds__(64) void encode_fixup_kernel(
    const void* __restrict__ params, const void* __restrict__ x, int dtype, int64_t n_tok,
    int64_t x_stride, int layout, uint8_t* __restrict__ codes, uint16_t* __restrict__ alpha,
    int64_t cap, int64_t pos) {
  __shared__ uint32_t rec[kRecWords];
  const int head = blockIdx.y, lane = threadIdx.x;
  const HeadParams* hp = head_params(params, head);
  for (int64_t b = (int64_t)blockIdx.x * 64; b < n_tok; b += (int64_t)gridDim.x * 64) {
    const int64_t t = pos + b + lane;
    const bool mark = b + lane < n_tok && alpha[(int64_t)head * cap + t] == kRedo;
    uint64_t m = __builtin_amdgcn_ballot_w64(mark);
    while (m) {
      const int64_t tk = pos + b + __builtin_ctzll(m);
      m &= m - 1;
      if (lane < kRecWords) rec[lane] = 0u;
      __syncthreads();
      const void* xrow = static_cast<const char*>(x) +
                         ((tk - pos) * x_stride + (int64_t)head * kD) * (dtype == AATC_BF16 ? 2 : 4);
      encode_token_wave(hp, xrow, dtype, layout, codes, alpha, cap, tk, head, rec);
      __syncthreads();                              // (rec is cleared for the next token)
    }
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
    // A grid-stride loop of at most 64 workgroups per KV head (each builds the head's limb
    // tables once; two per compute unit over the 8 heads of the reference shapes).
    dim3 grid((unsigned)std::min<int64_t>(n_tiles, 64), (unsigned)n_heads);
    if (x_dtype == AATC_BF16)
      hipLaunchKernelGGL(encode_mfma_kernel<true>, grid, dim3(kEncThreads), 0,
                         (hipStream_t)stream, params, x, n_tok, x_tok_stride, (int)layout,
                         static_cast<uint8_t*>(codes), alpha, cap, pos);
    else
      hipLaunchKernelGGL(encode_mfma_kernel<false>, grid, dim3(kEncThreads), 0,
                         (hipStream_t)stream, params, x, n_tok, x_tok_stride, (int)layout,
                         static_cast<uint8_t*>(codes), alpha, cap, pos);
    if (hipGetLastError() != hipSuccess) return AATC_E_DEVICE;
    // The tokens whose certificate failed, exactly (stream order: after the kernel above).
    const dim3 fgrid((unsigned)std::min<int64_t>((n_tok + 63) / 64, 512), (unsigned)n_heads);
    hipLaunchKernelGGL(encode_fixup_kernel, fgrid, dim3(64), 0, (hipStream_t)stream, params, x,
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
