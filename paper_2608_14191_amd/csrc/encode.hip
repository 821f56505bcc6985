// AATC encode on gfx950: transform, per-token scale, quantize, pack (Algorithm 1,
// inference part; Sec. 5.2).  Exact VALU kernel: the transform is evaluated as an exact
// integer dot product on fixed-point operands, so every code is reproducible bit for
// bit.  Works for any token count; one workgroup per (64-token tile, KV head).
#include <algorithm>

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "encode_core.h"
#include "launch.h"
#include "params.h"

namespace aatc {
namespace {

constexpr int kEncThreads = 256;                 // two tokens in flight, 128 lanes each
constexpr int kRecWords = kMaxBudget / 32;       // words of the largest record
constexpr int kSmallBatch = 16;                  // appends up to this many tokens: per-token kernel

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__global__ __launch_bounds__(kEncThreads) void encode_exact_kernel(
    const void* __restrict__ params, const void* __restrict__ x, int dtype, int64_t n_tok,
    int64_t x_stride, int layout, uint8_t* __restrict__ codes, uint16_t* __restrict__ alpha,
    int64_t cap, int64_t pos) {
  __shared__ int16_t tq[kD * kD];                 // fixed-point transform of this head
  __shared__ uint32_t rec[kTile][kRecWords];      // records of the tile's tokens
  __shared__ int xs[2][kD];
  __shared__ float red_x[4], red_a[4];

  const int head = blockIdx.y;
  const HeadParams* hp = head_params(params, head);
  const int rbytes = hp->record_bytes;
  const int rwords = rbytes / 4;
  const int64_t tile = pos / kTile + blockIdx.x;
  const int64_t tile_base = tile * kTile;
  const int64_t t_begin = max(tile_base, pos);
  const int64_t t_end = min(tile_base + kTile, pos + n_tok);

  const int tid = threadIdx.x;
  const int slot = tid >> 7;
  const int c = tid & (kD - 1);
  const int wave = tid >> 6;

  for (int i = tid; i < kD * kD / 2; i += kEncThreads)
    reinterpret_cast<uint32_t*>(tq)[i] = reinterpret_cast<const uint32_t*>(hp->Tq)[i];
  for (int i = tid; i < kTile * kRecWords; i += kEncThreads) (&rec[0][0])[i] = 0u;
  const int b = hp->bits[c];
  const int off = hp->bit_off[c];
  const float inv_s = hp->inv_s[c];
  __syncthreads();

  for (int64_t t0 = t_begin; t0 < t_end; t0 += 2) {
    const int64_t t = t0 + slot;
    const bool valid = t < t_end;
    const float xv = valid ? load_elem(x, dtype, (t - pos) * x_stride + (int64_t)head * kD + c) : 0.f;
    // Per-token fixed-point scale: max |x_j| goes to [2^13, 2^14).
    float m = wave_max(fabsf(xv));
    if ((tid & 63) == 0) red_x[wave] = m;
    __syncthreads();
    m = fmaxf(red_x[2 * slot], red_x[2 * slot + 1]);
    const int shift = token_shift(m);
    xs[slot][c] = (int)rintf(ldexpf(xv, shift));
    __syncthreads();
    // Exact integer transform h_c = sum_j X_j Tq_jc (|sum| < 2^36).
    long long acc = 0;
#pragma unroll 8
    for (int j = 0; j < kD; ++j) acc += (long long)xs[slot][j] * (long long)tq[j * kD + c];
    const float r = fixed_point_result(acc, shift) * inv_s;
    float a = wave_max(b > 0 ? fabsf(r) : 0.f);
    if ((tid & 63) == 0) red_a[wave] = a;
    __syncthreads();
    a = fmaxf(red_a[2 * slot], red_a[2 * slot + 1]);
    const __half a16 = token_alpha(a);
    const float inv_a = inverse_alpha(a16);
    if (valid && b > 0) {
      const uint32_t u = quantize_code(r, inv_a, b);
      const int li = (int)(t - tile_base);
      atomicOr(&rec[li][off >> 5], u << (off & 31));
      if ((off & 31) + b > 32) atomicOr(&rec[li][(off >> 5) + 1], u >> (32 - (off & 31)));
    }
    if (valid && c == 0) alpha[(int64_t)head * cap + t] = __half_as_ushort(a16);
    __syncthreads();
  }

  const int lo = (int)(t_begin - tile_base), hi = (int)(t_end - tile_base);
  if (layout == AATC_LAYOUT_RECORDS) {
    uint32_t* out = reinterpret_cast<uint32_t*>(codes) + ((int64_t)head * cap + tile_base) * rwords;
    for (int i = lo * rwords + tid; i < hi * rwords; i += kEncThreads)
      out[i] = rec[i / rwords][i % rwords];
  } else {
    // Bit-transposed tile: word 2 v + W holds record bit v of the tile's tokens
    // t = 16 d + 4 g + i with d / 2 = W, at bit 8 i + 2 g + d % 2.
    uint32_t* out = reinterpret_cast<uint32_t*>(codes) +
                    ((int64_t)head * (cap / kTile) + tile) * (16 * rbytes);
    for (int wi = tid; wi < 16 * rbytes; wi += kEncThreads) {
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
  }
}

// The same canonical encode with the transform on the matrix cores.  The exact integer
// dot product h_c = sum_j X_j Tq_jc is split into int8 limbs, X = 256 X1 + X0 and
// Tq = 256 B1 + B0 (X0, B0 in [-128, 127]; X1, B1 in [-64, 64]), and formed from three
// v_mfma_i32_16x16x64_i8 sums that stay exact in int32: S11 = sum X1 B1 (< 2^19),
// S10 = sum X1 B0 + X0 B1 (< 2^22), S00 = sum X0 B0 (< 2^21); then
// h_c = 65536 S11 + (256 S10 + S00) in int64.  Everything after the dot product is the
// exact kernel's arithmetic, so the codes agree bit for bit.
// One workgroup of 4 waves per 64-token tile at a time (a grid-stride loop over the tiles
// of a KV head, so the limb tables of the head's transform are built once per workgroup);
// wave w takes the tile's tokens 16 w .. 16 w + 15 against all 128 channels.  Lane
// 16 kg + n reads token n's elements j = 64 kc + 16 kg .. + 15 (kc = 0, 1): the B operand
// columns; the A operand lane (channel 16 ct + n) reads the same j of row c of Tq^T.  The
// products leave lane 16 kg + n with channels 16 ct + 4 kg + i, i < 4, of its own token, so
// a lane's four consecutive codes go into the record as one bit field.
// Needs 16-byte aligned token rows (checked by the launcher).
constexpr int kTbPitch = 144;                    // bytes per channel row of the limb tables

typedef int ev4i __attribute__((ext_vector_type(4)));

// The canonical quantizer without branches: the same code as quantize_code for b >= 1,
// and 0 for b = 0 (whose r is 0: 1/s is stored as 0 for dropped channels).  The rounding
// floor(xq) + (frac(xq) >= 0.5) is one v_cvt_rpi_i32_f32, which rounds the exact
// xq + 1/2 down (checked against the two-step form on the hardware: boundary values
// k + 1/2 and k within 64 ulps for |k| <= 130, and 2^24 values in all).
__device__ inline uint32_t quantize_code_nb(float r, float inv_a, int b) {
  const int bb = max(b, 1);
  const float xq = ldexpf(r * inv_a, bb - 1);
  int code;
  asm("v_cvt_rpi_i32_f32 %0, %1" : "=v"(code) : "v"(xq));
  const int half = 1 << (bb - 1);
  code = min(max(code, -half), half - 1);
  return __builtin_amdgcn_ubfe((uint32_t)code, 0u, (uint32_t)b);
}

// Low balanced int8 limb of |v| <= 2^14: v = 256 hi + lo with lo in [-128, 127].
__device__ inline int limb_lo(int v) { return ((v + 128) & 255) - 128; }

template <int CTRL>
__device__ inline float enc_dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
// Maximum over each row of 16 lanes.
__device__ inline float enc_row16_max(float v) {
  v = fmaxf(v, enc_dpp<0xB1>(v));
  v = fmaxf(v, enc_dpp<0x4E>(v));
  v = fmaxf(v, enc_dpp<0x124>(v));
  return fmaxf(v, enc_dpp<0x128>(v));
}
// Maximum over lanes l, l ^ 16, l ^ 32 and l ^ 48 (the gfx950 row swaps).
__device__ inline float enc_cross_row_max(float v) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
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

template <bool BF16>
__global__ __attribute__((amdgpu_flat_work_group_size(kEncThreads, kEncThreads),
                          amdgpu_waves_per_eu(3, 3))) void encode_mfma_kernel(
    const void* __restrict__ params, const void* __restrict__ x, int64_t n_tok,
    int64_t x_stride, int layout, uint8_t* __restrict__ codes, uint16_t* __restrict__ alpha,
    int64_t cap, int64_t pos) {
  static_assert(kEncThreads == 256, "four waves of 16 tokens per 64-token tile");
  __shared__ __align__(16) int8_t tb[2][kD * kTbPitch];   // [limb][channel c][j]
  __shared__ uint32_t rec[kTile][kRecWords];              // records of the tile's tokens
  __shared__ __align__(16) float tab_is[kD];              // 1 / s_c
  __shared__ __align__(16) uint32_t tab_b[kD / 4];        // widths, four channels a word
  __shared__ __align__(16) uint16_t tab_o[kD];            // first record bits

  const int head = blockIdx.y;
  const HeadParams* hp = head_params(params, head);
  const int rbytes = hp->record_bytes;
  const int rwords = rbytes / 4;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, n = lane & 15, kg = lane >> 4;

  // Limb tables of the transposed fixed-point transform: thread tid converts elements
  // 8 (tid + 256 k) .. + 7 of Tq^T (all 16-byte loads issued first).
  {
    uint4 tw[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) tw[k] = reinterpret_cast<const uint4*>(hp->Tqt)[tid + kEncThreads * k];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int e0 = 8 * (tid + kEncThreads * k), c = e0 >> 7, j = e0 & (kD - 1);
      const uint32_t wv[4] = {tw[k].x, tw[k].y, tw[k].z, tw[k].w};
      uint32_t lo[2] = {0u, 0u}, hi[2] = {0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int v = (int)(int16_t)((e & 1) ? (wv[e >> 1] >> 16) : (wv[e >> 1] & 0xffffu));
        const int l = limb_lo(v);
        lo[e >> 2] |= (uint32_t)(l & 255) << (8 * (e & 3));
        hi[e >> 2] |= (uint32_t)(((v - l) >> 8) & 255) << (8 * (e & 3));
      }
      *reinterpret_cast<uint2*>(&tb[0][c * kTbPitch + j]) = make_uint2(lo[0], lo[1]);
      *reinterpret_cast<uint2*>(&tb[1][c * kTbPitch + j]) = make_uint2(hi[0], hi[1]);
    }
  }
  // Channel tables (read per tile by the lanes that hold channels 16 ct + 4 kg + i).
  if (tid < kD) {
    tab_is[tid] = hp->inv_s[tid];
    tab_o[tid] = hp->bit_off[tid];
  }
  if (tid < kD / 4) tab_b[tid] = reinterpret_cast<const uint32_t*>(hp->bits)[tid];
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
    for (int i = tid; i < kTile * kRecWords; i += kEncThreads) (&rec[0][0])[i] = 0u;
    // (1) The token's fixed-point shift (max over its 128 elements: 4 lanes).
    float m = 0.f;
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int e = 0; e < 16; ++e) m = fmaxf(m, fabsf(xv[kc][e]));
    const int shift = token_shift(enc_cross_row_max(m));
    // (2) The limbs of X = rint(x 2^shift) as A operands (byte e: element e).
    ev4i A0[2], A1[2];
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        // The low limb's byte is X mod 256 and the high limb is floor((X + 128) / 256);
        // byte e of each dword gathered with two byte permutes.
        uint32_t X[4], H[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          X[e] = (uint32_t)(int)rintf(ldexpf(xv[kc][4 * q + e], shift));
          H[e] = (uint32_t)(((int)X[e] + 128) >> 8);
        }
        // v_perm_b32(a, b, sel): byte k of the result is byte sel_k of the pair {a: 4..7, b: 0..3}
        const uint32_t lo01 = __builtin_amdgcn_perm(X[1], X[0], 0x0c0c0400u);
        const uint32_t lo23 = __builtin_amdgcn_perm(X[3], X[2], 0x04000c0cu);
        const uint32_t hi01 = __builtin_amdgcn_perm(H[1], H[0], 0x0c0c0400u);
        const uint32_t hi23 = __builtin_amdgcn_perm(H[3], H[2], 0x04000c0cu);
        A0[kc][q] = (int)(lo01 | lo23);
        A1[kc][q] = (int)(hi01 | hi23);
      }
    fetch(tile + gridDim.x);                      // the next tile's elements, in flight
    if (tile == first + blockIdx.x) __syncthreads();   // (the limb and channel tables)
    // (3) Four channel tiles at a time: the three limb sums, then r_c for channels
    //     16 ct + 4 kg + i of this lane's token.
    float r[8][4], am = 0.f;
#pragma unroll
    for (int c4 = 0; c4 < 8; c4 += 4) {
      ev4i s11[4], s10[4], s00[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int ct = c4 + u;
        s11[u] = s10[u] = s00[u] = (ev4i){0, 0, 0, 0};
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
          const int o = (16 * ct + n) * kTbPitch + 64 * kc + 16 * kg;
          const ev4i b0 = *reinterpret_cast<const ev4i*>(&tb[0][o]);
          const ev4i b1 = *reinterpret_cast<const ev4i*>(&tb[1][o]);
          s11[u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b1, A1[kc], s11[u], 0, 0, 0);
          s10[u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b0, A1[kc], s10[u], 0, 0, 0);
          s10[u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b1, A0[kc], s10[u], 0, 0, 0);
          s00[u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b0, A0[kc], s00[u], 0, 0, 0);
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int ct = c4 + u, c0 = 16 * ct + 4 * kg;
        const float4 is4 = *reinterpret_cast<const float4*>(&tab_is[c0]);
        const float isv[4] = {is4.x, is4.y, is4.z, is4.w};
        const uint32_t bw = tab_b[c0 >> 2];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // 65536 S11 + (256 S10 + S00), exact in fp64 (< 2^37), then the one rounding
          // of the canonical result.
          const int low = s10[u][i] * 256 + s00[u][i];
          const double h = fma((double)s11[u][i], 65536.0, (double)low);
          r[ct][i] = (float)ldexp(h, -(shift + kTFrac)) * isv[i];
          am = fmaxf(am, fabsf(r[ct][i]));          // (r = 0 on dropped channels)
        }
      }
      // (one half's accumulators at a time)
      __builtin_amdgcn_sched_barrier(0);
    }
    // (4) The token's scale (its 128 channels: 4 lanes), its codes and record: channels
    //     16 ct + 4 kg .. + 3 are consecutive in the record, one bit field of <= 32 bits.
    const __half a16 = token_alpha(enc_cross_row_max(am));
    const float inv_a = inverse_alpha(a16);
    if (valid) {
#pragma unroll
      for (int ct = 0; ct < 8; ++ct) {
        const int c0 = 16 * ct + 4 * kg;
        const uint32_t bw = tab_b[c0 >> 2];
        uint32_t field = 0u;
        int width = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int b = (int)((bw >> (8 * i)) & 255u);
          const uint32_t u = quantize_code_nb(r[ct][i], inv_a, b);
          field |= u << width;
          width += b;
        }
        const int off = tab_o[c0];
        if (width > 0) {
          atomicOr(&rec[tl][off >> 5], field << (off & 31));
          if ((off & 31) + width > 32) atomicOr(&rec[tl][(off >> 5) + 1], field >> (32 - (off & 31)));
        }
      }
      if (kg == 0) alpha[(int64_t)head * cap + tile_base + tl] = __half_as_ushort(a16);
    }
    __syncthreads();
    const int lo = (int)(t_begin - tile_base), hi = (int)(t_end - tile_base);
    if (layout == AATC_LAYOUT_RECORDS) {
      uint32_t* out = reinterpret_cast<uint32_t*>(codes) + ((int64_t)head * cap + tile_base) * rwords;
      for (int i = lo * rwords + tid; i < hi * rwords; i += kEncThreads)
        out[i] = rec[i / rwords][i % rwords];
    } else {
      // Record word w of the tile's tokens -> tile words 64 w .. 64 w + 63.  Lane p holds
      // the word of the token at position p; a 32 x 32 bit transpose within each half of
      // the wave (five butterfly stages on lane-xor swizzles) leaves lane 32 W + b with bit
      // 32 w + b over the positions of half W: tile word 2 (32 w + b) + W.
      uint32_t* out = reinterpret_cast<uint32_t*>(codes) +
                      ((int64_t)head * (cap / kTile) + tile) * (16 * rbytes);
      const uint64_t vmask = __builtin_amdgcn_ballot_w64(ptok >= lo && ptok < hi);
      const uint32_t keep = ~(uint32_t)((lane >> 5) ? (vmask >> 32) : vmask);
      for (int w = wave; w < rwords; w += kEncThreads / 64) {
        uint32_t x = rec[ptok][w];
        x = bit_transpose_stage<16, 0x0000ffffu>(x, lane);
        x = bit_transpose_stage<8, 0x00ff00ffu>(x, lane);
        x = bit_transpose_stage<4, 0x0f0f0f0fu>(x, lane);
        x = bit_transpose_stage<2, 0x33333333u>(x, lane);
        x = bit_transpose_stage<1, 0x55555555u>(x, lane);
        uint32_t* o = out + 64 * w + 2 * (lane & 31) + (lane >> 5);
        *o = keep ? ((*o & keep) | (x & ~keep)) : x;
      }
    }
    __syncthreads();
  }
}

// One workgroup per (token, KV head), for appends of a few tokens: the same canonical
// arithmetic as encode_exact_kernel, with the exact dot product split over two halves
// of j and the transposed fixed-point transform read straight from global memory.
// Tile bits are set and cleared with device atomics, so tokens that share a tile word
// may be encoded by different workgroups.
// With `seq_len` set, block x is a sequence instead: it encodes token seq_len[b] - 1 of
// sequence b (nothing for an empty sequence) into caches `codes_bstride` bytes and
// `alpha_bstride` scales apart.
__global__ __launch_bounds__(kEncThreads) void encode_token_kernel(
    const void* __restrict__ params, const void* __restrict__ x, int dtype, int64_t x_stride,
    int layout, uint8_t* __restrict__ codes, uint16_t* __restrict__ alpha, int64_t cap,
    int64_t pos, const int32_t* __restrict__ seq_len, int64_t codes_bstride,
    int64_t alpha_bstride) {
  __shared__ __align__(16) int xs[kD];
  __shared__ long long part[kD];
  __shared__ uint32_t rec[kRecWords];
  __shared__ float red_x[4], red_a[4];

  int64_t t = pos + blockIdx.x;
  if (seq_len) {
    t = min<int64_t>(max(seq_len[blockIdx.x], 0), cap) - 1;
    if (t < 0) return;
    codes += blockIdx.x * codes_bstride;
    alpha += blockIdx.x * alpha_bstride;
  }
  const int head = blockIdx.y;
  const HeadParams* hp = head_params(params, head);
  const int tid = threadIdx.x, c = tid & (kD - 1), half = tid >> 7, wave = tid >> 6;
  // Loads: row c of the transposed transform, columns 64 half .. 64 half + 63; the
  // channel tables; the token.
  uint4 tq[8];
  const uint4* trow = reinterpret_cast<const uint4*>(hp->Tqt + c * kD + 64 * half);
#pragma unroll
  for (int k = 0; k < 8; ++k) tq[k] = trow[k];
  const int b = hp->bits[c], off = hp->bit_off[c];
  const float inv_s = hp->inv_s[c];
  const int rbytes = hp->record_bytes;
  const float xv = (tid < kD) ? load_elem(x, dtype, (int64_t)blockIdx.x * x_stride +
                                                        (int64_t)head * kD + tid)
                              : 0.f;
  if (tid < kRecWords) rec[tid] = 0u;
  // Per-token fixed-point scale: max |x_j| goes to [2^13, 2^14).
  float m = wave_max(fabsf(xv));
  if ((tid & 63) == 0) red_x[wave] = m;
  __syncthreads();
  m = fmaxf(red_x[0], red_x[1]);
  const int shift = token_shift(m);
  if (tid < kD) xs[tid] = (int)rintf(ldexpf(xv, shift));
  __syncthreads();
  // Exact integer transform h_c = sum_j X_j Tq_jc.
  long long acc = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int4 x0 = reinterpret_cast<const int4*>(xs + 64 * half + 8 * k)[0];
    const int4 x1 = reinterpret_cast<const int4*>(xs + 64 * half + 8 * k)[1];
    const int xv8[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
    const uint32_t tw[4] = {tq[k].x, tq[k].y, tq[k].z, tq[k].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc += (long long)xv8[2 * i] * (long long)(int16_t)(tw[i] & 0xffffu);
      acc += (long long)xv8[2 * i + 1] * (long long)(int16_t)(tw[i] >> 16);
    }
  }
  if (half) part[c] = acc;
  __syncthreads();
  float r = 0.f;
  if (!half) {
    acc += part[c];
    r = fixed_point_result(acc, shift) * inv_s;
  }
  float a = wave_max((!half && b > 0) ? fabsf(r) : 0.f);
  if ((tid & 63) == 0) red_a[wave] = a;
  __syncthreads();
  a = fmaxf(red_a[0], red_a[1]);
  const __half a16 = token_alpha(a);
  const float inv_a = inverse_alpha(a16);
  if (!half && b > 0) {
    const uint32_t u = quantize_code(r, inv_a, b);
    atomicOr(&rec[off >> 5], u << (off & 31));
    if ((off & 31) + b > 32) atomicOr(&rec[(off >> 5) + 1], u >> (32 - (off & 31)));
  }
  if (tid == 0) alpha[(int64_t)head * cap + t] = __half_as_ushort(a16);
  __syncthreads();

  if (layout == AATC_LAYOUT_RECORDS) {
    uint32_t* out = reinterpret_cast<uint32_t*>(codes + ((int64_t)head * cap + t) * rbytes);
    for (int i = tid; i < rbytes / 4; i += kEncThreads) out[i] = rec[i];
  } else {
    const int p = (int)(t % kTile);
    const uint32_t bit = 1u << tile_bit(p);
    uint32_t* tw = reinterpret_cast<uint32_t*>(codes) +
                   ((int64_t)head * (cap / kTile) + t / kTile) * (16 * rbytes) + tile_word(p);
    for (int v = tid; v < 8 * rbytes; v += kEncThreads) {
      if ((rec[v >> 5] >> (v & 31)) & 1u)
        __hip_atomic_fetch_or(tw + 2 * v, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      else
        __hip_atomic_fetch_and(tw + 2 * v, ~bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

}  // namespace

aatc_status launch_encode(const void* params, int n_heads, const void* x, aatc_dtype x_dtype,
                          int64_t n_tok, int64_t x_tok_stride, aatc_layout layout,
                          void* codes, uint16_t* alpha, int64_t cap, int64_t pos,
                          void* stream) {
  if (n_tok <= kSmallBatch) {
    hipLaunchKernelGGL(encode_token_kernel, dim3((unsigned)n_tok, (unsigned)n_heads),
                       dim3(kEncThreads), 0, (hipStream_t)stream, params, x, (int)x_dtype,
                       x_tok_stride, (int)layout, static_cast<uint8_t*>(codes), alpha, cap, pos,
                       nullptr, (int64_t)0, (int64_t)0);
    return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
  }
  const int64_t first = pos / kTile, last = (pos + n_tok - 1) / kTile;
  const int64_t n_tiles = last - first + 1;
  const size_t esize = x_dtype == AATC_BF16 ? 2 : 4;
  const bool aligned = (reinterpret_cast<uintptr_t>(x) % 16 == 0) &&
                       ((size_t)x_tok_stride * esize) % 16 == 0;
  if (aligned) {
    // A grid-stride loop of at most 96 workgroups per KV head (each builds the head's limb
    // tables once).
    dim3 grid((unsigned)std::min<int64_t>(n_tiles, 96), (unsigned)n_heads);
    if (x_dtype == AATC_BF16)
      hipLaunchKernelGGL(encode_mfma_kernel<true>, grid, dim3(kEncThreads), 0,
                         (hipStream_t)stream, params, x, n_tok, x_tok_stride, (int)layout,
                         static_cast<uint8_t*>(codes), alpha, cap, pos);
    else
      hipLaunchKernelGGL(encode_mfma_kernel<false>, grid, dim3(kEncThreads), 0,
                         (hipStream_t)stream, params, x, n_tok, x_tok_stride, (int)layout,
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
  hipLaunchKernelGGL(encode_token_kernel, dim3((unsigned)batch, (unsigned)n_heads),
                     dim3(kEncThreads), 0, (hipStream_t)stream, params, x, (int)x_dtype,
                     (int64_t)n_heads * kD, (int)layout, static_cast<uint8_t*>(codes), alpha,
                     cap, (int64_t)0, seq_len, (int64_t)n_heads * cap * record_bytes,
                     (int64_t)n_heads * cap);
  return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
}

}  // namespace aatc
