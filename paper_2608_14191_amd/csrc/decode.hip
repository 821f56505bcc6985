// AATC decode attention on gfx950 (Algorithm 1, inference part, evaluated in the
// transformed domain of App. B: q~ = T_K^T q; the inverse transform T_V is applied once
// to each output).
//
// Grid: one workgroup per (sequence, KV head, token split).  Each workgroup scores its
// split's tokens for the G query heads of its KV head, runs a split-local softmax and
// accumulates the value codes into a partial (m, l, o~) in the workspace.  The last
// workgroup of each (sequence, KV head) to finish merges the partials and applies T_V.
//
// Two kernels share that structure:
//  * decode_mfma_kernel: G <= 8 and records of at most 64 bytes (budgets <= 512 bits);
//    both contractions run on int8 MFMA over the bits of the packed codes;
//  * decode_split_kernel: any G <= 16 and budget; plain VALU.
//
// Codes are b-bit two's complement patterns, code = sum_{k < b-1} 2^k bit_k -
// 2^(b-1) bit_(b-1): every record bit is a virtual channel whose weight is its
// channel's weight times +-2^k, and sums over bits need no offset term.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>

#include "encode_core.h"
#include "launch.h"
#include "params.h"
#include "workspace.h"

namespace aatc {
namespace {

constexpr int kThreads = 256;                    // generic kernel: four waves
constexpr int kSplit = 512;                      // tokens per workgroup, generic kernel
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kMaxNH = 8;                        // head slots of the MFMA kernel
constexpr int kRsrcWord3 = 0x00020000;           // raw buffer descriptor word 3 (gfx950)
constexpr int kCoherent = 16;                    // cache policy sc1: device-coherent access
constexpr int kMergeU = 8;                       // split partials in flight per merging thread

typedef int v4i __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(1))) uint32_t* gdword;   // global-memory dword
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v2f __attribute__((ext_vector_type(2)));

struct DecodeArgs {
  const void* params_k;
  const void* params_v;
  const void* q;
  uint8_t* k_codes;               // written only by the fused append
  uint16_t* k_alpha;
  uint8_t* v_codes;
  uint16_t* v_alpha;
  const int32_t* seq_len;
  const void* x_k;                // fused append: new token [batch][n_kv_heads][d], or null
  const void* x_v;
  int x_dtype;
  float* out;
  unsigned* counters;
  Partial* partials;
  float* append_r;                // fused append: [rows][kAppStride] coefficients, bounds
  const Partial* seg;             // full-precision segment partials [rows][G], or null
  int64_t cap;
  int n_q_heads, n_kv_heads, G, q_dtype;
  int n_splits, n_blocks;         // splits per (sequence, KV head); rows x splits
  int rk, rv;                     // record bytes
  float scale_log2e;
  int off_v, off_ak, off_av, off_ql, off_pb, off_ob, ob_stride, off_es;   // dynamic LDS layout
};

__device__ inline float load_q(const void* q, int dtype, int64_t idx) {
  if (dtype == AATC_BF16) {
    uint32_t b = static_cast<const uint16_t*>(q)[idx];
    return __uint_as_float(b << 16);
  }
  return static_cast<const float*>(q)[idx];
}

__device__ inline float half_bits_to_float(uint16_t h) {
  return __half2float(__ushort_as_half(h));
}

// Buffer descriptors: loads past `bytes` return 0, stores past it are dropped.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           kRsrcWord3);
}
template <int AUX>
__device__ inline v4i buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return (v4i)__builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, AUX);
}
__device__ inline v2f buf_load8_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return (v2f)__builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, kCoherent);
}
__device__ inline v4f buf_load16_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return (v4f)__builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kCoherent);
}
__device__ inline void buf_store16_coherent(v4f v, __amdgpu_buffer_rsrc_t r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b128((v4i)v, r, (int)off, 0, kCoherent);
}
__device__ inline void buf_store4_coherent(float v, __amdgpu_buffer_rsrc_t r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_int(v), r, (int)off, 0, kCoherent);
}

// Device-coherent scalar store: a relaxed agent-scope atomic is performed where every
// compute unit of the device sees it (it bypasses the per-XCD caches).
__device__ inline void st_dev(float* p, float v) {
  __hip_atomic_store(reinterpret_cast<unsigned*>(p), __float_as_uint(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Wave-wide maximum and sum without LDS round trips: quad butterflies and row rotations
// (DPP), then the four row results read as scalars.
template <int CTRL>
__device__ inline float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
// Lane l and lane l ^ 16 (l ^ 32) combined without LDS: the row swaps of gfx950 return
// both halves of the exchange, so op(r[0], r[1]) is op(v, partner) in every lane.
__device__ inline float xor16_max(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float xor32_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float xor16_sum(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ inline float xor32_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ inline int xor16_sum(int v) {
  const auto r = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v, false, false);
  return (int)r[0] + (int)r[1];
}
__device__ inline int xor32_sum(int v) {
  const auto r = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
  return (int)r[0] + (int)r[1];
}

// Wave-wide maximum and sum without LDS round trips: quad butterflies and row rotations
// (DPP), then the row swaps; every lane ends with the result.
__device__ inline float wave_max_dpp(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));            // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp_f<0x4E>(v));            // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp_f<0x124>(v));           // row_ror:4
  v = fmaxf(v, dpp_f<0x128>(v));           // row_ror:8
  return xor32_max(xor16_max(v));
}
__device__ inline float wave_sum_dpp(float v) {
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  v += dpp_f<0x124>(v);
  v += dpp_f<0x128>(v);
  return xor32_sum(xor16_sum(v));
}
// Maximum and sum over each row of 16 lanes (every lane of the row ends with it).
__device__ inline float row16_max(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));
  v = fmaxf(v, dpp_f<0x4E>(v));
  v = fmaxf(v, dpp_f<0x124>(v));
  return fmaxf(v, dpp_f<0x128>(v));
}
__device__ inline float row16_sum(float v) {
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  v += dpp_f<0x124>(v);
  return v + dpp_f<0x128>(v);
}
template <int CTRL>
__device__ inline int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
__device__ inline int wave_sum_i32(int v) {         // exact while the sum fits 32 bits
  v += dpp_i<0xB1>(v);
  v += dpp_i<0x4E>(v);
  v += dpp_i<0x124>(v);
  v += dpp_i<0x128>(v);
  return xor32_sum(xor16_sum(v));
}
// One step of a reduce-scatter across lanes l and l ^ BIT (BIT = 8, 16 or 32): the lane
// with that bit clear keeps the sums of the lower half of the C values, the other the
// upper half.  (The row swaps return the pair ordered by lane: lower lane's value first.)
template <int C, int BIT>
__device__ inline void reduce_scatter_step(const float (&in)[C], float (&out)[C / 2]) {
  const bool up = (threadIdx.x & BIT) != 0;
#pragma unroll
  for (int i = 0; i < C / 2; ++i) {
    const float k = up ? in[C / 2 + i] : in[i];
    const float s = up ? in[i] : in[C / 2 + i];
    float p;
    if constexpr (BIT == 32) {
      const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(s), __float_as_uint(s), false, false);
      p = __uint_as_float(up ? r[0] : r[1]);
    } else if constexpr (BIT == 16) {
      const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(s), __float_as_uint(s), false, false);
      p = __uint_as_float(up ? r[0] : r[1]);
    } else {
      static_assert(BIT == 8, "bits 3, 4, 5");
      p = dpp_f<0x128>(s);                     // row_ror:8 within rows of 16: lane l ^ 8
    }
    out[i] = k + p;
  }
}

// N independent reductions taken step by step together, so that each step's exchanges
// overlap (a single chain waits on every step).
template <int N>
__device__ inline void wave_max_n(float (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = fmaxf(v[i], dpp_f<0xB1>(v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = fmaxf(v[i], dpp_f<0x4E>(v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = fmaxf(v[i], dpp_f<0x124>(v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = fmaxf(v[i], dpp_f<0x128>(v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = xor16_max(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = xor32_max(v[i]);
}
template <int N>
__device__ inline void wave_sum_n(float (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] += dpp_f<0xB1>(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] += dpp_f<0x4E>(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] += dpp_f<0x124>(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] += dpp_f<0x128>(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = xor16_sum(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = xor32_sum(v[i]);
}
template <int N>
__device__ inline void wave_sum_i32_n(int (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] += dpp_i<0xB1>(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] += dpp_i<0x4E>(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] += dpp_i<0x124>(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] += dpp_i<0x128>(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = xor16_sum(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = xor32_sum(v[i]);
}

__device__ inline float block_reduce(float v, bool is_max, float* scratch) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    float w = __shfl_xor(v, o, 64);
    v = is_max ? fmaxf(v, w) : v + w;
  }
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) scratch[wave] = v;
  __syncthreads();
  float r = scratch[0];
  for (int i = 1; i < kThreads / 64; ++i) r = is_max ? fmaxf(r, scratch[i]) : r + scratch[i];
  return r;
}

// Lane-quad data movement (lanes 4k .. 4k + 3): xor 1 and xor 2 within the quad.
__device__ inline uint32_t quad_xor1(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
}
__device__ inline uint32_t quad_xor2(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);
}
__device__ inline float quad_xor1(float v) { return __uint_as_float(quad_xor1(__float_as_uint(v))); }
__device__ inline float quad_xor2(float v) { return __uint_as_float(quad_xor2(__float_as_uint(v))); }

// Four balanced int8 limbs of a 32-bit value |x| < 2^30, packed in one dword (limb L in
// byte L, two's complement): x = sum_L limb_L 256^L.
__device__ inline uint32_t pack_limbs(int x) {
  return ((uint32_t)x + 0x80808080u) ^ 0x80808080u;
}

// s_waitcnt immediates (gfx9 layout: vmcnt [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
constexpr int kWaitVm0 = (0x7 << 4) | (0xF << 8);            // vmcnt(0) only
constexpr int kWaitLgkm0 = 0xF | (0x7 << 4) | (0x3 << 14);    // lgkmcnt(0) only

// s_barrier alone, with no wait on outstanding memory operations (unlike __syncthreads(),
// whose fence waits for every load of the wave, LDS transfers included).  The memory
// clobber keeps the compiler's memory accesses on their side; the scheduling barriers
// keep other instructions (and the waits they would bring) there too.
__device__ inline void plain_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// s_waitcnt vmcnt(n) for a wave-uniform n known only at run time (0 <= n < 64).
__device__ inline void wait_vmcnt(int n) {
#define AATC_VMW(k)                                                                         \
  case k:                                                                                  \
    __builtin_amdgcn_s_waitcnt(((k) & 0xF) | (0x7 << 4) | (0xF << 8) | (((k) >> 4) << 14)); \
    break;
#define AATC_VMW4(k) AATC_VMW(k) AATC_VMW(k + 1) AATC_VMW(k + 2) AATC_VMW(k + 3)
  switch (__builtin_amdgcn_readfirstlane(n)) {
    AATC_VMW4(0) AATC_VMW4(4) AATC_VMW4(8) AATC_VMW4(12) AATC_VMW4(16) AATC_VMW4(20)
    AATC_VMW4(24) AATC_VMW4(28) AATC_VMW4(32) AATC_VMW4(36) AATC_VMW4(40) AATC_VMW4(44)
    AATC_VMW4(48) AATC_VMW4(52) AATC_VMW4(56) AATC_VMW4(60)
    default: __builtin_amdgcn_s_waitcnt(0); break;
  }
#undef AATC_VMW4
#undef AATC_VMW
}

__device__ inline v4i mfma_i8(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// Bytes of LDS the merge of an NTHR-thread workgroup needs (at the start of the dynamic
// LDS).
constexpr size_t merge_lds_bytes(int G, int NTHR) {
  return (size_t)(6 * NTHR + G * kD + (NTHR / 32) * G * kD) * sizeof(float);
}

// Inverse transform o = T_V o~ of G vectors with NTHR threads: thread (j4, cb) holds T_V
// rows 4 j4 .. 4 j4 + 3 at columns CW cb .. CW cb + CW - 1 (CW = 4096 / NTHR).
template <int NTHR>
struct TvBlock {
  static constexpr int NCB = NTHR / 32, CW = kD / NCB;
  v4f t[4][CW / 4];
  __device__ void load(const HeadParams* hv) {
    const int j4 = threadIdx.x & 31, cb = threadIdx.x >> 5;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
#pragma unroll
      for (int k = 0; k < CW / 4; ++k)
        t[jj][k] = reinterpret_cast<const v4f*>(hv->T)[(4 * j4 + jj) * (kD / 4) + (CW / 4) * cb + k];
  }
  // osum: LDS [G][kD] input; ored: LDS [NCB][G][kD] scratch.  Calls sink(h, j, o_hj) once
  // per output, after a barrier; the caller synchronizes before osum is reused.
  template <class Sink>
  __device__ void apply(const float* osum, float* ored, int G, Sink sink) const {
    const int tid = threadIdx.x, j4 = tid & 31, cb = tid >> 5;
    for (int h = 0; h < G; ++h) {
      const v4f* oh = reinterpret_cast<const v4f*>(osum + h * kD) + (CW / 4) * cb;
      v4f ov4[CW / 4];
#pragma unroll
      for (int k = 0; k < CW / 4; ++k) ov4[k] = oh[k];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        v4f p = t[jj][0] * ov4[0];
#pragma unroll
        for (int k = 1; k < CW / 4; ++k) p += t[jj][k] * ov4[k];
        ored[(cb * G + h) * kD + 4 * j4 + jj] = p.x + p.y + p.z + p.w;
      }
    }
    __syncthreads();
    for (int i = tid; i < G * kD; i += NTHR) {
      const int h = i / kD, j = i % kD;
      float acc = 0.f;
#pragma unroll
      for (int b = 0; b < NCB; ++b) acc += ored[(b * G + h) * kD + j];
      sink(h, j, acc);
    }
  }
};

// o = T_V o~ on the matrix cores in bf16 pairs: with T = Th + Tl and o~ = oh + ol (each
// term bf16, the second the first's remainder), T o~ = Th oh + Th ol + Tl oh up to
// |Tl ol| + rounding, about 2^-16 relative; the three products accumulate in fp32
// (v_mfma_f32_16x16x32_bf16).  Wave w computes output rows 16 w' .. + 15 (w' = w + NTHR /
// 64 p over the passes p) for up to 16 vectors: A = its 16-row block of T (the
// parameter block's operand-ordered copy), B column n = vector n.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// bf16 of x (round to nearest even) and of the remainder x - bf16(x).
__device__ inline void bf16_pair(float x, __bf16& hi, __bf16& lo) {
  hi = (__bf16)x;
  lo = (__bf16)(x - (float)hi);
}

template <int NTHR>
struct TvMfma {
  static constexpr int NPASS = 512 / NTHR;
  static_assert(NPASS * NTHR == 512, "256 or 512 threads");
  bf16x8 a[NPASS][4][2];                  // [pass][k-step][Th, Tl]
  __device__ void load(const HeadParams* hv) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) load_step(hv, kk);
  }
  // The operands of k-step kk only (the loads can be spread out).
  __device__ void load_step(const HeadParams* hv, int kk) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const bf16x8* tp = reinterpret_cast<const bf16x8*>(hv->Tm);
#pragma unroll
    for (int p = 0; p < NPASS; ++p)
#pragma unroll
      for (int t = 0; t < 2; ++t)
        a[p][kk][t] = tp[(((wave + (NTHR / 64) * p) * 4 + kk) * 2 + t) * 64 + lane];
  }
  // B operands in LDS: ob[t] (t = 0: oh, 1: ol) holds [k-step][lane] 16-byte units, lane
  // 16 g + n: vector n at elements 32 kk + 8 g .. + 7 (put() writes one element).
  __device__ static void put(__bf16* ob_hi, __bf16* ob_lo, int n, int c, float x) {
    const int i = ((c >> 5) * 64 + 16 * ((c >> 3) & 3) + n) * 8 + (c & 7);
    bf16_pair(x, ob_hi[i], ob_lo[i]);
  }
  // Calls sink(n, j0, o[j0 .. j0 + 3] of vector n) for n < G (the caller synchronizes
  // after the puts).
  template <class Sink>
  __device__ void apply(const __bf16* ob_hi, const __bf16* ob_lo, int G, Sink sink) const {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, n = lane & 15;
    const bf16x8* bh = reinterpret_cast<const bf16x8*>(ob_hi);
    const bf16x8* bl = reinterpret_cast<const bf16x8*>(ob_lo);
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
      v4f acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = acc0, acc2 = acc0;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const bf16x8 h8 = bh[kk * 64 + lane], l8 = bl[kk * 64 + lane];
        acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[p][kk][0], h8, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[p][kk][0], l8, acc1, 0, 0, 0);
        acc2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[p][kk][1], h8, acc2, 0, 0, 0);
      }
      if (n < G) sink(n, 16 * (wave + (NTHR / 64) * p) + 4 * (lane >> 4), acc0 + acc1 + acc2);
    }
  }
};

// Extra work of the merging workgroup (the fused append supplies one, below).
struct NoHook {
  __device__ void prefetch() {}
  __device__ void during_loads() {}
  __device__ void encode() {}
  __device__ void publish() {}
  __device__ void fold(int, int, float&, float&, v4f&) const {}
  __device__ void fold1(int, int, float&, float&, float&) const {}
  __device__ void finish() {}
};

// Called by every workgroup after it stored its partial with device-coherent stores.
// The last of a (sequence, KV head) to arrive merges the split partials.  The hook's
// loads go out ahead of the partials', its during_loads() (encode(), then the barrier of
// publish()) runs while they are in flight, fold() adds one more (score, value) term per output slot, finish() runs at the end.
template <int NTHR, bool TV, bool ONE_PASS = false, class Hook = NoHook>
__device__ __forceinline__ void merge_if_last(const void* params_v, int kvh, int64_t row, int G,
                                              int n_splits, const Partial* partials,
                                              unsigned* counters, float* out_rows, float* lds,
                                              Hook& hook) {
  constexpr int NCB = NTHR / 32;          // column blocks of the T_V product
  __shared__ unsigned last_s;
  const int tid = threadIdx.x;
  __builtin_amdgcn_s_waitcnt(0);          // this thread's partial stores have completed
  __syncthreads();
  // The arrival count goes out first; every workgroup then fetches T_V, which the merge
  // would need, under the count's round trip.
  unsigned prev = 0u;
  if (tid == 0)
    prev = __hip_atomic_fetch_add(&counters[row * kCtrStride], 1u, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT);
  const HeadParams* hv = head_params(params_v, kvh);
  TvBlock<NTHR> tv;
  if (TV) tv.load(hv);
  if (tid == 0) last_s = (prev == (unsigned)n_splits - 1u) ? 1u : 0u;
  __syncthreads();
  if (!last_s) return;
  hook.prefetch();
  __builtin_amdgcn_sched_barrier(0);
  float* cm = lds;                                         // [NTHR] group maxima
  float* cl = cm + NTHR;                                   // [NTHR] group sums
  v4f* cacc = reinterpret_cast<v4f*>(cl + NTHR);           // [NTHR]
  float* osum = reinterpret_cast<float*>(cacc + NTHR);     // [G][kD]
  float* ored = osum + G * kD;                             // [NCB][G][kD]
  const __amdgpu_buffer_rsrc_t prs =
      make_rsrc(partials + row * n_splits * G, (uint32_t)(n_splits * G * sizeof(Partial)));

  // (a) Online merge over the splits: slot (head, float4 column) per thread; groups of
  //     threads take interleaved splits and combine at the end.
  // (ONE_PASS: G kD / 4 <= NTHR, one slot per thread, no loop.)
  const int slots = G * (kD / 4);
  for (int base = 0; base < (ONE_PASS ? 1 : slots); base += NTHR) {
    const int width = min(slots - base, NTHR);
    const int ngroups = NTHR / width;
    const int slot = base + tid % width, grp = tid / width;
    const int h = slot >> 5, c4 = slot & 31;
    const bool active = grp < ngroups;
    float M = -INFINITY, Ls = 0.f;
    v4f acc = {0.f, 0.f, 0.f, 0.f};
    bool bad = false;
    v2f hd[kMergeU];
    v4f ov[kMergeU];
    auto issue = [&](int s0) {                     // past the last split the loads read 0
#pragma unroll
      for (int u = 0; u < kMergeU; ++u) {
        const uint32_t off = (uint32_t)(((s0 + u * ngroups) * G + h) * sizeof(Partial));
        hd[u] = buf_load8_coherent(prs, off);
        ov[u] = (v4f)__builtin_amdgcn_raw_buffer_load_b128(prs, (int)(off + 16 + 16 * c4), 0,
                                                          kCoherent);
      }
    };
    // Branch-free, so that every load of a batch is issued before the first wait (an
    // empty split has o~ = 0, and loads past the last split read 0).
    auto consume = [&](int s0) {
#pragma unroll
      for (int u = 0; u < kMergeU; ++u) {
        const float ms = (active && s0 + u * ngroups < n_splits) ? hd[u].x : -INFINITY;
        bad |= (ms != ms);
        const float mn = fmaxf(M, ms);
        const float sa = (mn == -INFINITY) ? 1.f : exp2f(M - mn);
        const float sb = (ms == -INFINITY) ? 0.f : exp2f(ms - mn);
        acc = acc * sa + ov[u] * sb;
        Ls = Ls * sa + hd[u].y * sb;
        M = mn;
      }
    };
    issue(grp);
    if (base == 0) hook.during_loads();
    consume(grp);
    for (int s0 = grp + kMergeU * ngroups; s0 < n_splits; s0 += kMergeU * ngroups) {
      issue(s0);
      consume(s0);
    }
    cm[tid] = bad ? NAN : M;
    cl[tid] = Ls;
    cacc[tid] = acc;
    __syncthreads();
    if (tid < width) {
      M = cm[tid];
      Ls = cl[tid];
      acc = cacc[tid];
      bad = M != M;
      for (int q = 1; q < ngroups; ++q) {
        const float ms = cm[q * width + tid];
        bad |= (ms != ms);
        if (ms > -INFINITY) {
          const float mn = fmaxf(M, ms);
          const float sa = exp2f(M - mn), sb = exp2f(ms - mn);
          acc = acc * sa + cacc[q * width + tid] * sb;
          Ls = Ls * sa + cl[q * width + tid] * sb;
          M = mn;
        }
      }
      hook.fold(h, c4, M, Ls, acc);
      const float inv_l = bad ? NAN : (Ls > 0.f ? 1.f / Ls : 0.f);
      reinterpret_cast<v4f*>(osum)[h * (kD / 4) + c4] = acc * inv_l;
    }
    __syncthreads();
  }
  // (b) o = T_V o~ (transformed-domain partials), or o~ itself.
  if constexpr (TV) {
    tv.apply(osum, ored, G, [&](int h, int j, float o) { out_rows[(int64_t)h * kD + j] = o; });
  } else {
    for (int i = tid; i < G * kD; i += NTHR) out_rows[i] = osum[i];
  }
  hook.finish();
  if (tid == 0) counters[row * kCtrStride] = 0u;
}

// The merge of the MFMA kernel.  The partials go in batches of SB splits.  For each head
// one of waves 2.. (the table waves) keeps the running maximum M and sum L, and per batch
// writes the rescale 2^(M_old - M) and the splits' weights 2^(m_s - M) to LDS; every
// thread loads the partial vectors of one (head, channel quad) unit for its group's SU
// splits of the batch (16-byte loads) and adds them up with those weights after the
// batch's barrier.  Waves 0 and 1 run the hook's encode while their loads are in flight
// (the first barrier also publishes it).  The NG group sums of a unit meet in LDS; then
// each output element (head h, channel c) takes its one more hook term and goes into the
// B operands of o = T_V o~.
// LDS: T_V B operands (8 KiB) | weights [2][NH][SB] | rescales [2][NH] | (M, L, bad) [NH]
// | group sums [NG][NU] (16 B each).  TV_HELD: the caller has loaded tv (every split does,
// during its value phase, so the merging one starts with T_V in registers); otherwise the
// merge loads it after the partials.
template <int NTHR, int NH>
struct WideMerge {
  static constexpr int NW = NTHR / 64;
  static constexpr int NU = NH * (kD / 4);            // (head, channel quad) units
  static constexpr int NG = NTHR / NU;                // split groups
  static constexpr int SU = 8;                        // splits per thread and batch
  static constexpr int SB = SU * NG;                  // splits per batch
  static constexpr int NTW = NW - 2;                  // table waves
  static constexpr int NHW = (NH + NTW - 1) / NTW;    // heads per table wave
  static constexpr int NP = (NH * kD + NTHR - 1) / NTHR;   // output elements per thread
  static_assert(NG >= 1 && NG * NU == NTHR && SB <= 64 && NTW >= 1, "thread mapping");
  static constexpr int kWt = 2 * 4 * 64 * 8 / 2;     // float offsets of the regions
  static constexpr int kSa = kWt + 2 * NH * SB;
  static constexpr int kFin = kSa + 2 * NH;
  static constexpr int kRed = (kFin + 4 * NH + 3) / 4 * 4;
  static constexpr int kFloats = kRed + 4 * NTHR;
};

template <int NTHR, int NH>
constexpr size_t wide_merge_lds_bytes() { return WideMerge<NTHR, NH>::kFloats * sizeof(float); }

template <int NTHR, int NH, bool TV_HELD, class Hook>
__device__ __forceinline__ void merge_if_last_wide(const void* params_v, int kvh, int64_t row,
                                                   int G, int n_splits, const Partial* partials,
                                                   unsigned* counters, float* out_rows,
                                                   float* lds, TvMfma<NTHR>& tv, Hook& hook) {
  using WM = WideMerge<NTHR, NH>;
  constexpr int SU = WM::SU, SB = WM::SB, NU = WM::NU, NTW = WM::NTW, NHW = WM::NHW;
  __shared__ unsigned last_s;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  __builtin_amdgcn_s_waitcnt(0);          // this thread's partial stores have completed
  __syncthreads();
  unsigned prev = 0u;
  if (tid == 0)
    prev = __hip_atomic_fetch_add(&counters[row * kCtrStride], 1u, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT);
  if (tid == 0) last_s = (prev == (unsigned)n_splits - 1u) ? 1u : 0u;
  __syncthreads();
  if (!last_s) return;
  hook.prefetch();
  __builtin_amdgcn_sched_barrier(0);
  __bf16* ob_hi = reinterpret_cast<__bf16*>(lds);
  __bf16* ob_lo = ob_hi + 4 * 64 * 8;
  float* wt = lds + WM::kWt;
  float* sat = lds + WM::kSa;
  v4f* fin = reinterpret_cast<v4f*>(lds + WM::kFin);
  v4f* red = reinterpret_cast<v4f*>(lds + WM::kRed);
  const __amdgpu_buffer_rsrc_t prs =
      make_rsrc(partials + row * n_splits * G, (uint32_t)(n_splits * G * sizeof(Partial)));
  // 32-bit offsets: the descriptor covers less than 2^31 bytes.
  const uint32_t step = (uint32_t)G * (uint32_t)sizeof(Partial);
  const int u = tid % NU, q = tid / NU, h = u / (kD / 4), c4 = u % (kD / 4);
  const bool unit_on = h < G;
  const bool table = wave >= 2;
  float tM[NHW], tL[NHW];
  bool tbad[NHW];
#pragma unroll
  for (int i = 0; i < NHW; ++i) {
    tM[i] = -INFINITY;
    tL[i] = 0.f;
    tbad[i] = false;
  }
  v2f thd[NHW];
  v4f ov[SU];
  v4f acc = {0.f, 0.f, 0.f, 0.f};
  // A batch's loads (past the last split or head they read 0): the table waves' (m, l)
  // first, then every thread's vectors.
  auto issue = [&](int s0) {
    if (table) {
#pragma unroll
      for (int i = 0; i < NHW; ++i) {
        const int h2 = wave - 2 + NTW * i;
        const bool on = (h2 < G) & (lane < SB) & (s0 + lane < n_splits);
        thd[i] = buf_load8_coherent(
            prs, on ? (uint32_t)(s0 + lane) * step + (uint32_t)h2 * (uint32_t)sizeof(Partial)
                    : 0x80000000u);
      }
    }
#pragma unroll
    for (int k = 0; k < SU; ++k) {
      const int sp = s0 + q * SU + k;
      const bool on = unit_on & (sp < n_splits);
      ov[k] = buf_load16_coherent(
          prs, on ? (uint32_t)sp * step + (uint32_t)h * (uint32_t)sizeof(Partial) + 16u +
                        16u * (uint32_t)c4
                  : 0x80000000u);
    }
  };
  // The table waves' part of a batch (NaN maxima mark records that did not match).
  auto tables = [&](int s0, int b) {
    if (!table) return;
#pragma unroll
    for (int i = 0; i < NHW; ++i) {
      const int h2 = wave - 2 + NTW * i;
      if (h2 >= G) continue;                         // (uniform over the wave)
      const bool in = (lane < SB) & (s0 + lane < n_splits);
      const float ms = in ? thd[i].x : -INFINITY;
      tbad[i] |= __builtin_amdgcn_ballot_w64(ms != ms) != 0;
      const float mn = fmaxf(tM[i], wave_max_dpp(ms));    // (NaN lanes are ignored)
      // (the hardware exp2: weights below 2^-126 of the largest flush to 0)
      const float sa = (mn == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(tM[i] - mn);
      const float w = (ms == -INFINITY || ms != ms) ? 0.f : __builtin_amdgcn_exp2f(ms - mn);
      tL[i] = tL[i] * sa + wave_sum_dpp(w * thd[i].y);
      tM[i] = mn;
      if (lane < SB) wt[((b & 1) * NH + h2) * SB + lane] = w;
      if (lane == 0) sat[(b & 1) * NH + h2] = sa;
    }
  };
  auto accumulate = [&](int b) {
    if (!unit_on) return;
    const v4f* wv = reinterpret_cast<const v4f*>(wt + ((b & 1) * NH + h) * SB + q * SU);
    const float sa = sat[(b & 1) * NH + h];
    float w[SU];
#pragma unroll
    for (int k = 0; k < SU / 4; ++k) {
      const v4f x = wv[k];
      w[4 * k] = x[0], w[4 * k + 1] = x[1], w[4 * k + 2] = x[2], w[4 * k + 3] = x[3];
    }
    v4f a0 = acc * sa, a1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < SU; k += 2) {
      a0 += w[k] * ov[k];
      a1 += w[k + 1] * ov[k + 1];
    }
    acc = a0 + a1;
  };
  issue(0);
  hook.encode();                          // waves 0 and 1, while the loads are in flight
  for (int s0 = 0, b = 0;; ++b) {
    tables(s0, b);
    __syncthreads();                      // the batch's weights (first: the hook's encode)
    accumulate(b);
    s0 += SB;
    if (s0 >= n_splits) break;
    issue(s0);
  }
  if (table && lane == 0) {
#pragma unroll
    for (int i = 0; i < NHW; ++i) {
      const int h2 = wave - 2 + NTW * i;
      if (h2 < G) fin[h2] = (v4f){tM[i], tL[i], tbad[i] ? 1.f : 0.f, 0.f};
    }
  }
  red[q * NU + u] = acc;
  __syncthreads();
#pragma unroll
  for (int p = 0; p < WM::NP; ++p) {
    const int slot = p * NTHR + tid, hh = slot / kD, c = slot % kD;
    if (hh < G) {
      float a = 0.f;
#pragma unroll
      for (int g = 0; g < WM::NG; ++g)
        a += reinterpret_cast<const float*>(red + g * NU + hh * (kD / 4))[c];
      const v4f f = fin[hh];
      float M = f[0], Ls = f[1];
      hook.fold1(hh, c, M, Ls, a);
      TvMfma<NTHR>::put(ob_hi, ob_lo, hh, c, f[2] != 0.f ? NAN : (Ls > 0.f ? a / Ls : 0.f));
    }
  }
  // T_V (its L2 lines touched by every split) after the partials: a compute unit serves its
  // loads in order, and T_V is needed last.
  if constexpr (!TV_HELD) tv.load(head_params(params_v, kvh));
  __syncthreads();
  // o = T_V o~ (the partials are in the transformed domain).
  tv.apply(ob_hi, ob_lo, G, [&](int hh, int j0, v4f o) {
    *reinterpret_cast<v4f*>(out_rows + (int64_t)hh * kD + j0) = o;
  });
  hook.finish();
  if (tid == 0) counters[row * kCtrStride] = 0u;
}

// ---------------------------------------------------------------------------------------
// Full-precision segment (the first tokens and the recent window kept at input precision,
// Sec. 6 and App. E): exact softmax attention of each query head over the segment's tokens
// in the original domain, one workgroup per (sequence, KV head), written as one more split
// partial in the transformed domain (o~ = T_V^T sum_t p_t v_t, with the log2-domain maximum
// and sum of its weights), which the merge of the compressed-cache splits folds in.
// ---------------------------------------------------------------------------------------
constexpr int kSegThreads = 256;
constexpr int kSegMax = 256;           // tokens of one segment

__global__ __launch_bounds__(kSegThreads) void segment_partial_kernel(
    const void* __restrict__ params_v, int n_q_heads, int n_kv_heads,
    const void* __restrict__ q, int q_dtype, const void* __restrict__ seg_k,
    const void* __restrict__ seg_v, int seg_dtype, const int32_t* __restrict__ seg_len,
    int seg_cap, float scale_log2e, Partial* __restrict__ seg_out) {
  __shared__ float qs[kMaxGroup][kD];
  __shared__ float z[kMaxGroup][kSegMax];
  __shared__ float orw[kMaxGroup][kD];
  __shared__ float red[kSegThreads / 64][kMaxGroup];
  __shared__ float mh[kMaxGroup], lh[kMaxGroup];
  const int row = blockIdx.x, kvh = row % n_kv_heads, seq = row / n_kv_heads;
  const int G = n_q_heads / n_kv_heads;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = min(max(seg_len[seq], 0), seg_cap);
  const int64_t tok0 = (int64_t)row * seg_cap;        // [batch][n_kv_heads][seg_cap][d]
  for (int i = tid; i < G * kD; i += kSegThreads)
    qs[i / kD][i % kD] =
        load_q(q, q_dtype, ((int64_t)seq * n_q_heads + kvh * G) * kD + i) * scale_log2e;
  __syncthreads();
  // Logits: thread t takes token t for every head.
  for (int t = tid; t < n; t += kSegThreads) {
    float acc[kMaxGroup];
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) acc[h] = 0.f;
    for (int j = 0; j < kD; ++j) {
      const float kv = load_elem(seg_k, seg_dtype, (tok0 + t) * kD + j);
#pragma unroll
      for (int h = 0; h < kMaxGroup; ++h)
        if (h < G) acc[h] = fmaf(qs[h][j], kv, acc[h]);
    }
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h)
      if (h < G) z[h][t] = acc[h];
  }
  __syncthreads();
  // Maximum and sum per head (the log2-domain weights 2^(z - m)).
  for (int h = 0; h < G; ++h) {
    float m = -INFINITY;
    for (int t = tid; t < n; t += kSegThreads) m = fmaxf(m, z[h][t]);
    m = wave_max_dpp(m);
    if (lane == 0) red[wave][h] = m;
  }
  __syncthreads();
  if (tid < G) {
    float m = red[0][tid];
    for (int w = 1; w < kSegThreads / 64; ++w) m = fmaxf(m, red[w][tid]);
    mh[tid] = m;
  }
  __syncthreads();
  for (int h = 0; h < G; ++h) {
    float l = 0.f;
    for (int t = tid; t < n; t += kSegThreads) {
      const float p = exp2f(z[h][t] - mh[h]);
      z[h][t] = p;
      l += p;
    }
    l = wave_sum_dpp(l);
    if (lane == 0) red[wave][h] = l;
  }
  __syncthreads();
  if (tid < G) {
    float l = 0.f;
    for (int w = 0; w < kSegThreads / 64; ++w) l += red[w][tid];
    lh[tid] = l;
  }
  // Value sums in the original domain: thread (half, j) over its half of the heads.
  {
    const int j = tid % kD, h0 = (tid / kD) * (kMaxGroup / 2);
    float acc[kMaxGroup / 2];
#pragma unroll
    for (int i = 0; i < kMaxGroup / 2; ++i) acc[i] = 0.f;
    for (int t = 0; t < n; ++t) {
      const float vv = load_elem(seg_v, seg_dtype, (tok0 + t) * kD + j);
#pragma unroll
      for (int i = 0; i < kMaxGroup / 2; ++i)
        if (h0 + i < G) acc[i] = fmaf(z[h0 + i][t], vv, acc[i]);
    }
#pragma unroll
    for (int i = 0; i < kMaxGroup / 2; ++i)
      if (h0 + i < G) orw[h0 + i][j] = acc[i];
  }
  __syncthreads();
  // Into the transformed domain of the merge: o~_c = sum_j T_V[j][c] o_j.
  const HeadParams* hv = head_params(params_v, kvh);
  Partial* out = seg_out + (int64_t)row * G;
  {
    const int c = tid % kD, h0 = (tid / kD) * (kMaxGroup / 2);
    float acc[kMaxGroup / 2];
#pragma unroll
    for (int i = 0; i < kMaxGroup / 2; ++i) acc[i] = 0.f;
    for (int j = 0; j < kD; ++j) {
      const float t = hv->T[j * kD + c];
#pragma unroll
      for (int i = 0; i < kMaxGroup / 2; ++i)
        if (h0 + i < G) acc[i] = fmaf(t, orw[h0 + i][j], acc[i]);
    }
#pragma unroll
    for (int i = 0; i < kMaxGroup / 2; ++i)
      if (h0 + i < G) out[h0 + i].o[c] = acc[i];
  }
  if (tid < G) {
    out[tid].m = n > 0 ? mh[tid] : -INFINITY;
    out[tid].l = n > 0 ? lh[tid] : 0.f;
  }
}

// The merging workgroup folds the segment's partial of its (sequence, KV head) into every
// output element (written by segment_partial_kernel, which ran before this launch).
struct SegHook {
  const Partial* seg;                  // this row's G partials
  __device__ void prefetch() {}
  __device__ void during_loads() {}
  __device__ void encode() {}
  __device__ void publish() {}
  __device__ void fold1(int h, int c, float& M, float& Ls, float& acc) const {
    const float ms = seg[h].m;
    if (ms == -INFINITY) return;
    const float mn = fmaxf(M, ms);
    const float sa = exp2f(M - mn), sb = exp2f(ms - mn);
    acc = acc * sa + seg[h].o[c] * sb;
    Ls = Ls * sa + seg[h].l * sb;
    M = mn;
  }
  __device__ void fold(int h, int c4, float& M, float& Ls, v4f& acc) const {
    const float ms = seg[h].m;
    if (ms == -INFINITY) return;
    const float mn = fmaxf(M, ms);
    const float sa = exp2f(M - mn), sb = exp2f(ms - mn);
    acc = acc * sa + reinterpret_cast<const v4f*>(seg[h].o)[c4] * sb;
    Ls = Ls * sa + seg[h].l * sb;
    M = mn;
  }
  __device__ void finish() {}
};

// ---------------------------------------------------------------------------------------
// Generic VALU kernel (any G <= 16, any budget).
// ---------------------------------------------------------------------------------------
// Fused append.  The splits stop short of the new token (position len - 1) and share its
// encode (exactly the encode kernels' arithmetic): split s computes the transformed
// coefficients r_c = h_c / s_c of the dot products d = s + n_splits (w + 8 i) of the
// 2 x 128 (key channels, then value channels), one per wave, and stores them in the
// workspace.  The merging workgroup loads the 256 coefficients ahead of the partials and,
// while those are in flight, takes the token scales, quantizes, and forms the token's score
// z = alpha^K sum_c Q_c 2^(1 - b_c) code_c per head (Q_c: the key phase's channel weights)
// and transformed value v~_c = alpha^V s_c 2^(1 - b_c) code_c; it folds them into the
// merge as one more term and writes the codes into both caches.  Every split has been read
// when the last one arrives, so nothing else touches the new slot.
// ---------------------------------------------------------------------------------------
struct AppendScratch {                 // LDS region of its own
  uint32_t erec[2][kMaxBudget / 32];   // key record, value record
  float vnew[kD];                      // transformed value of the token
  float znew[16];                      // the token's log2-domain score per head
  uint32_t ea16[2];                    // fp16 scales
};

// r = h~ / s of F transformed coefficients of the appended token (the encode kernels'
// arithmetic, reductions interleaved), from this lane's two elements of the token (raw
// dwords: bf16 halves or fp32) and of the coefficient's column of the integer transform:
// X_j = rint(x_j 2^S) with max |X| in [2^21, 2^22), H = sum_j X_j Tq_jc exact (each lane's
// two products below 2^45, the wave sums taken as 24-bit halves in int32), h~ =
// fl32(H 2^-(S+22)).  eh = E 2^-S (1 + 2^-16), E = sum_j |x_j 2^S - X_j|, bounds |h - h~|
// for the exact h (eh = 0: h~ is exact).
template <int F>
__device__ inline void append_coefficients(const uint32_t (&x)[F][2], const int (&t)[F][2],
                                           int x_dtype, const float (&inv_s)[F], float (&out)[F],
                                           float (&eh)[F]) {
  const int lane = threadIdx.x & 63;
  const bool bf = x_dtype == AATC_BF16;
  float xa[F], xb[F], m[F];
#pragma unroll
  for (int f = 0; f < F; ++f) {
    xa[f] = bf ? __uint_as_float(((lane & 1) ? (x[f][0] >> 16) : (x[f][0] & 0xffffu)) << 16)
               : __uint_as_float(x[f][0]);
    xb[f] = bf ? __uint_as_float(((lane & 1) ? (x[f][1] >> 16) : (x[f][1] & 0xffffu)) << 16)
               : __uint_as_float(x[f][1]);
    m[f] = fmaxf(fabsf(xa[f]), fabsf(xb[f]));
  }
  wave_max_n(m);
  int shift[F], hl[2 * F];
  float E[F];
#pragma unroll
  for (int f = 0; f < F; ++f) {
    shift[f] = token_shift(m[f]);
    const float va = ldexpf(xa[f], shift[f]), vb = ldexpf(xb[f], shift[f]);
    const float ra = rintf(va), rb = rintf(vb);
    E[f] = fabsf(va - ra) + fabsf(vb - rb);
    const long long p = (long long)(int)ra * t[f][0] + (long long)(int)rb * t[f][1];
    hl[2 * f] = (int)(p >> 24);
    hl[2 * f + 1] = (int)(p & 0xffffff);
  }
  wave_sum_i32_n(hl);
  wave_sum_n(E);
#pragma unroll
  for (int f = 0; f < F; ++f) {
    const double H = fma((double)hl[2 * f], 16777216.0, (double)hl[2 * f + 1]);
    out[f] = integer_result(H, shift[f]) * inv_s[f];
    eh[f] = ldexpf(E[f] * (1.f + 0x1p-16f), -shift[f]);
  }
}

template <int NTHR, int NH>
struct AppendHook {
  static_assert(NTHR >= 2 * kD && NH <= 16, "thread mapping");
  uint8_t* k_codes;
  uint16_t* k_alpha;
  uint8_t* v_codes;
  uint16_t* v_alpha;
  const float* coeff;                  // this row's coefficients and bounds (workspace)
  const HeadParams* ehp[2];            // key and value parameters of this KV head
  const void* xrow[2];                 // the new key and value token of this row
  int x_dtype;
  int64_t row, cap;
  int len, G, rk, rv;
  bool on;                             // the sequence has a token to append
  // Wave 0 encodes the key token, wave 1 the value token, lane l channels l and l + 64:
  int e_b[2], e_off[2];                // their widths and first record bits
  bool e_mr;                           // the wave's tensor uses the midrise reading
  float e_s[2];                        // their scales s_c (value token)
  float qk[2][NH];                     // Q_c of every head for them (key token)
  AppendScratch* sc;
  float r2[2];                         // their coefficients r_c = h_c / s_c
  float eh;                            // the wave's token: fixed-point error bound

  __device__ void prefetch() {
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const __amdgpu_buffer_rsrc_t rs =
        make_rsrc(coeff, (on && wave < 2) ? (uint32_t)(kAppStride * 4) : 0u);
#pragma unroll
    for (int i = 0; i < 2; ++i)
      r2[i] = __int_as_float(__builtin_amdgcn_raw_buffer_load_b32(
          rs, 4 * ((wave & 1) * kD + lane + 64 * i), 0, kCoherent));
    eh = __int_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, 4 * (2 * kD + (wave & 1)), 0,
                                                             kCoherent));
  }

  // The token's codes, scales, score per head and transformed value, each tensor by one
  // wave (wave reductions only); the barrier of publish() makes them visible.
  __device__ void during_loads() {
    encode();
    publish();
  }
  __device__ void publish() {
    if (on) __syncthreads();           // (uniform over the workgroup)
  }
  __device__ void encode() {
    if (!on) return;                   // uniform over the workgroup
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (wave < 2) {
      const int et = wave;
      if (lane < kMaxBudget / 32) sc->erec[et][lane] = 0u;
      // A token that is not exact in fixed point keeps its coefficients if the certificate
      // holds; otherwise (rarely) the exact routine recomputes them.
      const float ehw = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(eh)));
      const HeadParams* ep = et ? ehp[1] : ehp[0];
      if (ehw > 0.f && !wave_certify(ep, r2, ehw)) {
        const void* xr = et ? xrow[1] : xrow[0];
        float xl[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) xl[i] = load_elem(xr, x_dtype, lane + 64 * i);
        exact_r_wave<true>(ep, xl, xr, x_dtype, r2);
      }
      float m = 0.f;
#pragma unroll
      for (int i = 0; i < 2; ++i) m = fmaxf(m, e_b[i] > 0 ? fabsf(r2[i]) : 0.f);
      const __half a16 = token_alpha(wave_max_dpp(m));
      const float inv = inverse_alpha(a16);
      const bool midrise = e_mr;
      float code[2];                   // the level in steps: code, or code + 1/2 (midrise)
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        code[i] = 0.f;
        const int eb = e_b[i], eoff = e_off[i];
        if (eb > 0) {
          const uint32_t u = quantize_code(r2[i], inv, eb, midrise);
          atomicOr(&sc->erec[et][eoff >> 5], u << (eoff & 31));
          if ((eoff & 31) + eb > 32) atomicOr(&sc->erec[et][(eoff >> 5) + 1], u >> (32 - (eoff & 31)));
          code[i] = (float)((int)(u << (32 - eb)) >> (32 - eb)) + (midrise ? 0.5f : 0.f);
        }
      }
      const float af = __half2float(a16);
      if (et == 0) {
        float z[NH];
#pragma unroll
        for (int h = 0; h < NH; ++h) {
          z[h] = 0.f;
#pragma unroll
          for (int i = 0; i < 2; ++i)
            z[h] += e_b[i] ? qk[i][h] * ldexpf(code[i], 1 - e_b[i]) : 0.f;
        }
        wave_sum_n(z);
#pragma unroll
        for (int h = 0; h < NH; ++h)
          if (lane == 0) sc->znew[h] = af * z[h];
      } else {
#pragma unroll
        for (int i = 0; i < 2; ++i)
          sc->vnew[lane + 64 * i] = e_b[i] ? ldexpf(af * e_s[i] * code[i], 1 - e_b[i]) : 0.f;
      }
      if (lane == 0) sc->ea16[et] = __half_as_ushort(a16);
    }
  }
  // The token's log2-domain score for head h.
  __device__ float znew(int h) const { return sc->znew[h]; }

  __device__ void fold(int h, int c4, float& M, float& Ls, v4f& acc) const {
    if (!on) return;
    const float ms = znew(h);
    const v4f v = reinterpret_cast<const v4f*>(sc->vnew)[c4];
    const float mn = fmaxf(M, ms);
    const float sa = exp2f(M - mn), sb = exp2f(ms - mn);
    acc = acc * sa + v * sb;
    Ls = Ls * sa + sb;
    M = mn;
  }

  __device__ void fold1(int h, int c, float& M, float& Ls, float& acc) const {
    if (!on) return;
    const float ms = znew(h);
    const float mn = fmaxf(M, ms);
    const float sa = __builtin_amdgcn_exp2f(M - mn), sb = __builtin_amdgcn_exp2f(ms - mn);
    acc = acc * sa + sc->vnew[c] * sb;
    Ls = Ls * sa + sb;
    M = mn;
  }

  // The codes go to the caches last: the key record and both scales, and the token's
  // bits of its value tile (one atomic per record bit: the tile's other tokens share
  // those words).
  __device__ void finish() {
    if (!on) return;
    const int tid = threadIdx.x;
    const int64_t tg = row * cap + (len - 1);
    for (int i = tid; i < rk / 4; i += NTHR)
      reinterpret_cast<uint32_t*>(k_codes + tg * rk)[i] = sc->erec[0][i];
    if (tid == 0) {
      k_alpha[tg] = (uint16_t)sc->ea16[0];
      v_alpha[tg] = (uint16_t)sc->ea16[1];
    }
    const int p = len - 1, tp = p & (kTile - 1);
    const uint32_t bit = 1u << tile_bit(tp);
    uint32_t* gt = reinterpret_cast<uint32_t*>(v_codes + (row * cap + (p - tp)) * rv) + tile_word(tp);
    for (int v = tid; v < 8 * rv; v += NTHR) {
      if ((sc->erec[1][v >> 5] >> (v & 31)) & 1u)
        __hip_atomic_fetch_or(&gt[2 * v], bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      else
        __hip_atomic_fetch_and(&gt[2 * v], ~bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
};

// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void decode_split_kernel(
    const void* __restrict__ params_k, const void* __restrict__ params_v, int n_q_heads,
    int n_kv_heads, const void* __restrict__ q, int q_dtype,
    const uint8_t* __restrict__ k_codes, const uint16_t* __restrict__ k_alpha,
    const uint8_t* __restrict__ v_codes, const uint16_t* __restrict__ v_alpha,
    const int32_t* __restrict__ seq_len, int64_t cap, float scale, float* __restrict__ out,
    unsigned* __restrict__ counters, Partial* __restrict__ partials, int n_splits, int rk,
    int rv, const Partial* __restrict__ seg) {
  extern __shared__ float dyn[];
  __shared__ float qs[kMaxGroup][kD];
  __shared__ float qp[kMaxGroup][kD];
  __shared__ float red[kThreads / 64];
  __shared__ float mh[kMaxGroup], lh[kMaxGroup];
  __shared__ float chq[kMaxGroup];      // midrise: the half-step term of the scores
  __shared__ float wh[kMaxGroup];       // sum over the split of P alpha^V

  const int split = blockIdx.x, kvh = blockIdx.y, seq = blockIdx.z;
  const int G = n_q_heads / n_kv_heads;
  const int tid = threadIdx.x;
  const HeadParams* hk = head_params(params_k, kvh);
  const HeadParams* hv = head_params(params_v, kvh);
  const bool layout_ok = hk->record_bytes == rk && hv->record_bytes == rv;
  const int bk = hk->budget, bv = hv->budget;
  const int VS = 8 * max(rk, rv);                   // record bits of the wider tensor
  float* sc = dyn;                                  // [G][kSplit] logits, then weights
  float* vq = dyn + G * kSplit;                     // [G][VS] per-bit weights / sums

  const int len = (int)min<int64_t>(max(seq_len[seq], 0), cap);   // out-of-range lengths clamp
  const int t0 = split * kSplit;
  const int nt = layout_ok ? max(0, min(kSplit, len - t0)) : 0;

  // Queries of the group, then q'_c = (T_K^T q)_c * s_c * 2^(1-b_c) * scale * log2(e).
  for (int i = tid; i < G * kD; i += kThreads)
    qs[i / kD][i % kD] = load_q(q, q_dtype, ((int64_t)seq * n_q_heads + kvh * G) * kD + i);
  __syncthreads();
  for (int i = tid; i < G * kD; i += kThreads) {
    const int h = i / kD, c = i % kD;
    float acc = 0.f;
#pragma unroll 16
    for (int j = 0; j < kD; ++j) acc += hk->T[j * kD + c] * qs[h][j];
    const int b = hk->bits[c];
    qp[h][c] = b ? acc * hk->s[c] * ldexpf(1.f, 1 - b) * scale * kLog2e : 0.f;
  }
  __syncthreads();
  // Weight of record bit v: q'_c 2^k, negated for the sign bit k = b_c - 1.
  for (int i = tid; i < G * bk; i += kThreads) {
    const int h = i / bk, v = i % bk;
    const int c = hk->virt_chan[v], k = hk->virt_bit[v];
    const float w = ldexpf(qp[h][c], k);
    vq[h * VS + v] = (k == hk->bits[c] - 1) ? -w : w;
  }
  // Midrise levels (code + 1/2) add (1/2) sum_c q'_c to every score (before alpha^K).
  if (tid < G) {
    float a = 0.f;
    if (hk->quantizer == AATC_QUANT_MIDRISE)
      for (int c = 0; c < kD; ++c) a += qp[tid][c];
    chq[tid] = 0.5f * a;
  }
  __syncthreads();

  // Scores z = alpha^K sum_v Q_v bit_v in the log2 domain.
  const int64_t kv_row = (int64_t)seq * n_kv_heads + kvh;
  for (int tl = tid; tl < kSplit; tl += kThreads) {
    float acc[kMaxGroup];
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) acc[h] = 0.f;
    if (tl < nt) {
      const int64_t t = t0 + tl;
      const uint32_t* rec = reinterpret_cast<const uint32_t*>(k_codes + (kv_row * cap + t) * rk);
      for (int w = 0; w < rk / 4; ++w) {
        uint32_t bits = rec[w];
        while (bits) {
          const int v = 32 * w + __builtin_ctz(bits);
          bits &= bits - 1;
#pragma unroll
          for (int h = 0; h < kMaxGroup; ++h)
            if (h < G) acc[h] += vq[h * VS + v];
        }
      }
      const float ak = half_bits_to_float(k_alpha[kv_row * cap + t]);
#pragma unroll
      for (int h = 0; h < kMaxGroup; ++h)
        if (h < G) sc[h * kSplit + tl] = ak * (acc[h] + chq[h]);
    } else {
      for (int h = 0; h < G; ++h) sc[h * kSplit + tl] = -INFINITY;
    }
  }
  __syncthreads();

  // Split-local softmax statistics per head; weights become 2^(z - m) * alpha^V.
  for (int h = 0; h < G; ++h) {
    float m = -INFINITY;
    for (int tl = tid; tl < kSplit; tl += kThreads) m = fmaxf(m, sc[h * kSplit + tl]);
    m = block_reduce(m, true, red);
    float l = 0.f;
    for (int tl = tid; tl < kSplit; tl += kThreads) {
      float p = (tl < nt) ? exp2f(sc[h * kSplit + tl] - m) : 0.f;
      float w = (tl < nt) ? p * half_bits_to_float(v_alpha[kv_row * cap + t0 + tl]) : 0.f;
      sc[h * kSplit + tl] = w;
      l += p;
    }
    l = block_reduce(l, false, red);
    float ws = 0.f;
    for (int tl = tid; tl < nt; tl += kThreads) ws += sc[h * kSplit + tl];
    ws = block_reduce(ws, false, red);
    if (tid == 0) {
      mh[h] = m;
      lh[h] = l;
      wh[h] = ws;
    }
  }
  __syncthreads();

  // Value bits: sum over tokens of w_t * bit_v(t), one thread per record bit.
  const uint32_t* vt = reinterpret_cast<const uint32_t*>(v_codes) +
                       (kv_row * (cap / kTile) + t0 / kTile) * (16 * rv);
  for (int v = tid; v < bv; v += kThreads) {
    float acc[kMaxGroup];
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) acc[h] = 0.f;
    for (int tile = 0; tile * kTile < nt; ++tile) {
      for (int W = 0; W < 2; ++W) {
        uint32_t word = vt[tile * 16 * rv + 2 * v + W];
        while (word) {
          const int p = __builtin_ctz(word);
          word &= word - 1;
          // bit p of word W: token 16 d + 4 g + i, d = 2 W + p % 2, g = p / 2 % 4, i = p / 8
          const int t = tile * kTile + 16 * (2 * W + (p & 1)) + 4 * ((p >> 1) & 3) + (p >> 3);
          if (t >= nt) continue;
#pragma unroll
          for (int h = 0; h < kMaxGroup; ++h)
            if (h < G) acc[h] += sc[h * kSplit + t];
        }
      }
    }
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h)
      if (h < G) vq[h * VS + v] = acc[h];
  }
  __syncthreads();

  // Partial o~_c = s_c 2^(1-b_c) (sum_{k < b-1} 2^k S_(c,k) - 2^(b-1) S_(c,b-1)).
  Partial* part = partials + (kv_row * n_splits + split) * G;
  for (int i = tid; i < G * kD; i += kThreads) {
    const int h = i / kD, c = i % kD;
    const int b = hv->bits[c];
    float o = 0.f;
    if (b && nt > 0) {
      float acc = 0.f;
      for (int k = 0; k < b; ++k) {
        const float t = ldexpf(vq[h * VS + hv->bit_off[c] + k], k);
        acc += (k == b - 1) ? -t : t;
      }
      // (midrise: the half step of every level, s_c 2^(-b_c) sum_t P_t alpha^V_t)
      o = fmaf(hv->s[c] * hv->half_step[c], wh[h], hv->s[c] * ldexpf(acc, 1 - b));
    }
    st_dev(&part[h].o[c], o);
  }
  if (tid < G) {
    st_dev(&part[tid].m, !layout_ok ? NAN : (nt > 0) ? mh[tid] : -INFINITY);
    st_dev(&part[tid].l, !layout_ok ? NAN : (nt > 0) ? lh[tid] : 0.f);
  }
  float* out_rows = out + ((int64_t)seq * n_q_heads + kvh * G) * kD;
  if (seg) {
    SegHook sh{seg + kv_row * G};
    merge_if_last<kThreads, true>(params_v, kvh, kv_row, G, n_splits, partials, counters,
                                  out_rows, dyn, sh);
  } else {
    NoHook none;
    merge_if_last<kThreads, true>(params_v, kvh, kv_row, G, n_splits, partials, counters,
                                  out_rows, dyn, none);
  }
}

// ---------------------------------------------------------------------------------------
// MFMA decode kernel (G <= 8 query heads per KV head, records of at most 64 bytes).
//
// Both contractions run on v_mfma_i32_16x16x64_i8 over the bits of the codes.
//  * Keys: D[token, (head, limb)] = sum_bits bit(token) * Qlimb[bit, (head, limb)].
//    One record dword w (32 bits of one token) expands to MFMA bytes by
//    r_d = w & (0x01010101 << d): byte j of r_d is 2^d * bit (8j + d).  The factor 2^d
//    (and the sign of int8 0x80 for d = 7) is folded into the query weights, which are
//    32-bit fixed point split into four int8 limbs: four heads times four limbs fill
//    the 16 MFMA columns.  Lane (column (h, L), row group g) of the result holds limb L
//    of the scores of tokens 4g .. 4g + 3; a reduce-scatter over the lane quad leaves
//    lane L with the full score of token 4g + L.
//  * Values: D[bit, (head, limb)] = sum_tokens bit(token) * Plimb[token, (head, limb)]
//    with P = 2^(z - m) alpha^V in 32-bit fixed point (one exponent per workgroup).
//    The value tiles store the bit of token 16 d + 4 g + i at bit 8 i + 2 g + d % 2 of
//    word d / 2, so a lane of row group g expands its two words with two masks into
//    exactly the tokens whose scores its quad computed; a byte transpose inside the quad
//    turns (one token, four limbs) per lane into (four tokens, one limb).
// Each wave scores and weights its own share of the split; the value bits are then
// split across the waves, over all tokens of the split.  Integer accumulation is exact;
// limbs are recombined in fp32.
//
// Every workgroup derives its query bit weights itself, while its cache loads are in
// flight: q~ = T_K^T q (fp32), then per bit the 32-bit fixed-point limbs.
// ---------------------------------------------------------------------------------------
template <int NT, int NTILE, int NP, int NW, bool APPEND>
// At most two waves per SIMD ever share a compute unit with this kernel (LDS holds one
// eight-wave workgroup), so it may use up to 256 VGPRs per lane.
__global__ __attribute__((amdgpu_flat_work_group_size(64 * NW, 64 * NW),
                          amdgpu_waves_per_eu(2, 2)))
void decode_mfma_kernel(const DecodeArgs a) {
  constexpr int NTHR = 64 * NW;       // threads per workgroup
  constexpr int NH = 4 * NT;          // head slots: 4 per column tile
  constexpr int TW = 16 * NTILE;      // tokens per wave
  constexpr int S = NW * TW;          // tokens per workgroup
  constexpr int NCH = S / 64;         // 64-token chunks per workgroup
  constexpr int CPW = NTILE / 4;      // chunks per wave
  constexpr int NLD = S * 64 / 16 / NTHR;   // 16-byte loads per thread per cache (64-byte records)
  // With eight waves the cache streams straight into LDS, issued by the upper half of the
  // waves; the lower half builds the query planes meanwhile (a wave whose loads wait for
  // queue space can do nothing else).  With four, every wave loads into registers.
  constexpr bool DMA = NW == 8;
  constexpr int NWC = DMA ? NW / 2 : NW;    // waves that build the query planes
  constexpr int NTC = 64 * NWC;             // their threads
  constexpr int NJQ = NTC / 32;       // row blocks of the query transform
  constexpr int RJ = kD / NJQ;        // rows per block
  constexpr int AL = S / 8;           // 16-byte loads of one alpha array (one per thread)
  constexpr int NR = NH * kD / NTHR;  // (head, channel) items per thread
  constexpr int NRC = NH * kD / NTC;  // the same per plane-building thread
  constexpr int NPI = (NH * 4 * NP * 8 + NTC - 1) / NTC;    // plane items per thread
  static_assert(NTILE % 4 == 0, "a wave owns whole 64-token chunks (and tile pairs)");
  static_assert(kMaxNH * (kD / 4) <= 64 * NW, "the merge takes one (head, 4 columns) slot per thread");
  static_assert(AL <= NTHR && NR >= 1, "thread mapping");
  static_assert(!APPEND || NW == 8, "the fused append maps one tensor to 256 threads");
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ unsigned qmx[NH];
  __shared__ int fexp_s[NH];
  __shared__ float wmax[NW][NH], wsum[NW][NH], wpa[NW][NH];
  __shared__ int fv_s[NH];
  __shared__ float chs[NH];           // midrise: the half-step term of each head's scores
  __shared__ float wpav[NW][NH];      // sum of P alpha^V per wave and head
  __shared__ unsigned csync;          // arrivals of the plane-building waves

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 15, g = lane >> 4, hc = n >> 2, L = n & 3;
  // XCD-aware order (grid a multiple of 8): workgroups are dealt to the 8 XCDs round
  // robin, so consecutive splits of a (sequence, KV head) are given block ids that land
  // on one XCD.  The grid is exactly rows x splits, so no workgroup exits early (an early
  // exit would split the argument loads into dependent round trips).
  const int nb8 = (int)(gridDim.x >> 3);
  const int lb = (gridDim.x & 7) ? (int)blockIdx.x
                                 : (int)(blockIdx.x & 7) * nb8 + (int)(blockIdx.x >> 3);
  const int row32 = lb / a.n_splits;                 // (32-bit: rows x splits < 2^30)
  const int split = lb - row32 * a.n_splits;
  const int seq = row32 / a.n_kv_heads, kvh = row32 - seq * a.n_kv_heads;
  const int64_t row = row32;
  const int len_raw = a.seq_len[seq];               // first: its round trip gates the cache loads
  __builtin_amdgcn_sched_barrier(0);
  const int G = a.G, RK = a.rk, RV = a.rv;
  const int RWK = RK >> 2;
  const HeadParams* hk = head_params(a.params_k, kvh);
  const HeadParams* hv = head_params(a.params_v, kvh);
  const int t0 = split * S;

  // (0) Loads that need nothing, by the plane-building threads (tc < NTC): the channel
  //     tables of channel cq, T_K rows RJ jq .. RJ jq + RJ - 1 at columns 4 c4 .. + 3,
  //     the bit descriptors, the queries, and (fused append) their share of the new
  //     token's transform.  Loads are unconditional (clamped indices or empty
  //     descriptors), so the wait counters stay exact.
  const bool cw = !DMA || wave < NWC;                 // builds the query planes (per wave)
  // The query transform: lane l of plane-building wave w holds T_K rows RJ jq .. + RJ - 1
  // (row block jq = l / 8) at columns 4 c4 .. + 3 (c4 = 8 w + l % 8), so the sums over the
  // row blocks stay inside the wave.
  static_assert(NJQ == 8 && RJ == 16 && NWC == 4, "query transform mapping");
  const int jq = lane >> 3, c4 = 8 * (wave % NWC) + (lane & 7), cq = tid & (kD - 1);
  constexpr int NVL = NH / 2;                   // q~ values a lane ends with
  // Scale and width of the lane's channels 4 c4 + (NVL jq + i) % 4 (head (NVL jq + i) / 4).
  float ksq[NVL];
  int kbq[NVL];
  float khs[2];                       // key half steps of channels lane and lane + 64
  // The channel tables (used only after the value phase): with eight waves every wave loads
  // them after the join.  In the front they would queue behind the cache stream, and the
  // wait before the join would then cover them.
  int vbc = 0, voc = 0, v_budget = 0, v_maxb = 0;
  float vsc = 0.f, vhs = 0.f;
  // Fused append: waves 0 and 1 encode the key and the value token, lane l channels l and
  // l + 64 (their widths, first bits and scales).
  int e_b[2] = {0, 0}, e_off[2] = {0, 0};
  float e_s[2] = {0.f, 0.f};
  bool e_mr = false;
  auto load_tables = [&]() {
    v_budget = hv->budget;
    if (APPEND && wave < 2) {
      const HeadParams* eh = wave == 0 ? hk : hv;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        e_b[i] = eh->bits[lane + 64 * i];
        e_off[i] = eh->bit_off[lane + 64 * i];
        e_s[i] = eh->s[lane + 64 * i];
      }
      // (read here, not in the merge: a load there waits a full round trip)
      e_mr = eh->quantizer == AATC_QUANT_MIDRISE;
    }
    vbc = hv->bits[cq];
    voc = hv->bit_off[cq];
    vsc = hv->s[cq];
    vhs = hv->half_step[cq];
    v_maxb = hv->max_bits;
  };
  v4f tr[RJ];
  uint2 desc[NPI];
  const bool q_bf = a.q_dtype == AATC_BF16;
  uint32_t qraw[NRC];
  bool qhi[NRC];
  // Fused append: dot products d = split + n_splits k, k = wave + NWC i, of the 2 x 128
  // (key channels, then value channels); the first two of each plane-building wave are
  // fetched up front (the token's two elements of this lane and the matching two of
  // column d % kD of Tq), further ones (fewer than 32 splits) when they are computed.
  const int x_eb = a.x_dtype == AATC_BF16 ? 2 : 4;
  constexpr int KF = 2;                               // coefficients fetched up front
  int adk[KF];
  uint32_t ax[KF][2];
  int atq[KF][2];
  float a_inv_s[KF];
  auto front_loads = [&]() {
#pragma unroll
    for (int i = 0; i < NVL; ++i) {
      const int c = 4 * c4 + ((NVL * jq + i) & 3);
      ksq[i] = hk->s[c];
      kbq[i] = hk->bits[c];
    }
#pragma unroll
    for (int jj = 0; jj < RJ; ++jj)
      tr[jj] = reinterpret_cast<const v4f*>(hk->T)[(RJ * jq + jj) * (kD / 4) + c4];
    khs[0] = hk->half_step[lane];
    khs[1] = hk->half_step[lane + 64];
    // Plane items (head, record dword D, bit d of each byte): the 4 record bits 32 D +
    // 8 j + d, j = 0..3, of one head.
#pragma unroll
    for (int r = 0; r < NPI; ++r) {
      const int dd = (r * NTC + tid) % (8 * RWK);                // < 128: in the table
      desc[r] = reinterpret_cast<const uint2*>(hk->bit_desc)[dd];
    }
    // Queries, element r NTC + tid, read as the aligned dword that holds the element
    // (either type, no branch; the dword never leaves the element's page).
    const int64_t qb = ((int64_t)seq * a.n_q_heads + kvh * G) * kD;
#pragma unroll
    for (int r = 0; r < NRC; ++r) {
      const int64_t i = qb + min(r * NTC + tid, G * kD - 1);
      const uintptr_t ad = reinterpret_cast<uintptr_t>(a.q) + (q_bf ? 2 * i : 4 * i);
      qraw[r] = *reinterpret_cast<gdword>(ad & ~(uintptr_t)3);
      qhi[r] = (ad & 2) != 0;
    }
    if constexpr (APPEND) {
#pragma unroll
      for (int f = 0; f < KF; ++f) {
        const int d = __builtin_amdgcn_readfirstlane(split + a.n_splits * (wave + NWC * f));
        adk[f] = d;
        const bool on = d < 2 * kD;
        const HeadParams* eh = d >= kD ? hv : hk;
        const int ac = d & (kD - 1);
        const __amdgpu_buffer_rsrc_t xrs =
            make_rsrc(static_cast<const uint8_t*>(d >= kD ? a.x_v : a.x_k) + row * kD * x_eb,
                      on ? (uint32_t)(kD * x_eb) : 0u);
        const __amdgpu_buffer_rsrc_t trs = make_rsrc(eh->Tqt + ac * kD, on ? 4u * kD : 0u);
        ax[f][0] = __builtin_amdgcn_raw_buffer_load_b32(xrs, (lane * x_eb) & ~3, 0, 0);
        ax[f][1] = __builtin_amdgcn_raw_buffer_load_b32(xrs, ((lane + 64) * x_eb) & ~3, 0, 0);
        atq[f][0] = (int)__builtin_amdgcn_raw_buffer_load_b32(trs, 4 * lane, 0, 0);
        atq[f][1] = (int)__builtin_amdgcn_raw_buffer_load_b32(trs, 4 * (lane + 64), 0, 0);
        a_inv_s[f] = eh->inv_s[ac];
      }
    }
  };

  Partial* parts = a.partials + row * a.n_splits * G;
  float* out_rows = a.out + ((int64_t)seq * a.n_q_heads + kvh * G) * kD;
  const int len = (int)min<int64_t>(max(len_raw, 0), a.cap);
  // With a fused append the splits stop short of the new token at len - 1; the merging
  // workgroup encodes it and adds it to the merge.
  const int nt = max(0, min(S, (APPEND ? len - 1 : len) - t0));

  // (1) This split's packed cache (loads past the capacity read 0).  The layout check
  //     below gates the compute, not these loads.
  const int n_load = min(S, (nt + kTile - 1) / kTile * kTile);
  const int nk16 = n_load * RK / 16, nv16 = n_load * RV / 16, na16 = n_load / 8;
  const __amdgpu_buffer_rsrc_t krs = make_rsrc(a.k_codes + row * a.cap * RK, (uint32_t)(a.cap * RK));
  const __amdgpu_buffer_rsrc_t vrs = make_rsrc(a.v_codes + row * a.cap * RV, (uint32_t)(a.cap * RV));
  const __amdgpu_buffer_rsrc_t akrs = make_rsrc(a.k_alpha + row * a.cap, (uint32_t)(a.cap * 2));
  const __amdgpu_buffer_rsrc_t avrs = make_rsrc(a.v_alpha + row * a.cap, (uint32_t)(a.cap * 2));
  uint8_t* kbuf = smem;
  uint8_t* vbuf = smem + a.off_v;
  uint16_t* akb = reinterpret_cast<uint16_t*>(smem + a.off_ak);
  uint16_t* avb = reinterpret_cast<uint16_t*>(smem + a.off_av);
  // Loads a thread does not need get an offset past the descriptor (they return 0).
  constexpr uint32_t kNone = 0x80000000u;
  v4i rk[DMA ? 1 : NLD], rv[DMA ? 1 : NLD], rak, rav;
  int nv_mine = 0;                                    // value-tile transfers of this wave
  // 1 KiB transfers straight into LDS (lane l's 16 bytes at 16 l): key records, the token
  // scales, then the value tiles, dealt to the issuing waves round robin.  Only whole
  // 1 KiB blocks of the regions are written (their sizes are 1 KiB multiples).
  auto issue_cache = [&]() {
    constexpr int NWD = NW - NWC;
    const int wd = __builtin_amdgcn_readfirstlane(wave - NWC);
    const int nki = (n_load * RK + 1023) >> 10, nai = (2 * n_load + 1023) >> 10;
    const int nvi = (n_load * RV + 1023) >> 10;
    for (int j = wd; j < nki; j += NWD)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          krs, (__attribute__((address_space(3))) void*)(kbuf + 1024 * j), 16,
          t0 * RK + 1024 * j + 16 * lane, 0, 0, 0);
    for (int j = wd; j < nai; j += NWD) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          akrs, (__attribute__((address_space(3))) void*)((uint8_t*)akb + 1024 * j), 16,
          2 * t0 + 1024 * j + 16 * lane, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          avrs, (__attribute__((address_space(3))) void*)((uint8_t*)avb + 1024 * j), 16,
          2 * t0 + 1024 * j + 16 * lane, 0, 0, 0);
    }
    for (int j = wd; j < nvi; j += NWD) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          vrs, (__attribute__((address_space(3))) void*)(vbuf + 1024 * j), 16,
          t0 * RV + 1024 * j + 16 * lane, 0, 0, 0);
      ++nv_mine;
    }
  };
  // No branch on the split's contents: an empty split computes on masked tokens and
  // stores (m, l, o~) = (-inf, 0, 0); records that do not match the parameters store a
  // NaN maximum (the value budget is clamped to the record so LDS accesses stay in range).
  const bool layout_ok = (hk->record_bytes == RK) & (hv->record_bytes == RV);
  const __amdgpu_buffer_rsrc_t prs =
      make_rsrc(parts, (uint32_t)(a.n_splits * G * sizeof(Partial)));

  // (2) Query planes, by the plane-building waves; they synchronize among themselves
  //     (the other waves are busy issuing the cache) through an LDS arrival count, or
  //     through workgroup barriers when every wave builds.
  unsigned csync_target = 0u;
  auto plane_sync = [&]() {
    if constexpr (DMA) {
      csync_target += NWC;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      if (lane == 0) __hip_atomic_fetch_add(&csync, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      while (__hip_atomic_load(&csync, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) < csync_target)
        __builtin_amdgcn_s_sleep(1);
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    } else {
      __syncthreads();
    }
  };
  // Scratch of the planes: over the value operands (written only after the planes) with
  // eight waves, over the cache region with four (the cache lands after the planes).
  float* scr = reinterpret_cast<float*>(smem + (DMA ? a.off_pb : 0));   // [NJQ][NH][kD]
  float* qs = scr + NJQ * NH * kD;                                     // [NH][kD]
  float* qcl = scr;                                  // [NH][kD]
  uint8_t* ql = smem + a.off_ql;                     // [4][NH][2 NP][64]
  float rcf[KF] = {0.f, 0.f};                        // fused append: this wave's coefficients
  float reh[KF] = {0.f, 0.f};                        // and the token's error bounds
  auto build_planes = [&]() {
#pragma unroll
    for (int r = 0; r < NRC; ++r) {
      const uint32_t w = qraw[r];
      const float qv = q_bf ? __uint_as_float((qhi[r] ? (w >> 16) : (w & 0xffffu)) << 16)
                            : __uint_as_float(w);
      qs[r * NTC + tid] = ((r * NTC + tid) / kD < G) ? qv : 0.f;
    }
    plane_sync();                                    // qs, qmx
    // q~ = T_K^T q: RJ-row partial sums per lane, then over the wave's 8 row blocks
    // (reduce-scatter across lane bits 3..5): lane l ends with value NVL jq + i of the 4 NH
    // (head, column) sums of its column quad.
    {
      v4f acc[NH];
#pragma unroll
      for (int h = 0; h < NH; ++h) acc[h] = (v4f){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jj = 0; jj < RJ; jj += 4)
#pragma unroll
        for (int h = 0; h < NH; ++h) {
          const v4f qv = *reinterpret_cast<const v4f*>(qs + h * kD + RJ * jq + jj);
          acc[h] += tr[jj] * qv.x + tr[jj + 1] * qv.y + tr[jj + 2] * qv.z + tr[jj + 3] * qv.w;
        }
      float v0[4 * NH], v1[2 * NH], v2[NH], v3[NVL];
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        v0[4 * h] = acc[h].x;
        v0[4 * h + 1] = acc[h].y;
        v0[4 * h + 2] = acc[h].z;
        v0[4 * h + 3] = acc[h].w;
      }
      reduce_scatter_step<4 * NH, 32>(v0, v1);
      reduce_scatter_step<2 * NH, 16>(v1, v2);
      reduce_scatter_step<NH, 8>(v2, v3);
      // Channel weight Q_c = q~_c s_c scale log2(e) (the weight of the code's sign bit up
      // to sign), kept in LDS; the largest |Q_c| of a head sets its fixed-point exponent.
      const int hl = (NVL * jq) >> 2;                // the lane's head
      float mloc = 0.f;
#pragma unroll
      for (int i = 0; i < NVL; ++i) {
        const int c = 4 * c4 + ((NVL * jq + i) & 3);
        const float qc = (hl < G && kbq[i] > 0) ? v3[i] * ksq[i] * a.scale_log2e : 0.f;
        qcl[hl * kD + c] = qc;
        mloc = fmaxf(mloc, fabsf(qc));
      }
      // Over the lanes that hold head hl: lane bits 0..2, and bit 3 when NH = 4.
      mloc = fmaxf(mloc, dpp_f<0xB1>(mloc));         // quad_perm [1,0,3,2]
      mloc = fmaxf(mloc, dpp_f<0x4E>(mloc));         // quad_perm [2,3,0,1]
      mloc = fmaxf(mloc, dpp_f<0x141>(mloc));        // row_half_mirror
      if constexpr (NH == 4) mloc = fmaxf(mloc, dpp_f<0x128>(mloc));   // row_ror:8
      if ((lane & (NH == 4 ? 15 : 7)) == 0) atomicMax(&qmx[hl], __float_as_uint(mloc));
    }
    plane_sync();                                    // qcl, qmx
    // Midrise: every score has the term alpha^K C_h with C_h = sum_c Q_c 2^(-b_c) over the
    // stored channels (the half step of each level); 0 for the midtread reading.
    for (int h = wave % NWC; h < NH; h += NWC) {
      const float cp = wave_sum_dpp(qcl[h * kD + lane] * khs[0] + qcl[h * kD + lane + 64] * khs[1]);
      if (lane == 0) chs[h] = cp;
    }
    if (tid < NH) {
      int e = 0;
      frexpf(__uint_as_float(qmx[tid]), &e);
      fexp_s[tid] = qmx[tid] ? 30 - e : 0;
    }
    // Record bit v = 32 D + 8 j + d  ->  K-step 2 (D % NP) + d / 4, lane group D / NP,
    // byte 4 (d % 4) + j of the 16-byte operand; dwords RWK .. 4 NP - 1 get weight 0.
    // Weight 2^(k + 1 - b) Q_c / 2^d, negated for the sign bit and for d = 7 (int8 0x80 =
    // -128); the four limbs of the four bits j = 0..3 are transposed into one dword per
    // limb plane.
    for (int i = tid; i < 4 * NH * 2 * 4 * (4 * NP - RWK); i += NTC) {
      const int D = RWK + i / (4 * NH * 2 * 4), rest = i % (4 * NH * 2 * 4);
      const int plane = rest / 8, st = 2 * (D % NP) + ((rest >> 2) & 1);
      *reinterpret_cast<uint32_t*>(ql + (plane * 2 * NP + st) * 64 + ((D / NP) << 4) +
                                   4 * (rest & 3)) = 0u;
    }
    // Items without branches or divisions, all channel-weight reads issued together:
    // the fixed-point exponent of every head first, then every item's four weights.
    const int nbh = 8 * RWK;                         // items per head
    int fe_h[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      int e = 0;
      const unsigned qm = qmx[h];
      frexpf(__uint_as_float(qm), &e);
      fe_h[h] = qm ? 30 - e : 0;
    }
    int hi_[NPI], dd_[NPI];
    float qv_[NPI][4];
#pragma unroll
    for (int r = 0; r < NPI; ++r) {
      const int i = r * NTC + tid;
      int h = 0;
#pragma unroll
      for (int hh = 1; hh < NH; ++hh) h += (i >= hh * nbh) ? 1 : 0;
      hi_[r] = h;
      dd_[r] = i - h * nbh;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t ent = ((j < 2 ? desc[r].x : desc[r].y) >> (16 * (j & 1))) & 0xffffu;
        qv_[r][j] = qcl[h * kD + (ent & 127)];
      }
    }
#pragma unroll
    for (int r = 0; r < NPI; ++r) {
      const int i = r * NTC + tid, h = hi_[r], D = dd_[r] >> 3, d = dd_[r] & 7;
      int fe = fe_h[0];
#pragma unroll
      for (int hh = 1; hh < NH; ++hh) fe = (h == hh) ? fe_h[hh] : fe;
      uint32_t x[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t ent = ((j < 2 ? desc[r].x : desc[r].y) >> (16 * (j & 1))) & 0xffffu;
        int fx = (int)rintf(ldexpf(qv_[r][j], (int)((ent >> 8) & 15) - kDescBias + fe - d));
        if ((((ent >> 14) & 1) != 0) != (d == 7)) fx = -fx;
        x[j] = (ent & 0x8000u) ? pack_limbs(fx) : 0u;
      }
      // x[j] = (limb 0..3 of bit j)  ->  y[L] = (limb L of bits 0..3)
      const uint32_t t0 = __builtin_amdgcn_perm(x[1], x[0], 0x05010400u);
      const uint32_t t1 = __builtin_amdgcn_perm(x[3], x[2], 0x05010400u);
      const uint32_t t2 = __builtin_amdgcn_perm(x[1], x[0], 0x07030602u);
      const uint32_t t3 = __builtin_amdgcn_perm(x[3], x[2], 0x07030602u);
      const uint32_t y[4] = {__builtin_amdgcn_perm(t1, t0, 0x05040100u),
                             __builtin_amdgcn_perm(t1, t0, 0x07060302u),
                             __builtin_amdgcn_perm(t3, t2, 0x05040100u),
                             __builtin_amdgcn_perm(t3, t2, 0x07060302u)};
      const int st = 2 * (D % NP) + (d >> 2);
      const int pos = ((D / NP) << 4) + ((d & 3) << 2);
      // Items past the last head's go to the consumed queries instead.
      const bool ok = i < G * nbh;
#pragma unroll
      for (int l4 = 0; l4 < 4; ++l4) {
        uint8_t* dst = ok ? ql + ((l4 * NH + h) * 2 * NP + st) * 64 + pos
                          : reinterpret_cast<uint8_t*>(qs) + 16 * (tid & 63) + 4 * l4;
        *reinterpret_cast<uint32_t*>(dst) = y[l4];
      }
    }
    // Fused append: this wave's coefficients (stored after the value phase, when no
    // cache transfer is queued ahead of the stores).
    if constexpr (APPEND)
      append_coefficients<KF>(ax, atq, a.x_dtype, a_inv_s, rcf, reh);  // (past 2 kD: unused)
  };

  // (3) Front.  Eight waves: the plane-building and the issuing waves take separate arms
  //     up to the barrier where the key records and scales have landed; the value tiles
  //     keep landing through the key phase.  The barriers are plain s_barrier after
  //     explicit waits: __syncthreads() would make the issuing waves wait for all of their
  //     transfers.  The explicit vmcnt(0) waits cost nothing (no load of the wave is in
  //     flight there) but tell the compiler so: with the two arms merged, it would
  //     otherwise take the other arm's loads as pending and wait on them later with counts
  //     that also cover the cache transfers.
  if constexpr (DMA) {
    if (cw) {
      front_loads();
      if (tid < NH) qmx[tid] = 0u;
      if (tid == 0) csync = 0u;
      __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
      plain_barrier();                               // the small loads are queued first
      build_planes();
      __builtin_amdgcn_s_waitcnt(kWaitVm0);
    } else {
      plain_barrier();
      __builtin_amdgcn_s_waitcnt(kWaitVm0);
      issue_cache();
      wait_vmcnt(nv_mine);                           // key records and scales landed
    }
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    plain_barrier();
    load_tables();
  } else {
    front_loads();
    load_tables();
    if (tid < NH) qmx[tid] = 0u;
    if (tid == 0) csync = 0u;
    // Each wave issues its key records and token scales ahead of its value tiles.
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int idx = tid + i * NTHR;
      rk[i] = buf_load16<0>(krs, idx < nk16 ? (uint32_t)(t0 * RK + 16 * idx) : kNone);
    }
    {
      const uint32_t aoff = (tid < na16) ? (uint32_t)(2 * t0 + 16 * tid) : kNone;
      rak = buf_load16<0>(akrs, aoff);
      rav = buf_load16<0>(avrs, aoff);
    }
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int idx = tid + i * NTHR;
      rv[i] = buf_load16<0>(vrs, idx < nv16 ? (uint32_t)(t0 * RV + 16 * idx) : kNone);
    }
    // Keep the compiler from moving work that waits on the early loads above the cache loads.
    __builtin_amdgcn_sched_barrier(0);
    build_planes();
    __syncthreads();                                 // the planes' scratch is consumed
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int idx = tid + i * NTHR;
      if (idx < nk16) reinterpret_cast<v4i*>(kbuf)[idx] = rk[i];
    }
    if (tid < na16) {
      reinterpret_cast<v4i*>(akb)[tid] = rak;
      reinterpret_cast<v4i*>(avb)[tid] = rav;
    }
    __syncthreads();
  }
  v4i bq[NT][2 * NP];
  float sfx[NT], chk[NT];
#pragma unroll
  for (int rt = 0; rt < NT; ++rt) {
    const int h = 4 * rt + hc;
#pragma unroll
    for (int s = 0; s < 2 * NP; ++s)
      bq[rt][s] = *reinterpret_cast<const v4i*>(ql + ((L * NH + h) * 2 * NP + s) * 64 + 16 * g);
    sfx[rt] = ldexpf(1.f, -fexp_s[4 * rt + g]);   // (the head of this lane's scores)
    chk[rt] = chs[4 * rt + g];
  }
  // Q_c of every head for channels lane and lane + 64, for the fused append's key token
  // (eight waves: the planes' scratch is intact until the softmax writes the value
  // operands).
  float qk[2][NH] = {};
  if constexpr (APPEND) {
    if (wave == 0) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int h = 0; h < NH; ++h) qk[i][h] = qcl[h * kD + lane + 64 * i];
    }
  }

  // (4) Key scores of this wave's tokens.  The query planes are the A operand (row 4 h + L:
  //     head h, limb L) and the record bits the B operand (column: token), so lane 16 h + n
  //     ends with the four limb sums of head h for token n of the tile and recombines them
  //     itself.
  const int wb = wave * TW;
  float zr[NTILE][NT];
  float avt[NTILE];
  float lav[NTILE];                      // log2 alpha^V (-inf for 0 and past the tokens)
  // Every tile's record dwords and token scales first (one LDS round trip), then the
  // products; lane group g holds record dwords g NP .. g NP + NP - 1, and dwords past the
  // record (they belong to the next token) meet zero query weights.
  uint32_t wda[NTILE][NP];
  uint16_t aka[NTILE], ava[NTILE];
#pragma unroll
  for (int tt = 0; tt < NTILE; ++tt) {
    const uint8_t* rec = kbuf + (wb + 16 * tt + n) * RK;
#pragma unroll
    for (int P = 0; P < NP; ++P) wda[tt][P] = *reinterpret_cast<const uint32_t*>(rec + 4 * (g * NP + P));
    aka[tt] = akb[wb + 16 * tt + n];
    ava[tt] = avb[wb + 16 * tt + n];
  }
  __builtin_amdgcn_sched_barrier(0);
  // Tiles go in pairs: two independent MFMA chains interleave.
#pragma unroll
  for (int tp = 0; tp < NTILE; tp += 2) {
    v4i acc[2][NT];
    uint32_t wd[2][NP];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
#pragma unroll
      for (int P = 0; P < NP; ++P) wd[u][P] = wda[tp + u][P];
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) acc[u][rt] = (v4i){0, 0, 0, 0};
    }
#pragma unroll
    for (int P = 0; P < NP; ++P) {
      v4i a0[2], a1[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const uint32_t w = wd[u][P];
        a0[u] = (v4i){(int)(w & 0x01010101u), (int)(w & 0x02020202u), (int)(w & 0x04040404u),
                      (int)(w & 0x08080808u)};
        a1[u] = (v4i){(int)(w & 0x10101010u), (int)(w & 0x20202020u), (int)(w & 0x40404040u),
                      (int)(w & 0x80808080u)};
      }
#pragma unroll
      for (int rt = 0; rt < NT; ++rt)
#pragma unroll
        for (int u = 0; u < 2; ++u) acc[u][rt] = mfma_i8(bq[rt][2 * P], a0[u], acc[u][rt]);
#pragma unroll
      for (int rt = 0; rt < NT; ++rt)
#pragma unroll
        for (int u = 0; u < 2; ++u) acc[u][rt] = mfma_i8(bq[rt][2 * P + 1], a1[u], acc[u][rt]);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int tt = tp + u;
      const int tok = wb + 16 * tt + n;
      const bool tok_ok = tok < nt;
      const float ak = half_bits_to_float(aka[tt]);
      const float av = half_bits_to_float(ava[tt]);
      avt[tt] = tok_ok ? av : 0.f;
      lav[tt] = avt[tt] > 0.f ? __builtin_amdgcn_logf(avt[tt]) : -INFINITY;
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) {
        const v4i d = acc[u][rt];                 // limbs 0..3 (weights 256^i)
        float f = fmaf((float)d[3], 256.f, (float)d[2]);
        f = fmaf(f, 256.f, (float)d[1]);
        f = fmaf(f, 256.f, (float)d[0]);
        zr[tt][rt] = (tok_ok && 4 * rt + g < G) ? fmaf(f, sfx[rt], chk[rt]) * ak : -INFINITY;
      }
    }
  }

  // (5) Softmax: one maximum per head over the workgroup, and one fixed-point exponent
  //     per head for P alpha^V from its largest value, max_i 2^(z_i - m) alpha^V_i =
  //     2^(max_i (z_i + log2 alpha^V_i) - m) (both maxima in one reduction).
#pragma unroll
  for (int rt = 0; rt < NT; ++rt) {
    float m = -INFINITY, m2 = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < NTILE; ++tt) {
      m = fmaxf(m, zr[tt][rt]);
      m2 = fmaxf(m2, zr[tt][rt] + lav[tt]);
    }
    m = row16_max(m);
    m2 = row16_max(m2);
    if (n == 0) {
      wmax[wave][4 * rt + g] = m;
      wpa[wave][4 * rt + g] = m2;
    }
  }
  __syncthreads();
  float mh[NT];
  int fvh[NT];
#pragma unroll
  for (int rt = 0; rt < NT; ++rt) {
    mh[rt] = wmax[0][4 * rt + g];
    float m2 = wpa[0][4 * rt + g];
#pragma unroll
    for (int w = 1; w < NW; ++w) {
      mh[rt] = fmaxf(mh[rt], wmax[w][4 * rt + g]);
      m2 = fmaxf(m2, wpa[w][4 * rt + g]);
    }
    // P alpha^V <= 2^(m2 - m) < 2^e; one bit of margin for the hardware exp2 and log2,
    // so P alpha^V 2^fv < 2^30.
    int e = 0;
    frexpf(__builtin_amdgcn_exp2f(m2 - mh[rt]), &e);
    fvh[rt] = m2 > -INFINITY ? 29 - e : 0;
    if (n == 0 && wave == 0) fv_s[4 * rt + g] = fvh[rt];
  }
  // Token 16 q + 4 e + L of a chunk sits at bit d = 2 e + q % 2 of its value byte; this
  // lane's tokens have e = hc.
  float sc_even[NT], sc_odd[NT];
#pragma unroll
  for (int rt = 0; rt < NT; ++rt) {
    sc_even[rt] = ldexpf(1.f, fvh[rt] - 2 * hc);
    sc_odd[rt] = (hc == 3 ? -1.f : 1.f) * ldexpf(1.f, fvh[rt] - 2 * hc - 1);
  }
  const uint32_t sel_a = (L & 2) ? 0x03020706u : 0x05040100u;
  const uint32_t sel_b = (L & 1) ? 0x03070105u : 0x06020400u;
  v4i* pb = reinterpret_cast<v4i*>(smem + a.off_pb);  // [NCH][NT][64] value operands
#pragma unroll
  for (int rt = 0; rt < NT; ++rt) {
    float lsum = 0.f, pasum = 0.f;
#pragma unroll
    for (int ch = 0; ch < CPW; ++ch) {
      uint32_t y[4];
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int tt = 4 * ch + qd;
        const float z = zr[tt][rt];
        // (the hardware exp2: results below 2^-126 flush to 0, below any weight that counts)
        const float p = (z == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(z - mh[rt]);
        lsum += p;
        pasum = fmaf(p, avt[tt], pasum);
        const int fx = (int)rintf(p * avt[tt] * ((qd & 1) ? sc_odd[rt] : sc_even[rt]));
        uint32_t x = pack_limbs(fx);
        // quad byte transpose: (token L, limbs 0..3) -> (limb L, tokens 0..3)
        x = __builtin_amdgcn_perm(quad_xor2(x), x, sel_a);
        y[qd] = __builtin_amdgcn_perm(quad_xor1(x), x, sel_b);
      }
      // Limb L of head g for tokens 16 q + 4 hc + (0..3): lane 16 hc + 4 g + L of the
      // value phase's B operand.
      pb[((wave * CPW + ch) * NT + rt) * 64 + 16 * hc + 4 * g + L] =
          (v4i){(int)y[0], (int)y[1], (int)y[2], (int)y[3]};
    }
    lsum = row16_sum(lsum);
    pasum = row16_sum(pasum);
    if (n == 0) {
      wsum[wave][4 * rt + g] = lsum;
      wpav[wave][4 * rt + g] = pasum;
    }
  }
  // The value tiles: the issuing waves wait for the rest of their transfers, or every
  // wave stores its registers (their region held nothing since the query transform).
  if constexpr (DMA) {
    // (Every wave: no load of the plane-building waves is in flight here, and the explicit
    // wait keeps the compiler from carrying the issuing waves' loads past this point.)
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
  } else {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int idx = tid + i * NTHR;
      if (idx < nv16) reinterpret_cast<v4i*>(vbuf)[idx] = rv[i];
    }
  }
  __syncthreads();

  // (6) Value bits x P limbs; value-bit tiles of 16 bits are dealt to the waves round
  //     robin.  O'(v) goes to LDS (over the consumed key records).  With eight waves the
  //     chunks go in two halves: waves 0-3 take the first half of every tile, waves 4-7
  //     the second (each reads only its half's P operands, and O' has one copy per half),
  //     and the two groups walk the tiles in opposite orders, so that the two waves of a
  //     SIMD (s and s + 4) have the same number of tiles between them on every SIMD.
  const int BV = min(v_budget, 8 * RV);
  const int NVT = (BV + 15) >> 4;
  const uint32_t m0 = 0x01010101u << (2 * g), m1 = m0 << 1;
  constexpr bool kHalves = NW == 8 && NCH % 2 == 0;
  constexpr int NCW = kHalves ? NCH / 2 : NCH;        // chunks of a wave's tile pass
  constexpr int NWT = kHalves ? NW / 2 : NW;          // waves over the tiles of one half
  const int hf = kHalves ? (wave >> 2) : 0;           // this wave's chunk half
  const int wj = kHalves ? (hf ? 3 - (wave & 3) : (wave & 3)) : wave;   // its first tile
  float* ob = reinterpret_cast<float*>(smem + a.off_ob);   // [halves][NH][ob_stride]
  // T_V for the merge: with eight waves every split loads its matrix-core operands during
  // the value loop (32 VGPRs, one k-step per tile, so that the loads never back up the
  // memory queue), and the split that merges has them at hand.  Otherwise each split
  // touches a slice of T_V, so that the merging one finds it in its XCD's L2 (the splits of
  // a (sequence, KV head) run on one XCD: block order above).
  constexpr bool kTvHeld = TvMfma<NTHR>::NPASS == 1;
  TvMfma<NTHR> tv;
  uint32_t tv_touch = 0u;
  if constexpr (!kTvHeld)
    tv_touch = reinterpret_cast<gdword>(reinterpret_cast<uintptr_t>(hv->Tm))[
        (split * NTHR + tid) * 16 % (kD * kD)];
  // A operands (this half's chunks) stay in registers when they fit (16 x 4 VGPRs).
  constexpr bool kPbRegs = NCW * NT <= 16;
  const v4i* pbh = pb + hf * NCW * NT * 64;
  v4i pbr[kPbRegs ? NCW * NT : 1];
  if constexpr (kPbRegs) {
    // All reads first (one LDS round trip), then the pins that keep them in registers
    // rather than re-read per tile.
#pragma unroll
    for (int i = 0; i < NCW * NT; ++i) pbr[i] = pbh[i * 64 + lane];
#pragma unroll
    for (int i = 0; i < NCW * NT; ++i) asm volatile("" : "+v"(pbr[i]));
  }
  // LDS address of this lane's value-bit dword pair in each chunk of the half for tile
  // vt = wj; tile wj + NWT it is 128 NWT it bytes further (an immediate offset: no address
  // arithmetic in the loop).
  uint32_t vaddr[NCW];
  {
    const uint32_t vb = (uint32_t)reinterpret_cast<uintptr_t>(
        (__attribute__((address_space(3))) uint8_t*)vbuf) + 8 * n + 128 * wj;
#pragma unroll
    for (int ch = 0; ch < NCW; ++ch) {
      vaddr[ch] = vb + (hf * NCW + ch) * kTile * RV;
      asm volatile("" : "+v"(vaddr[ch]));          // computed once, not per tile
    }
  }
  float* obh = ob + hf * NH * a.ob_stride;
  constexpr int kMaxIt = (64 * 8 / 16 + NWT - 1) / NWT;   // records of at most 64 bytes
#pragma unroll
  for (int it = 0; it < kMaxIt; ++it) {
    const int vt = wj + NWT * it;
    if (vt >= NVT) break;                           // (uniform)
    if constexpr (kTvHeld)
      if (it < 4) tv.load_step(hv, it);
    // One accumulator per column tile: a dependent product takes its predecessor's result
    // straight from the matrix unit.
    v4i acc[NT];
#pragma unroll
    for (int rt = 0; rt < NT; ++rt) acc[rt] = (v4i){0, 0, 0, 0};
    // All of the tile's value-bit words first (one LDS round trip), then the products.
    typedef uint32_t v2u __attribute__((ext_vector_type(2)));
    v2u wws[NCW];
#pragma unroll
    for (int ch = 0; ch < NCW; ++ch)
      wws[ch] = *(const __attribute__((address_space(3))) v2u*)(uintptr_t)(
          vaddr[ch] + 128 * NWT * it);
    // (The scheduler would otherwise pair each read with its products: one LDS round
    // trip per chunk.)
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ch = 0; ch < NCW; ++ch) {
      const v2u ww = wws[ch];
      const v4i av4 = {(int)(ww.x & m0), (int)(ww.x & m1), (int)(ww.y & m0), (int)(ww.y & m1)};
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) {
        const v4i bop = kPbRegs ? pbr[kPbRegs ? ch * NT + rt : 0] : pbh[(ch * NT + rt) * 64 + lane];
        acc[rt] = mfma_i8(bop, av4, acc[rt]);
      }
    }
    // (P limbs are the A operand: lane 16 h + n ends with the four limb sums of head h for
    // value bit 16 vt + n.)
#pragma unroll
    for (int rt = 0; rt < NT; ++rt) {
      const v4i d = acc[rt];
      float f = fmaf((float)d[3], 256.f, (float)d[2]);
      f = fmaf(f, 256.f, (float)d[1]);
      f = fmaf(f, 256.f, (float)d[0]);
      obh[(4 * rt + g) * a.ob_stride + 16 * vt + n] = f;
    }
  }
  if constexpr (kTvHeld) {
    // (k-steps the loop did not reach: fewer than four tiles for this wave)
    const int nit = NVT > wj ? (NVT - wj + NWT - 1) / NWT : 0;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      if (kk >= nit) tv.load_step(hv, kk);
  }

  __syncthreads();

  asm volatile("" ::"v"(tv_touch));      // keeps the touch load
  if constexpr (APPEND) {
    // Fused append: the coefficients into the workspace (device-coherent, before this
    // workgroup's arrival), and further ones when the row has fewer than 32 splits.
    if (cw) {
      // Coefficient d at d; the wave with the token's first channel (d = 0 keys, 128
      // values) also stores the token's error bound at 2 kD + d / kD.
      const __amdgpu_buffer_rsrc_t rrs = make_rsrc(a.append_r + row * kAppStride, kAppStride * 4);
#pragma unroll
      for (int f = 0; f < KF; ++f) {
        if (adk[f] < 2 * kD && lane == 0) buf_store4_coherent(rcf[f], rrs, (uint32_t)(4 * adk[f]));
        if (adk[f] < 2 * kD && (adk[f] & (kD - 1)) == 0 && lane == 0)
          buf_store4_coherent(reh[f], rrs, (uint32_t)(4 * (2 * kD + adk[f] / kD)));
      }
      for (int d = split + a.n_splits * (wave + NWC * KF); d < 2 * kD; d += a.n_splits * NWC) {
        const HeadParams* eh = d >= kD ? hv : hk;
        const int c = d & (kD - 1);
        const uint8_t* xb = static_cast<const uint8_t*>(d >= kD ? a.x_v : a.x_k) + row * kD * x_eb;
        const uint32_t xw[1][2] = {{*reinterpret_cast<const uint32_t*>(xb + ((lane * x_eb) & ~3)),
                                    *reinterpret_cast<const uint32_t*>(xb + (((lane + 64) * x_eb) & ~3))}};
        const int tw[1][2] = {{eh->Tqt[c * kD + lane], eh->Tqt[c * kD + lane + 64]}};
        const float isv[1] = {eh->inv_s[c]};
        float rc[1], ec[1];
        append_coefficients<1>(xw, tw, a.x_dtype, isv, rc, ec);
        if (lane == 0) buf_store4_coherent(rc[0], rrs, (uint32_t)(4 * d));
        if (c == 0 && lane == 0) buf_store4_coherent(ec[0], rrs, (uint32_t)(4 * (2 * kD + d / kD)));
      }
    }
  }
  // (7) Partial: o~_c = s_c 2^(1-b_c-fv) (sum_{k < b-1} 2^k O'(c,k) - 2^(b-1) O'(c,b-1)),
  //     one (head, channel) per thread; midrise adds s_c 2^(-b_c) sum_i P_i alpha^V_i
  //     (the half step of every level).
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int h = (r * NTHR + tid) / kD;
    if (h < G) {
      const float* oh = ob + h * a.ob_stride;
      float acc = 0.f;
      auto bit_term = [&](int k) {
        const int v = min(voc + k, 8 * RV - 1);
        const float t = ldexpf(kHalves ? oh[v] + oh[NH * a.ob_stride + v] : oh[v], k);
        acc += (k < vbc) ? ((k == vbc - 1) ? -t : t) : 0.f;
      };
      // (the first eight bits unrolled with their reads issued together; wider codes take
      // the loop after)
#pragma unroll
      for (int k = 0; k < 8; ++k) bit_term(k);
      for (int k = 8; k < v_maxb; ++k) bit_term(k);
      float pa = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) pa += wpav[w][h];
      const float o = vbc ? fmaf(vsc * vhs, pa, ldexpf(vsc * acc, 1 - vbc - fv_s[h])) : 0.f;
      buf_store4_coherent(o, prs, (uint32_t)((split * G + h) * sizeof(Partial) + 16 + 4 * cq));
    }
  }
  if (tid < G) {
    float m = wmax[0][tid], l = wsum[0][tid];
#pragma unroll
    for (int w = 1; w < NW; ++w) {
      m = fmaxf(m, wmax[w][tid]);
      l += wsum[w][tid];
    }
    buf_store16_coherent((v4f){layout_ok ? m : NAN, l, 0.f, 0.f}, prs,
                         (uint32_t)((split * G + tid) * sizeof(Partial)));
  }
  // The merge's scratch: from the start of the front region (its cache and O' are consumed).
  float* merge_scratch = reinterpret_cast<float*>(smem);
  if constexpr (APPEND) {
    AppendHook<NTHR, NH> hook;
    hook.coeff = a.append_r + row * kAppStride;
    hook.ehp[0] = hk;
    hook.ehp[1] = hv;
    hook.xrow[0] = static_cast<const uint8_t*>(a.x_k) + row * kD * x_eb;
    hook.xrow[1] = static_cast<const uint8_t*>(a.x_v) + row * kD * x_eb;
    hook.x_dtype = a.x_dtype;
    hook.k_codes = a.k_codes;
    hook.k_alpha = a.k_alpha;
    hook.v_codes = a.v_codes;
    hook.v_alpha = a.v_alpha;
    hook.row = row;
    hook.cap = a.cap;
    hook.len = len;
    hook.G = G;
    hook.rk = RK;
    hook.rv = RV;
    hook.on = len > 0;
    hook.e_mr = e_mr;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      hook.e_b[i] = e_b[i];
      hook.e_off[i] = e_off[i];
      hook.e_s[i] = e_s[i];
#pragma unroll
      for (int h = 0; h < NH; ++h) hook.qk[i][h] = qk[i][h];
    }
    hook.sc = reinterpret_cast<AppendScratch*>(smem + a.off_es);
    merge_if_last_wide<NTHR, NH, kTvHeld>(a.params_v, kvh, row, G, a.n_splits, a.partials,
                                          a.counters, out_rows, merge_scratch, tv, hook);
  } else if (a.seg) {
    SegHook sh{a.seg + row * G};
    merge_if_last_wide<NTHR, NH, kTvHeld>(a.params_v, kvh, row, G, a.n_splits, a.partials,
                                          a.counters, out_rows, merge_scratch, tv, sh);
  } else {
    NoHook none;
    merge_if_last_wide<NTHR, NH, kTvHeld>(a.params_v, kvh, row, G, a.n_splits, a.partials,
                                          a.counters, out_rows, merge_scratch, tv, none);
  }
}

}  // namespace

size_t decode_workspace_bytes(int batch, int n_q_heads, int n_kv_heads, int64_t cap,
                              int counter_rows) {
  return ws_layout(batch, n_q_heads, n_kv_heads, cap, counter_rows).total;
}

// The dynamic LDS limit of one kernel, raised on each device the first time a launch there
// needs more.  Safe for concurrent callers: a race can only repeat the (idempotent)
// attribute call, and the recorded limit only grows.
class LdsLimit {
 public:
  bool ensure(const void* kernel, size_t lds) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return false;
    if (dev < 0 || dev >= kDevices)      // beyond the table: set it every time
      return hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)lds) == hipSuccess;
    size_t cur = set_[dev].load(std::memory_order_acquire);
    if (lds <= cur) return true;
    if (hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
        hipSuccess)
      return false;
    while (cur < lds && !set_[dev].compare_exchange_weak(cur, lds, std::memory_order_acq_rel)) {
    }
    return true;
  }

 private:
  static constexpr int kDevices = 64;
  std::atomic<size_t> set_[kDevices] = {};
};

template <int NT, int NTILE, int NP, int NW, bool APPEND>
static aatc_status launch_mfma(DecodeArgs a, int batch, hipStream_t st) {
  constexpr int NH = 4 * NT, NTHR = 64 * NW, S = NW * 16 * NTILE;
  a.n_splits = (int)((a.cap + S - 1) / S);
  const int64_t rows = (int64_t)batch * a.n_kv_heads;
  if (rows * a.n_splits > (1 << 30)) return AATC_E_UNSUPPORTED;
  a.n_blocks = (int)(rows * a.n_splits);
  // LDS: key records | value tiles | alpha^K | alpha^V   (front, also the query-transform
  // and merge scratch) | query limb planes | value operands | [O' if it does not fit
  // over the key records].
  // Eight waves: the cache streams into LDS while the query planes are built, so their
  // scratch shares the value-operand region (written only after the planes) instead of
  // the cache region.  The transfers write whole 1 KiB blocks of the cache regions.
  constexpr bool DMA = NW == 8;
  constexpr int NJQ = (DMA ? NTHR / 2 : NTHR) / 32;
  const size_t scr_bytes = (size_t)(NJQ + 1) * NH * kD * sizeof(float);
  if (DMA && (((size_t)S * a.rk) % 1024 || ((size_t)S * a.rv) % 1024 || (2 * S) % 1024))
    return AATC_E_UNSUPPORTED;
  a.off_v = S * a.rk;
  a.off_ak = a.off_v + S * a.rv;
  a.off_av = a.off_ak + 2 * S;
  size_t front = (size_t)a.off_av + 2 * S;
  if (!DMA) front = std::max(front, scr_bytes);
  front = std::max(front, wide_merge_lds_bytes<NTHR, NH>());
  front = round256(front);
  a.off_ql = (int)front;
  a.off_pb = a.off_ql + 4 * NH * 2 * NP * 64;
  size_t pb_bytes = (size_t)(S / 64) * NT * 64 * 16;
  if (DMA) pb_bytes = std::max(pb_bytes, scr_bytes);
  size_t off = (size_t)a.off_pb + pb_bytes;
  a.ob_stride = 8 * a.rv;
  // O' per (head, value bit); eight waves keep one copy per chunk half.
  const size_t ob_bytes = (size_t)(NW == 8 && S % 128 == 0 ? 2 : 1) * NH * a.ob_stride * 4;
  const size_t es_bytes = APPEND ? (sizeof(AppendScratch) + 15) / 16 * 16 : 0;
  constexpr size_t kLdsMax = 160 * 1024 - 4 * 1024;
  if (ob_bytes <= (size_t)S * a.rk) {
    a.off_ob = 0;
  } else {
    a.off_ob = (int)off;
    off += ob_bytes;
  }
  a.off_es = (int)off;
  off += es_bytes;
  const size_t lds = off;
  if (lds > kLdsMax) return AATC_E_UNSUPPORTED;
  static LdsLimit limit;
  if (!limit.ensure((const void*)decode_mfma_kernel<NT, NTILE, NP, NW, APPEND>, lds))
    return AATC_E_DEVICE;
  const unsigned grid = (unsigned)a.n_blocks;
  hipLaunchKernelGGL((decode_mfma_kernel<NT, NTILE, NP, NW, APPEND>), dim3(grid), dim3(NTHR), lds,
                     st, a);
  return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
}

template <int NT, int NTILE, int NW, bool APPEND>
static aatc_status launch_mfma_np(const DecodeArgs& a, int batch, hipStream_t st) {
  switch ((a.rk / 4 + 3) / 4) {
    case 1: return launch_mfma<NT, NTILE, 1, NW, APPEND>(a, batch, st);
    case 2: return launch_mfma<NT, NTILE, 2, NW, APPEND>(a, batch, st);
    case 3: return launch_mfma<NT, NTILE, 3, NW, APPEND>(a, batch, st);
    default: return launch_mfma<NT, NTILE, 4, NW, APPEND>(a, batch, st);
  }
}

// Split size: 1024 tokens on eight waves while that still gives every compute unit a
// workgroup (and always with a fused append), else 512 on four; records over 96 bytes in
// all halve both (LDS).
template <int NT>
static aatc_status launch_mfma_nt(const DecodeArgs& a, int batch, hipStream_t st) {
  const bool big = a.rk + a.rv > 96;
  if (a.x_k) return big ? launch_mfma_np<NT, 4, 8, true>(a, batch, st)
                        : launch_mfma_np<NT, 8, 8, true>(a, batch, st);
  const int64_t rows = (int64_t)batch * a.n_kv_heads;
  const int64_t wide = rows * ((a.cap + (big ? 511 : 1023)) / (big ? 512 : 1024));
  if (wide >= 256) return big ? launch_mfma_np<NT, 4, 8, false>(a, batch, st)
                              : launch_mfma_np<NT, 8, 8, false>(a, batch, st);
  return big ? launch_mfma_np<NT, 4, 4, false>(a, batch, st)
             : launch_mfma_np<NT, 8, 4, false>(a, batch, st);
}

aatc_status launch_decode(const void* params_k, const void* params_v, int batch,
                          int n_q_heads, int n_kv_heads, const void* q, aatc_dtype q_dtype,
                          const void* k_codes, const uint16_t* k_alpha, const void* v_codes,
                          const uint16_t* v_alpha, const int32_t* seq_len, int64_t cap,
                          int rk, int rv, float softmax_scale, float* out, void* workspace,
                          void* stream, const void* x_k, const void* x_v, aatc_dtype x_dtype,
                          int counter_rows, const void* seg_k, const void* seg_v,
                          aatc_dtype seg_dtype, const int32_t* seg_len, int seg_cap) {
  const int G = n_q_heads / n_kv_heads;
  const WsLayout wl = ws_layout(batch, n_q_heads, n_kv_heads, cap, counter_rows);
  char* ws = static_cast<char*>(workspace);
  auto* ctr = reinterpret_cast<unsigned*>(ws + wl.counters);
  auto* parts = reinterpret_cast<Partial*>(ws + wl.partials);
  const hipStream_t st = (hipStream_t)stream;
  // Buffer descriptors address at most 2^31 bytes of one (sequence, KV head).
  if (cap * std::max(rk, rv) >= ((int64_t)1 << 31)) return AATC_E_UNSUPPORTED;
  if ((cap / kMinSplit + 1) * G * (int64_t)sizeof(Partial) >= ((int64_t)1 << 31))
    return AATC_E_UNSUPPORTED;
  // The full-precision segment's partials first (stream order makes them visible to the
  // merging workgroups of the launch below).
  const Partial* seg = nullptr;
  if (seg_k) {
    if (seg_cap > kSegMax || x_k) return AATC_E_UNSUPPORTED;
    Partial* sp = reinterpret_cast<Partial*>(ws + wl.seg);
    hipLaunchKernelGGL(segment_partial_kernel, dim3((unsigned)(batch * n_kv_heads)),
                       dim3(kSegThreads), 0, st, params_v, n_q_heads, n_kv_heads, q,
                       (int)q_dtype, seg_k, seg_v, (int)seg_dtype, seg_len, seg_cap,
                       softmax_scale * kLog2e, sp);
    if (hipGetLastError() != hipSuccess) return AATC_E_DEVICE;
    seg = sp;
  }
  if (G <= kMaxNH && rk <= 64 && rv <= 64) {
    DecodeArgs a{};
    a.params_k = params_k;
    a.params_v = params_v;
    a.q = q;
    a.k_codes = static_cast<uint8_t*>(const_cast<void*>(k_codes));
    a.k_alpha = const_cast<uint16_t*>(k_alpha);
    a.v_codes = static_cast<uint8_t*>(const_cast<void*>(v_codes));
    a.v_alpha = const_cast<uint16_t*>(v_alpha);
    a.seq_len = seq_len;
    a.x_k = x_k;
    a.x_v = x_v;
    a.x_dtype = (int)x_dtype;
    a.out = out;
    a.counters = ctr;
    a.partials = parts;
    a.append_r = reinterpret_cast<float*>(ws + wl.append_r);
    a.seg = seg;
    a.cap = cap;
    a.n_q_heads = n_q_heads;
    a.n_kv_heads = n_kv_heads;
    a.G = G;
    a.q_dtype = (int)q_dtype;
    a.rk = rk;
    a.rv = rv;
    a.scale_log2e = softmax_scale * kLog2e;
    return G <= 4 ? launch_mfma_nt<1>(a, batch, st) : launch_mfma_nt<2>(a, batch, st);
  }
  if (x_k) {                // generic path: append with the per-token encode kernel first
    aatc_status e = launch_encode_last(params_k, n_kv_heads, batch, x_k, x_dtype,
                                       AATC_LAYOUT_RECORDS, const_cast<void*>(k_codes),
                                       const_cast<uint16_t*>(k_alpha), cap, rk, seq_len, stream);
    if (e == AATC_OK)
      e = launch_encode_last(params_v, n_kv_heads, batch, x_v, x_dtype, AATC_LAYOUT_TILES,
                             const_cast<void*>(v_codes), const_cast<uint16_t*>(v_alpha), cap, rv,
                             seq_len, stream);
    if (e != AATC_OK) return e;
  }
  const int n_splits = (int)((cap + kSplit - 1) / kSplit);
  size_t lds = std::max((size_t)G * (kSplit + 8 * std::max(rk, rv)) * sizeof(float),
                        merge_lds_bytes(G, kThreads));
  if (lds > 160 * 1024 - 24 * 1024) return AATC_E_UNSUPPORTED;
  static LdsLimit limit;
  if (!limit.ensure((const void*)decode_split_kernel, lds)) return AATC_E_DEVICE;
  dim3 grid((unsigned)n_splits, (unsigned)n_kv_heads, (unsigned)batch);
  hipLaunchKernelGGL(decode_split_kernel, grid, dim3(kThreads), lds, st, params_k, params_v,
                     n_q_heads, n_kv_heads, q, (int)q_dtype,
                     static_cast<const uint8_t*>(k_codes), k_alpha,
                     static_cast<const uint8_t*>(v_codes), v_alpha, seq_len, cap,
                     softmax_scale, out, ctr, parts, n_splits, rk, rv, seg);
  return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
}

}  // namespace aatc
