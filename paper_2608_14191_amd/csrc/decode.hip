// AATC decode attention on gfx950 (Algorithm 1, inference part, evaluated in the
// transformed domain of App. B: q~ = T_K^T q; the inverse transform T_V is applied once
// to each output).
//
// Grid: (token split, KV head, sequence).  Each workgroup scores its split's tokens for
// the G query heads of its KV head, runs a split-local softmax and accumulates the
// value codes into a partial (m, l, o~).  The last workgroup of each (sequence, KV
// head) to finish merges the partials and applies T_V.
//
// Two kernels share that structure:
//  * decode_mfma_kernel: G <= 8 and budgets <= 512 bits per token; both contractions
//    on int8 MFMA over the bits of the packed codes (see the comment above it);
//  * decode_split_kernel: any G <= 16 and budget; plain VALU.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <algorithm>

#include "launch.h"
#include "params.h"

namespace aatc {
namespace {

constexpr int kDecThreads = 256;
constexpr int kSplit = 512;                      // tokens per workgroup, generic kernel
constexpr int kMinSplit = 256;                   // smallest split of either kernel
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kMaxPairs = 4;     // record dword quads per key record (<= 512 bits)
constexpr int kMaxNH = 8;        // head slots of the MFMA kernel (G <= 8)
constexpr int kSpinLimit = 1000; // polls (~0.3 us each) for the published query planes

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

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
  for (int i = 1; i < kDecThreads / 64; ++i) r = is_max ? fmaxf(r, scratch[i]) : r + scratch[i];
  return r;
}

struct alignas(16) Partial {   // per (sequence, KV head, split, head-in-group)
  float m;                     // split max of the log2-domain logits
  float l;                     // sum of 2^(z - m)
  float pad_[2];
  float o[kD];                 // sum of 2^(z - m) h^V (transformed domain, storage channels)
};

// Query bit weights of one (sequence, KV head), published by split 0 of the MFMA kernel.
struct alignas(256) QPlanes {
  uint8_t ql[4 * kMaxNH * 2 * kMaxPairs * 64];   // [limb][head][K-step][64 bytes]
  int cofs[kMaxNH][4];                           // key offset per head and limb
  int fexp[kMaxNH];                              // fixed-point exponent per head
};

struct WsLayout {
  size_t counters, flags, planes, partials, total;
};

__host__ __device__ inline size_t round256(size_t x) { return (x + 255) / 256 * 256; }

__host__ __device__ inline WsLayout ws_layout(int batch, int n_q_heads, int n_kv_heads,
                                              int64_t cap) {
  const size_t rows = (size_t)batch * n_kv_heads;
  const size_t n_splits = (size_t)((cap + kMinSplit - 1) / kMinSplit);
  WsLayout w;
  w.counters = 0;
  w.flags = round256(rows * sizeof(unsigned));
  w.planes = w.flags + round256(rows * sizeof(unsigned));
  w.partials = w.planes + rows * sizeof(QPlanes);
  w.total = w.partials + (size_t)batch * n_q_heads * n_splits * sizeof(Partial);
  return w;
}

// Device-coherent accesses: relaxed agent-scope atomics are performed at the level all
// compute units of the device see (they bypass the per-XCD L2), so publishing a few
// values costs neither an L2 writeback nor an invalidate.
__device__ inline void st_dev(float* p, float v) {
  __hip_atomic_store(reinterpret_cast<unsigned*>(p), __float_as_uint(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void st_dev(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline unsigned ld_dev(const unsigned* p) {
  return __hip_atomic_load(const_cast<unsigned*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Called by every workgroup after it stored its partial (m, l, o~) with st_dev.  The
// last workgroup of a (sequence, KV head) to arrive merges the split partials of its G
// query heads and applies the inverse transform o = T_V o~ / l; it also resets the
// arrival counter and the query-plane flag for the next call.  `lds` must hold
// (9 G + 4) kD + 4 kDecThreads floats.
__device__ void merge_if_last(const void* params_v, int n_q_heads, int kvh, int seq,
                              int64_t kv_row, int G, float* out, unsigned* counters,
                              unsigned* flags, const Partial* partials, int n_splits,
                              float* lds) {
  __shared__ unsigned last_flag;
  __shared__ float mm[kMaxGroup], ll[kMaxGroup];
  const int tid = threadIdx.x;
  __builtin_amdgcn_s_waitcnt(0);          // this thread's partial stores have completed
  __syncthreads();
  if (tid == 0) {
    const unsigned prev = __hip_atomic_fetch_add(&counters[kv_row], 1u, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
    last_flag = (prev == (unsigned)n_splits - 1u) ? 1u : 0u;
  }
  __syncthreads();
  if (!last_flag) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");   // drop stale lines of this L2 once

  const HeadParams* hv = head_params(params_v, kvh);
  const Partial* all = partials + kv_row * n_splits * G;
  float* osum = lds;                                       // [G][kD]
  v4f* part4 = reinterpret_cast<v4f*>(osum + G * kD);      // [kDecThreads]
  float* ored = reinterpret_cast<float*>(part4 + kDecThreads);  // [8][G][kD]
  // (a) T_V rows 4 j4 .. 4 j4 + 3, columns 16 cq .. 16 cq + 15: 16 vector loads per
  //     thread, issued before the partials are read.
  const int j4 = tid & 31, cq = tid >> 5;
  v4f tr[4][4];
#pragma unroll
  for (int jj = 0; jj < 4; ++jj)
#pragma unroll
    for (int k = 0; k < 4; ++k)
      tr[jj][k] = reinterpret_cast<const v4f*>(hv->T)[(4 * j4 + jj) * (kD / 4) + 4 * cq + k];
  // (b) global max and normalizer per head
  if (tid < G) {
    float m = -INFINITY;
    for (int s = 0; s < n_splits; ++s) m = fmaxf(m, all[s * G + tid].m);
    float l = 0.f;
    for (int s = 0; s < n_splits; ++s) {
      const float ms = all[s * G + tid].m;
      l += (ms == -INFINITY) ? 0.f : exp2f(ms - m) * all[s * G + tid].l;
    }
    mm[tid] = m;
    ll[tid] = l;
  }
  __syncthreads();
  // (c) o~ = sum_s 2^(m_s - m) o~_s / l over float4 columns; the splits are strided
  // over thread groups when the columns do not fill the workgroup.
  const int slots = G * (kD / 4);
  for (int base = 0; base < slots; base += kDecThreads) {
    const int width = min(slots - base, kDecThreads);
    const int ngroups = kDecThreads / width;
    const int slot = base + tid % width, grp = tid / width;
    if (grp < ngroups) {
      const int h = slot / (kD / 4), c4 = slot % (kD / 4);
      const float m = mm[h];
      v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 16
      for (int s = grp; s < n_splits; s += ngroups) {
        const float ms = all[s * G + h].m;
        const float w = (ms == -INFINITY) ? 0.f : exp2f(ms - m);
        acc += w * reinterpret_cast<const v4f*>(all[s * G + h].o)[c4];
      }
      part4[tid] = acc;
    }
    __syncthreads();
    if (tid < width) {
      const int h = (base + tid) / (kD / 4), c4 = (base + tid) % (kD / 4);
      v4f acc = part4[tid];
      for (int g = 1; g < ngroups; ++g) acc += part4[g * width + tid];
      const float inv_l = ll[h] > 0.f ? 1.f / ll[h] : 0.f;
      reinterpret_cast<v4f*>(osum)[h * (kD / 4) + c4] = acc * inv_l;
    }
    __syncthreads();
  }
  // (d) o_j = sum_c T_V[j][c] o~_c: partial sums over this thread's 16 columns, then
  //     over the 8 column blocks.
  for (int h = 0; h < G; ++h) {
    const v4f* oh = reinterpret_cast<const v4f*>(osum + h * kD) + 4 * cq;
    const v4f o0 = oh[0], o1 = oh[1], o2 = oh[2], o3 = oh[3];
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const v4f p = tr[jj][0] * o0 + tr[jj][1] * o1 + tr[jj][2] * o2 + tr[jj][3] * o3;
      ored[(cq * G + h) * kD + 4 * j4 + jj] = p.x + p.y + p.z + p.w;
    }
  }
  __syncthreads();
  for (int i = tid; i < G * kD; i += kDecThreads) {
    const int h = i / kD, j = i % kD;
    float acc = 0.f;
#pragma unroll
    for (int b = 0; b < 8; ++b) acc += ored[(b * G + h) * kD + j];
    out[((int64_t)seq * n_q_heads + kvh * G + h) * kD + j] = acc;
  }
  if (tid == 0) {
    counters[kv_row] = 0u;
    flags[kv_row] = 0u;
  }
}

// ---------------------------------------------------------------------------------------
// Generic VALU kernel (any G <= 16, any budget).
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(kDecThreads) void decode_split_kernel(
    const void* __restrict__ params_k, const void* __restrict__ params_v, int n_q_heads,
    int n_kv_heads, const void* __restrict__ q, int q_dtype,
    const uint8_t* __restrict__ k_codes, const uint16_t* __restrict__ k_alpha,
    const uint8_t* __restrict__ v_codes, const uint16_t* __restrict__ v_alpha,
    const int32_t* __restrict__ seq_len, int64_t cap, float scale, float* __restrict__ out,
    unsigned* __restrict__ counters, unsigned* __restrict__ flags,
    Partial* __restrict__ partials, int n_splits, int rk, int rv) {
  extern __shared__ float dyn[];
  __shared__ float qs[kMaxGroup][kD];
  __shared__ float qp[kMaxGroup][kD];
  __shared__ float cterm[kMaxGroup];
  __shared__ float red[kDecThreads / 64];
  __shared__ float mh[kMaxGroup], lh[kMaxGroup], pah[kMaxGroup];

  const int split = blockIdx.x, kvh = blockIdx.y, seq = blockIdx.z;
  const int G = n_q_heads / n_kv_heads;
  const int tid = threadIdx.x;
  const HeadParams* hk = head_params(params_k, kvh);
  const HeadParams* hv = head_params(params_v, kvh);
  const bool layout_ok = hk->record_bytes == rk && hv->record_bytes == rv;
  const int bk = hk->budget, bv = hv->budget;
  float* sc = dyn;                                  // [G][kSplit] logits, then weights
  float* vq = dyn + G * kSplit;                     // [G][kMaxBudget] per-bit weights / sums

  const int len = (int)min<int64_t>(max(seq_len[seq], 0), cap);   // out-of-range lengths clamp
  const int t0 = split * kSplit;
  const int nt = layout_ok ? max(0, min(kSplit, len - t0)) : 0;

  // Queries of the group, then q'_c = (T_K^T q)_c * s_c * 2^(1-b_c) * scale * log2(e).
  for (int i = tid; i < G * kD; i += kDecThreads)
    qs[i / kD][i % kD] = load_q(q, q_dtype, ((int64_t)seq * n_q_heads + kvh * G) * kD + i);
  __syncthreads();
  for (int i = tid; i < G * kD; i += kDecThreads) {
    const int h = i / kD, c = i % kD;
    float acc = 0.f;
#pragma unroll 16
    for (int j = 0; j < kD; ++j) acc += hk->T[j * kD + c] * qs[h][j];
    const int b = hk->bits[c];
    qp[h][c] = b ? acc * hk->s[c] * ldexpf(1.f, 1 - b) * scale * kLog2e : 0.f;
  }
  __syncthreads();
  if (tid < G) {
    float acc = 0.f;
    for (int c = 0; c < kD; ++c)
      if (hk->bits[c]) acc += qp[tid][c] * ldexpf(1.f, hk->bits[c] - 1);
    cterm[tid] = acc;
  }
  for (int i = tid; i < G * bk; i += kDecThreads) {
    const int h = i / bk, v = i % bk;
    vq[h * kMaxBudget + v] = ldexpf(qp[h][hk->virt_chan[v]], hk->virt_bit[v]);
  }
  __syncthreads();

  // Scores z = alpha^K (sum_v Q_v bit_v - C) in the log2 domain.
  const int64_t kv_row = (int64_t)seq * n_kv_heads + kvh;
  for (int tl = tid; tl < kSplit; tl += kDecThreads) {
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
            if (h < G) acc[h] += vq[h * kMaxBudget + v];
        }
      }
      const float ak = half_bits_to_float(k_alpha[kv_row * cap + t]);
#pragma unroll
      for (int h = 0; h < kMaxGroup; ++h)
        if (h < G) sc[h * kSplit + tl] = ak * (acc[h] - cterm[h]);
    } else {
      for (int h = 0; h < G; ++h) sc[h * kSplit + tl] = -INFINITY;
    }
  }
  __syncthreads();

  // Split-local softmax statistics per head; weights become 2^(z - m) * alpha^V.
  for (int h = 0; h < G; ++h) {
    float m = -INFINITY;
    for (int tl = tid; tl < kSplit; tl += kDecThreads) m = fmaxf(m, sc[h * kSplit + tl]);
    m = block_reduce(m, true, red);
    float l = 0.f, pa = 0.f;
    for (int tl = tid; tl < kSplit; tl += kDecThreads) {
      float p = (tl < nt) ? exp2f(sc[h * kSplit + tl] - m) : 0.f;
      float w = (tl < nt) ? p * half_bits_to_float(v_alpha[kv_row * cap + t0 + tl]) : 0.f;
      sc[h * kSplit + tl] = w;
      l += p;
      pa += w;
    }
    l = block_reduce(l, false, red);
    pa = block_reduce(pa, false, red);
    if (tid == 0) {
      mh[h] = m;
      lh[h] = l;
      pah[h] = pa;
    }
  }
  __syncthreads();

  // Value bits: sum over tokens of w_t * bit_v(t), one thread per record bit.
  const uint32_t* vt = reinterpret_cast<const uint32_t*>(v_codes) +
                       (kv_row * (cap / kTile) + t0 / kTile) * (16 * rv);
  for (int v = tid; v < bv; v += kDecThreads) {
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
      if (h < G) vq[h * kMaxBudget + v] = acc[h];
  }
  __syncthreads();

  // Partial o~_c = s_c 2^(1-b_c) (sum_k 2^k S_(c,k) - 2^(b_c-1) sum_t w_t).
  Partial* part = partials + (kv_row * n_splits + split) * G;
  for (int i = tid; i < G * kD; i += kDecThreads) {
    const int h = i / kD, c = i % kD;
    const int b = hv->bits[c];
    float o = 0.f;
    if (b && nt > 0) {
      float acc = 0.f;
      for (int k = 0; k < b; ++k) acc += ldexpf(vq[h * kMaxBudget + hv->bit_off[c] + k], k);
      o = hv->s[c] * ldexpf(1.f, 1 - b) * (acc - ldexpf(pah[h], b - 1));
    }
    st_dev(&part[h].o[c], o);
  }
  if (tid < G) {
    st_dev(&part[tid].m, !layout_ok ? NAN : (nt > 0) ? mh[tid] : -INFINITY);
    st_dev(&part[tid].l, !layout_ok ? NAN : (nt > 0) ? lh[tid] : 0.f);
  }
  merge_if_last(params_v, n_q_heads, kvh, seq, kv_row, G, out, counters, flags, partials,
                n_splits, dyn);
}

// ---------------------------------------------------------------------------------------
// MFMA decode kernel (G <= 8 query heads per KV head, record budgets <= 512 bits).
//
// Both contractions run on v_mfma_i32_16x16x64_i8 over the bits of the codes: a code
// u_c = sum_k 2^k bit_k, so every record bit is a virtual channel whose weight is the
// channel's weight times 2^k.
//  * Keys: D[token, (head, limb)] = sum_bits bit(token) * Qlimb[bit, (head, limb)].
//    One record dword w (32 bits of one token) expands to MFMA bytes by
//    r_d = w & (0x01010101 << d): byte j of r_d is 2^d * bit (8j + d).  The factor 2^d
//    (and the sign of int8 0x80 for d = 7) is folded into the query weights, which are
//    32-bit fixed point split into four int8 limbs: four heads times four limbs fill
//    the 16 MFMA columns.  Lane (column (h, L), row group g) of the result holds limb L
//    of the scores of tokens 4g .. 4g + 3; a DPP sum over the lane quad recombines the
//    limbs.
//  * Values: D[bit, (head, limb)] = sum_tokens bit(token) * Plimb[token, (head, limb)]
//    with P = 2^(z - m) alpha^V in 32-bit fixed point.  The value tiles store the bit of
//    token 16 d + 4 g + i at bit 8 i + 2 g + d % 2 of word d / 2, so a lane of row
//    group g expands its two words with two masks into exactly the tokens whose
//    scores it computed: each lane's softmax weights are its own MFMA operand.
// The four waves of a workgroup work on disjoint quarters of the split and meet once,
// to combine their (m, l, o~) into the workgroup partial.  Integer accumulation is
// exact; limbs are recombined in fp32.
//
// The query bit weights of a (sequence, KV head) are computed once, by the workgroup
// of split 0, and published in the workspace; the other splits poll a flag a bounded
// number of times while their cache loads are in flight, and compute the weights
// themselves if the flag does not appear.
// ---------------------------------------------------------------------------------------
constexpr int kMaxLoads = 6;     // 16-byte loads per thread per cache region

__device__ inline v4i mfma_i8(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// Four balanced int8 limbs of a 32-bit value |x| < 2^30, packed in one dword (limb L in
// byte L, two's complement): x = sum_L limb_L 256^L.
__device__ inline uint32_t pack_limbs(int x) {
  return ((uint32_t)x + 0x80808080u) ^ 0x80808080u;
}

// Sum over the lane quad (lanes 4k .. 4k + 3); every lane of the quad gets the sum.
__device__ inline float quad_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
  return v;
}

// Query bit weights in MFMA operand order (limb planes), their offsets C and exponents,
// into LDS.  scratch: >= 8 * NH * kD floats of LDS not otherwise in use.
template <int NH>
__device__ void query_planes(const HeadParams* hk, const void* q, int q_dtype, int64_t qbase,
                             int G, float scale, int BK, int NP, float* scratch, uint8_t* ql,
                             int (*cofs)[4], int* fexp) {
  __shared__ float qs[NH][kD];
  __shared__ float qp[NH][kD];
  __shared__ unsigned qmax_bits[NH];
  __shared__ uint8_t tbits[kD];
  __shared__ float tscale[kD];
  __shared__ uint8_t vchan[kMaxBudget / 2], vbit[kMaxBudget / 2];
  const int tid = threadIdx.x;
  const int c4 = tid & 31, jq = tid >> 5;
  // One round of loads: T rows 16 jq .. 16 jq + 15 (columns 4 c4 ..), q, small tables.
  v4f tr[16];
  const v4f* t4 = reinterpret_cast<const v4f*>(hk->T);
#pragma unroll
  for (int jj = 0; jj < 16; ++jj) tr[jj] = t4[(16 * jq + jj) * (kD / 4) + c4];
  for (int i = tid; i < NH * kD; i += kDecThreads) {
    const int h = i / kD;
    qs[h][i % kD] = (h < G) ? load_q(q, q_dtype, qbase + i) : 0.f;
  }
  for (int i = tid; i < BK; i += kDecThreads) {
    vchan[i] = hk->virt_chan[i];
    vbit[i] = hk->virt_bit[i];
  }
  if (tid < kD) {
    tbits[tid] = hk->bits[tid];
    tscale[tid] = hk->s[tid];
  }
  for (int i = tid; i < 4 * NH * 2 * NP * 64 / 4; i += kDecThreads)
    reinterpret_cast<uint32_t*>(ql)[i] = 0u;
  if (tid < NH) qmax_bits[tid] = 0u;
  if (tid < NH * 4) cofs[tid / 4][tid % 4] = 0;
  __syncthreads();
  {
    v4f acc[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) acc[h] = (v4f){0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int jj = 0; jj < 16; ++jj)
#pragma unroll
      for (int h = 0; h < NH; ++h) acc[h] += tr[jj] * qs[h][16 * jq + jj];
#pragma unroll
    for (int h = 0; h < NH; ++h)
      reinterpret_cast<v4f*>(scratch)[(jq * NH + h) * (kD / 4) + c4] = acc[h];
  }
  __syncthreads();
  for (int i = tid; i < NH * kD; i += kDecThreads) {
    const int h = i / kD, c = i % kD;
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) acc += scratch[(j * NH + h) * kD + c];
    const int b = tbits[c];
    float qv = 0.f;
    if (h < G && b) {
      qv = acc * tscale[c] * ldexpf(1.f, 1 - b) * scale * kLog2e;
      atomicMax(&qmax_bits[h], __float_as_uint(ldexpf(fabsf(qv), b - 1)));
    }
    qp[h][c] = qv;
  }
  __syncthreads();
  if (tid < NH) {
    int e = 0;
    frexpf(__uint_as_float(qmax_bits[tid]), &e);
    fexp[tid] = qmax_bits[tid] ? 30 - e : 0;
  }
  __syncthreads();
  // Record bit v = 32 D + 8 j + d  ->  K-step 2 (D / 4) + d / 4, lane group D % 4,
  // byte 4 (d % 4) + j.  Weight 2^(k - d) q'_c, negated for d = 7 (int8 0x80 = -128).
  for (int i = tid; i < NH * BK; i += kDecThreads) {
    const int h = i / BK, v = i % BK;
    if (h >= G) continue;
    const int c = vchan[v], k = vbit[v];
    const int D = v >> 5, p = v & 31, j = p >> 3, d = p & 7;
    int fx = (int)rintf(ldexpf(qp[h][c], k - d + fexp[h]));
    if (d == 7) fx = -fx;
    const uint32_t limbs = pack_limbs(fx);
    const int s = 2 * (D >> 2) + (d >> 2);
    const int pos = ((D & 3) << 4) + ((d & 3) << 2) + j;
#pragma unroll
    for (int L = 0; L < 4; ++L)
      ql[((L * NH + h) * 2 * NP + s) * 64 + pos] = (uint8_t)(limbs >> (8 * L));
    if (k == tbits[c] - 1) {                    // offset C = sum_c Q(c, msb)
      const int bv = (d == 7) ? -128 : (1 << d);
#pragma unroll
      for (int L = 0; L < 4; ++L)
        atomicAdd(&cofs[h][L], (int)(int8_t)(limbs >> (8 * L)) * bv);
    }
  }
  __syncthreads();
}

template <int NT, int S>
__global__ __launch_bounds__(kDecThreads, 2) void decode_mfma_kernel(
    const void* __restrict__ params_k, const void* __restrict__ params_v, int n_q_heads,
    int n_kv_heads, const void* __restrict__ q, int q_dtype,
    const uint8_t* __restrict__ k_codes, const uint16_t* __restrict__ k_alpha,
    const uint8_t* __restrict__ v_codes, const uint16_t* __restrict__ v_alpha,
    const int32_t* __restrict__ seq_len, int64_t cap, float scale, float* __restrict__ out,
    unsigned* __restrict__ counters, unsigned* __restrict__ flags,
    QPlanes* __restrict__ planes, Partial* __restrict__ partials, int n_splits, int RK, int RV,
    int ob_base, int ob_wstride, int ql_base) {
  constexpr int NH = 4 * NT;          // head slots: 4 per column tile
  constexpr int TW = S / 4;           // tokens per wave
  constexpr int NTILE = TW / 16;      // 16-token key tiles per wave
  constexpr int NCH = TW / 64;        // 64-token value chunks per wave
  constexpr int VTP = 16 / NT;        // value-bit tiles per pass
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ int cofs_s[NH][4];
  __shared__ int fexp_s[NH];
  __shared__ unsigned ready;
  __shared__ float mw[4][NH], lw[4][NH];
  __shared__ double paw[4][NH];
  __shared__ float mfin[NH], lfin[NH], pafin[NH];

  const int G = n_q_heads / n_kv_heads;
  const int split = blockIdx.x, kvh = blockIdx.y, seq = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 15, g = lane >> 4, hc = n >> 2, L = n & 3;
  const HeadParams* hk = head_params(params_k, kvh);
  const HeadParams* hv = head_params(params_v, kvh);
  const int64_t kv_row = (int64_t)seq * n_kv_heads + kvh;
  const int len = (int)min<int64_t>(max(seq_len[seq], 0), cap);
  const int t0 = split * S;
  const int nt = max(0, min(S, len - t0));
  const int n_load = min(S, (nt + kTile - 1) / kTile * kTile);

  // Dynamic LDS: key records | value tiles | alpha^K | alpha^V | [Q limb planes]
  // [O' per wave, or inside each wave's own key records once they are consumed].
  // The front (records + tiles) also serves as prologue and merge scratch.
  uint8_t* kbuf = smem;
  uint8_t* vbuf = kbuf + S * RK + 16;
  uint16_t* akb = reinterpret_cast<uint16_t*>(vbuf + S * RV);
  uint16_t* avb = akb + S;
  uint8_t* ql = smem + ql_base;                                // [4][NH][2 NP][64]

  Partial* part = partials + (kv_row * n_splits + split) * G;
  const bool layout_ok = hk->record_bytes == RK && hv->record_bytes == RV;
  if (nt == 0 || !layout_ok) {
    for (int i = tid; i < G * kD; i += kDecThreads) st_dev(&part[i / kD].o[i % kD], 0.f);
    if (tid < G) {
      st_dev(&part[tid].m, layout_ok ? -INFINITY : NAN);
      st_dev(&part[tid].l, layout_ok ? 0.f : NAN);
    }
    merge_if_last(params_v, n_q_heads, kvh, seq, kv_row, G, out, counters, flags, partials,
                  n_splits, reinterpret_cast<float*>(smem));
    return;
  }
  const int BK = hk->budget, BV = hv->budget;
  const int RWK = RK / 4;
  const int NP = (RWK + 3) / 4;
  const int NVT = (BV + 15) / 16;

  // (1) Issue the loads of this split's packed cache (kept in registers for now).
  const v4i* gk = reinterpret_cast<const v4i*>(k_codes + (kv_row * cap + t0) * RK);
  const v4i* gv = reinterpret_cast<const v4i*>(v_codes + (kv_row * cap + t0) * RV);
  const int nk16 = n_load * RK / 16, nv16 = n_load * RV / 16, na16 = n_load * 2 / 16;
  v4i rk[kMaxLoads], rv[kMaxLoads], ra = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < kMaxLoads; ++i) rk[i] = rv[i] = (v4i){0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < kMaxLoads; ++i) {
    const int idx = tid + i * kDecThreads;
    if (idx < nk16) rk[i] = gk[idx];
  }
#pragma unroll
  for (int i = 0; i < kMaxLoads; ++i) {
    const int idx = tid + i * kDecThreads;
    if (idx < nv16) rv[i] = gv[idx];
  }
  {
    const uint16_t* src = (tid < 64) ? k_alpha : v_alpha;
    const int idx = tid & 63;
    if (tid < 128 && idx < na16)
      ra = reinterpret_cast<const v4i*>(src + kv_row * cap + t0)[idx];
  }

  // (2) Query operands (MFMA B for keys) while the loads are in flight.
  v4i bq[NT][2 * kMaxPairs];
  int cof[NT], fex[NT];
  bool have = false;
  QPlanes* qpl = planes + kv_row;
  if (split != 0) {
    if (tid == 0) {
      unsigned ok = 0u;
      for (int it = 0; it < kSpinLimit && !ok; ++it) {
        ok = ld_dev(&flags[kv_row]);
        if (!ok) __builtin_amdgcn_s_sleep(4);
      }
      ready = ok;
    }
    __syncthreads();
    have = ready != 0u;
    if (have) {
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) {
        const int h = 4 * rt + hc;
#pragma unroll
        for (int s = 0; s < 2 * kMaxPairs; ++s) {
          if (s < 2 * NP) {
            const unsigned* src = reinterpret_cast<const unsigned*>(
                qpl->ql + ((L * NH + h) * 2 * NP + s) * 64 + g * 16);
            bq[rt][s] = (v4i){(int)ld_dev(src), (int)ld_dev(src + 1), (int)ld_dev(src + 2),
                              (int)ld_dev(src + 3)};
          }
        }
        cof[rt] = (int)ld_dev(reinterpret_cast<const unsigned*>(&qpl->cofs[h][L]));
        fex[rt] = (int)ld_dev(reinterpret_cast<const unsigned*>(&qpl->fexp[h]));
      }
    }
  }
  if (!have) {
    query_planes<NH>(hk, q, q_dtype, ((int64_t)seq * n_q_heads + kvh * G) * kD, G, scale, BK,
                     NP, reinterpret_cast<float*>(smem), ql, cofs_s, fexp_s);
    if (split == 0) {
      const int words = 4 * NH * 2 * NP * 64 / 4;
      for (int i = tid; i < words; i += kDecThreads)
        st_dev(reinterpret_cast<int*>(qpl->ql) + i, reinterpret_cast<const int*>(ql)[i]);
      if (tid < NH * 4) st_dev(&qpl->cofs[tid / 4][tid % 4], cofs_s[tid / 4][tid % 4]);
      if (tid < NH) st_dev(&qpl->fexp[tid], fexp_s[tid]);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (tid == 0)
        __hip_atomic_store(&flags[kv_row], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
#pragma unroll
    for (int rt = 0; rt < NT; ++rt) {
      const int h = 4 * rt + hc;
#pragma unroll
      for (int s = 0; s < 2 * kMaxPairs; ++s)
        if (s < 2 * NP)
          bq[rt][s] = *reinterpret_cast<const v4i*>(ql + ((L * NH + h) * 2 * NP + s) * 64 + g * 16);
      cof[rt] = cofs_s[h][L];
      fex[rt] = fexp_s[h];
    }
    __syncthreads();                    // prologue scratch (the front) is reused below
  }

  // (3) Land the cache in LDS.
#pragma unroll
  for (int i = 0; i < kMaxLoads; ++i) {
    const int idx = tid + i * kDecThreads;
    if (idx < nk16) reinterpret_cast<v4i*>(kbuf)[idx] = rk[i];
  }
#pragma unroll
  for (int i = 0; i < kMaxLoads; ++i) {
    const int idx = tid + i * kDecThreads;
    if (idx < nv16) reinterpret_cast<v4i*>(vbuf)[idx] = rv[i];
  }
  if (tid < 128 && (tid & 63) < na16) reinterpret_cast<v4i*>(tid < 64 ? akb : avb)[tid & 63] = ra;
  __syncthreads();

  // (4) Key scores of this wave's tokens.
  const int wb = wave * TW;
  float z[NTILE][NT][4];
#pragma unroll
  for (int tt = 0; tt < NTILE; ++tt) {
    const int tok0 = wb + 16 * tt;
    const uint8_t* rec = kbuf + (tok0 + n) * RK;
    v4i acc[NT];
#pragma unroll
    for (int rt = 0; rt < NT; ++rt) acc[rt] = (v4i){0, 0, 0, 0};
#pragma unroll
    for (int P = 0; P < kMaxPairs; ++P) {
      if (P < NP) {
        const int D = 4 * P + g;
        const uint32_t w = (D < RWK) ? *reinterpret_cast<const uint32_t*>(rec + 4 * D) : 0u;
        const v4i a0 = {(int)(w & 0x01010101u), (int)(w & 0x02020202u),
                        (int)(w & 0x04040404u), (int)(w & 0x08080808u)};
        const v4i a1 = {(int)(w & 0x10101010u), (int)(w & 0x20202020u),
                        (int)(w & 0x40404040u), (int)(w & 0x80808080u)};
#pragma unroll
        for (int rt = 0; rt < NT; ++rt) {
          acc[rt] = mfma_i8(a0, bq[rt][2 * P], acc[rt]);
          acc[rt] = mfma_i8(a1, bq[rt][2 * P + 1], acc[rt]);
        }
      }
    }
    const uint2 akw = *reinterpret_cast<const uint2*>(akb + tok0 + 4 * g);
    const float ak[4] = {half_bits_to_float((uint16_t)(akw.x & 0xffff)),
                         half_bits_to_float((uint16_t)(akw.x >> 16)),
                         half_bits_to_float((uint16_t)(akw.y & 0xffff)),
                         half_bits_to_float((uint16_t)(akw.y >> 16))};
#pragma unroll
    for (int rt = 0; rt < NT; ++rt) {
      const bool head_ok = 4 * rt + hc < G;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float f = quad_sum(ldexpf((float)(acc[rt][i] - cof[rt]), 8 * L));
        z[tt][rt][i] = (tok0 + 4 * g + i < nt && head_ok) ? ak[i] * ldexpf(f, -fex[rt])
                                                          : -INFINITY;
      }
    }
  }

  // (5) Per-wave softmax: m, l, and the value-side operands P (fixed point, limb L).
  float av[NTILE][4];
  float am = 0.f;
#pragma unroll
  for (int tt = 0; tt < NTILE; ++tt) {
    const int tok0 = wb + 16 * tt;
    const uint2 avw = *reinterpret_cast<const uint2*>(avb + tok0 + 4 * g);
    av[tt][0] = half_bits_to_float((uint16_t)(avw.x & 0xffff));
    av[tt][1] = half_bits_to_float((uint16_t)(avw.x >> 16));
    av[tt][2] = half_bits_to_float((uint16_t)(avw.y & 0xffff));
    av[tt][3] = half_bits_to_float((uint16_t)(avw.y >> 16));
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (tok0 + 4 * g + i >= nt) av[tt][i] = 0.f;
      am = fmaxf(am, fabsf(av[tt][i]));
    }
  }
  am = fmaxf(am, __shfl_xor(am, 16, 64));
  am = fmaxf(am, __shfl_xor(am, 32, 64));
  int fv = 0;
  {
    int e = 0;
    frexpf(am, &e);
    fv = am > 0.f ? 30 - e : 0;    // P <= max alpha^V < 2^e, so P 2^fv < 2^30
  }
  uint32_t pdw[NT][NTILE];
#pragma unroll
  for (int rt = 0; rt < NT; ++rt) {
    float m = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < NTILE; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) m = fmaxf(m, z[tt][rt][i]);
    m = fmaxf(m, __shfl_xor(m, 16, 64));
    m = fmaxf(m, __shfl_xor(m, 32, 64));
    float lsum = 0.f;
    double pa = 0.0;
#pragma unroll
    for (int tt = 0; tt < NTILE; ++tt) {
      const int d = 2 * g + (tt & 1);     // bit of this lane's tokens inside the value bytes
      uint32_t dw = 0u;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = (z[tt][rt][i] == -INFINITY) ? 0.f : exp2f(z[tt][rt][i] - m);
        lsum += p;
        int fx = (int)rintf(ldexpf(p * av[tt][i], fv - d));
        pa += ldexp((double)fx, d);
        if (d == 7) fx = -fx;
        dw |= ((pack_limbs(fx) >> (8 * L)) & 0xffu) << (8 * i);
      }
      pdw[rt][tt] = dw;
    }
    lsum += __shfl_xor(lsum, 16, 64);
    lsum += __shfl_xor(lsum, 32, 64);
    pa += __shfl_xor(pa, 16, 64);
    pa += __shfl_xor(pa, 32, 64);
    if (g == 0 && L == 0) {
      mw[wave][4 * rt + hc] = m;
      lw[wave][4 * rt + hc] = lsum;
      paw[wave][4 * rt + hc] = ldexp(pa, -fv);
    }
  }

  // (6) Value bits x P limbs, in passes of VTP value-bit tiles.
  const uint32_t mask0 = 0x01010101u << (2 * g), mask1 = mask0 << 1;
  float* obw = reinterpret_cast<float*>(smem + ob_base + wave * ob_wstride);   // [NH][BV]
  for (int vb = 0; vb < NVT; vb += VTP) {
    v4i accv[VTP][NT];
#pragma unroll
    for (int k = 0; k < VTP; ++k)
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) accv[k][rt] = (v4i){0, 0, 0, 0};
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      v4i bp[NT];
#pragma unroll
      for (int rt = 0; rt < NT; ++rt)
        bp[rt] = (v4i){(int)pdw[rt][4 * c], (int)pdw[rt][4 * c + 1], (int)pdw[rt][4 * c + 2],
                       (int)pdw[rt][4 * c + 3]};
      const uint8_t* tile = vbuf + ((wb >> 6) + c) * (kTile * RV);
#pragma unroll
      for (int k = 0; k < VTP; ++k) {
        if (vb + k < NVT) {
          const int v = 16 * (vb + k) + n;
          const uint2 ww = *reinterpret_cast<const uint2*>(tile + 8 * v);
          const v4i a = {(int)(ww.x & mask0), (int)(ww.x & mask1), (int)(ww.y & mask0),
                         (int)(ww.y & mask1)};
#pragma unroll
          for (int rt = 0; rt < NT; ++rt) accv[k][rt] = mfma_i8(a, bp[rt], accv[k][rt]);
        }
      }
    }
    if (vb == 0) __builtin_amdgcn_wave_barrier();   // key records of this wave are consumed
#pragma unroll
    for (int k = 0; k < VTP; ++k) {
      if (vb + k < NVT) {
#pragma unroll
        for (int rt = 0; rt < NT; ++rt) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float f = quad_sum(ldexpf((float)accv[k][rt][i], 8 * L));
            const int v = 16 * (vb + k) + 4 * g + i;
            if (L == 0 && v < BV) obw[(4 * rt + hc) * BV + v] = ldexpf(f, -fv);
          }
        }
      }
    }
  }
  __syncthreads();

  // (7) Workgroup partial: merge the four waves, then per channel
  //     o~_c = s_c 2^(1-b_c) (sum_k 2^k O'(c,k) - 2^(b_c-1) sum_t P_t).
  if (tid < NH) {
    float m = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) m = fmaxf(m, mw[w][tid]);
    float l = 0.f;
    double pa = 0.0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float sw = (mw[w][tid] == -INFINITY) ? 0.f : exp2f(mw[w][tid] - m);
      l += sw * lw[w][tid];
      pa += (double)sw * paw[w][tid];
    }
    mfin[tid] = m;
    lfin[tid] = l;
    pafin[tid] = (float)pa;
  }
  __syncthreads();
  for (int i = tid; i < G * kD; i += kDecThreads) {
    const int h = i / kD, c = i % kD;
    const int b = hv->bits[c];
    float o = 0.f;
    if (b) {
      float sw[4];
#pragma unroll
      for (int w = 0; w < 4; ++w)
        sw[w] = (mw[w][h] == -INFINITY) ? 0.f : exp2f(mw[w][h] - mfin[h]);
      const int off = hv->bit_off[c];
      float acc = 0.f;
      for (int k = 0; k < b; ++k) {
        float ok = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w)
          ok += sw[w] * reinterpret_cast<const float*>(smem + ob_base + w * ob_wstride)[h * BV + off + k];
        acc += ldexpf(ok, k);
      }
      o = hv->s[c] * ldexpf(1.f, 1 - b) * (acc - ldexpf(pafin[h], b - 1));
    }
    st_dev(&part[h].o[c], o);
  }
  if (tid < G) {
    st_dev(&part[tid].m, mfin[tid]);
    st_dev(&part[tid].l, lfin[tid]);
  }
  __syncthreads();
  merge_if_last(params_v, n_q_heads, kvh, seq, kv_row, G, out, counters, flags, partials,
                n_splits, reinterpret_cast<float*>(smem));
}

}  // namespace

size_t decode_workspace_bytes(int batch, int n_q_heads, int n_kv_heads, int64_t cap) {
  return ws_layout(batch, n_q_heads, n_kv_heads, cap).total;
}

template <int NT, int S>
static aatc_status launch_mfma(const void* params_k, const void* params_v, int batch,
                               int n_q_heads, int n_kv_heads, const void* q, aatc_dtype q_dtype,
                               const void* k_codes, const uint16_t* k_alpha,
                               const void* v_codes, const uint16_t* v_alpha,
                               const int32_t* seq_len, int64_t cap, int rk, int rv,
                               float softmax_scale, float* out, unsigned* ctr, unsigned* flg,
                               QPlanes* pln, Partial* parts, size_t merge_lds, hipStream_t st) {
  constexpr int NH = 4 * NT, TW = S / 4;
  const int n_splits = (int)((cap + S - 1) / S);
  const int bv_max = 8 * rv;                           // value budget <= 8 R
  const size_t front = std::max((size_t)S * (rk + rv) + 16, (size_t)8 * NH * kD * 4);
  size_t off = front + 4 * (size_t)S;                  // alpha^K, alpha^V
  const int ql_base = (int)off;
  off += (size_t)4 * NH * 2 * kMaxPairs * 64;
  int ob_base, ob_wstride;
  if ((size_t)NH * bv_max * 4 <= (size_t)TW * rk) {    // O' fits in each wave's key records
    ob_base = 0;
    ob_wstride = TW * rk;
  } else {
    ob_base = (int)off;
    ob_wstride = NH * bv_max * 4;
    off += (size_t)4 * ob_wstride;
  }
  const size_t lds = std::max(off, merge_lds);
  if (lds > 160 * 1024 - 24 * 1024) return AATC_E_UNSUPPORTED;
  static size_t set_lds = 0;
  if (lds > set_lds) {
    if (hipFuncSetAttribute((const void*)decode_mfma_kernel<NT, S>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
      return AATC_E_DEVICE;
    set_lds = lds;
  }
  dim3 grid((unsigned)n_splits, (unsigned)n_kv_heads, (unsigned)batch);
  hipLaunchKernelGGL((decode_mfma_kernel<NT, S>), grid, dim3(kDecThreads), lds, st, params_k,
                     params_v, n_q_heads, n_kv_heads, q, (int)q_dtype,
                     static_cast<const uint8_t*>(k_codes), k_alpha,
                     static_cast<const uint8_t*>(v_codes), v_alpha, seq_len, cap,
                     softmax_scale, out, ctr, flg, pln, parts, n_splits, rk, rv, ob_base,
                     ob_wstride, ql_base);
  return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
}

aatc_status launch_decode(const void* params_k, const void* params_v, int batch,
                          int n_q_heads, int n_kv_heads, const void* q, aatc_dtype q_dtype,
                          const void* k_codes, const uint16_t* k_alpha, const void* v_codes,
                          const uint16_t* v_alpha, const int32_t* seq_len, int64_t cap,
                          int rk, int rv, float softmax_scale, float* out, void* workspace,
                          void* stream) {
  const int G = n_q_heads / n_kv_heads;
  const WsLayout wl = ws_layout(batch, n_q_heads, n_kv_heads, cap);
  char* ws = static_cast<char*>(workspace);
  auto* ctr = reinterpret_cast<unsigned*>(ws + wl.counters);
  auto* flg = reinterpret_cast<unsigned*>(ws + wl.flags);
  auto* pln = reinterpret_cast<QPlanes*>(ws + wl.planes);
  auto* parts = reinterpret_cast<Partial*>(ws + wl.partials);
  const hipStream_t st = (hipStream_t)stream;
  const size_t merge_lds = ((9 * (size_t)G + 4) * kD + 4 * kDecThreads) * sizeof(float);
  if (G <= kMaxNH && rk <= 64 && rv <= 64) {
    const bool big = rk > 48 || rv > 48;
#define AATC_MFMA(NT, S)                                                                   \
  launch_mfma<NT, S>(params_k, params_v, batch, n_q_heads, n_kv_heads, q, q_dtype, k_codes, \
                     k_alpha, v_codes, v_alpha, seq_len, cap, rk, rv, softmax_scale, out, ctr, \
                     flg, pln, parts, merge_lds, st)
    if (G <= 4) return big ? AATC_MFMA(1, 256) : AATC_MFMA(1, 512);
    return big ? AATC_MFMA(2, 256) : AATC_MFMA(2, 512);
#undef AATC_MFMA
  }
  const int n_splits = (int)((cap + kSplit - 1) / kSplit);
  size_t lds = std::max((size_t)G * (kSplit + kMaxBudget) * sizeof(float), merge_lds);
  if (lds > 160 * 1024 - 24 * 1024) return AATC_E_UNSUPPORTED;
  static size_t set_lds0 = 0;
  if (lds > set_lds0) {
    if (hipFuncSetAttribute((const void*)decode_split_kernel,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
      return AATC_E_DEVICE;
    set_lds0 = lds;
  }
  dim3 grid((unsigned)n_splits, (unsigned)n_kv_heads, (unsigned)batch);
  hipLaunchKernelGGL(decode_split_kernel, grid, dim3(kDecThreads), lds, st, params_k, params_v,
                     n_q_heads, n_kv_heads, q, (int)q_dtype,
                     static_cast<const uint8_t*>(k_codes), k_alpha,
                     static_cast<const uint8_t*>(v_codes), v_alpha, seq_len, cap,
                     softmax_scale, out, ctr, flg, parts, n_splits, rk, rv);
  return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
}

}  // namespace aatc
