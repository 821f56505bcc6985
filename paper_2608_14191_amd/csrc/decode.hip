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

// The last workgroup of a (sequence, KV head) to finish merges the split partials
// (m, l, o~) of its G query heads and applies the inverse transform o = T_V o~ / l.
// The arrival counter and the query-plane flag are reset, so the workspace is ready
// for the next call.  `lds` must hold 4 * kDecThreads + G * kD floats.
__device__ void merge_if_last(const void* params_v, int n_q_heads, int kvh, int seq,
                              int64_t kv_row, int G, float* out, unsigned* counters,
                              unsigned* flags, const Partial* partials, int n_splits,
                              float* lds, float* red) {
  __shared__ unsigned last_flag;
  __shared__ float mm[kMaxGroup], ll[kMaxGroup];
  const int tid = threadIdx.x;
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const unsigned prev = atomicAdd(&counters[kv_row], 1u);
    last_flag = (prev == (unsigned)n_splits - 1u) ? 1u : 0u;
  }
  __syncthreads();
  if (!last_flag) return;
  __threadfence();

  const HeadParams* hv = head_params(params_v, kvh);
  const Partial* all = partials + kv_row * n_splits * G;
  // (a) global max and normalizer per head
  for (int h = 0; h < G; ++h) {
    float m = -INFINITY;
    for (int s = tid; s < n_splits; s += kDecThreads) m = fmaxf(m, all[s * G + h].m);
    m = block_reduce(m, true, red);
    float l = 0.f;
    for (int s = tid; s < n_splits; s += kDecThreads) {
      const float ms = all[s * G + h].m;
      l += (ms == -INFINITY) ? 0.f : exp2f(ms - m) * all[s * G + h].l;
    }
    l = block_reduce(l, false, red);
    if (tid == 0) {
      mm[h] = m;
      ll[h] = l;
    }
  }
  __syncthreads();
  // (b) o~ = sum_s 2^(m_s - m) o~_s / l over float4 columns; the splits are strided
  // over thread groups when the columns do not fill the workgroup.
  float* osum = lds;                                       // [G][kD]
  v4f* part4 = reinterpret_cast<v4f*>(lds + G * kD);       // [kDecThreads]
  const int slots = G * (kD / 4);
  const int ngroups = slots >= kDecThreads ? 1 : kDecThreads / slots;
  for (int base = 0; base < slots; base += kDecThreads) {
    const int t = tid;
    const int slot = base + (t % min(slots - base, kDecThreads));
    const int grp = t / min(slots - base, kDecThreads);
    const bool active = grp < ngroups && slot < slots;
    if (active) {
      const int h = slot / (kD / 4), c4 = slot % (kD / 4);
      const float m = mm[h];
      v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
      for (int s = grp; s < n_splits; s += ngroups) {
        const float ms = all[s * G + h].m;
        const float w = (ms == -INFINITY) ? 0.f : exp2f(ms - m);
        acc += w * reinterpret_cast<const v4f*>(all[s * G + h].o)[c4];
      }
      part4[t] = acc;
    }
    __syncthreads();
    const int width = min(slots - base, kDecThreads);
    if (tid < width) {
      const int slot0 = base + tid;
      const int h = slot0 / (kD / 4), c4 = slot0 % (kD / 4);
      v4f acc = part4[tid];
      for (int g = 1; g < ngroups; ++g) acc += part4[g * width + tid];
      const float inv_l = ll[h] > 0.f ? 1.f / ll[h] : 0.f;
      reinterpret_cast<v4f*>(osum)[h * (kD / 4) + c4] = acc * inv_l;
    }
    __syncthreads();
  }
  // (c) o_j = sum_c T_V[j][c] o~_c, reading the transposed copy (coalesced over j)
  {
    const int j = tid & (kD - 1), hh = tid >> 7;
    float acc[kMaxGroup / 2];
#pragma unroll
    for (int k = 0; k < kMaxGroup / 2; ++k) acc[k] = 0.f;
#pragma unroll 16
    for (int c = 0; c < kD; ++c) {
      const float t = hv->Tt[c * kD + j];
#pragma unroll
      for (int k = 0; k < kMaxGroup / 2; ++k) {
        const int h = hh + 2 * k;
        if (h < G) acc[k] += t * osum[h * kD + c];
      }
    }
#pragma unroll
    for (int k = 0; k < kMaxGroup / 2; ++k) {
      const int h = hh + 2 * k;
      if (h < G) out[((int64_t)seq * n_q_heads + kvh * G + h) * kD + j] = acc[k];
    }
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
      for (int hh = 0; hh < 2; ++hh) {
        uint32_t word = vt[tile * 16 * rv + 2 * v + hh];
        const int base = tile * kTile + 32 * hh;
        if (base + 32 > nt) word &= (base >= nt) ? 0u : ((1u << (nt - base)) - 1u);
        while (word) {
          const int k = __builtin_ctz(word);
          word &= word - 1;
#pragma unroll
          for (int h = 0; h < kMaxGroup; ++h)
            if (h < G) acc[h] += sc[h * kSplit + base + k];
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
    part[h].o[c] = o;
  }
  if (tid < G) {
    part[tid].m = !layout_ok ? NAN : (nt > 0) ? mh[tid] : -INFINITY;
    part[tid].l = !layout_ok ? NAN : (nt > 0) ? lh[tid] : 0.f;
  }
  merge_if_last(params_v, n_q_heads, kvh, seq, kv_row, G, out, counters, flags, partials,
                n_splits, dyn, red);
}

// ---------------------------------------------------------------------------------------
// MFMA decode kernel (G <= 8 query heads per KV head, record budgets <= 512 bits).
//
// Both contractions run on v_mfma_i32_16x16x64_i8 over the bits of the codes: a code
// u_c = sum_k 2^k bit_k, so every record bit is a virtual channel whose weight is the
// channel's weight times 2^k.
//  * Keys: D[(head, limb), token] = sum_bits Qlimb[(head, limb), bit] * bit(token).
//    One record dword w (32 bits of one token) expands to MFMA bytes by
//    r_d = w & (0x01010101 << d): byte j of r_d is 2^d * bit (8j + d).  The factor 2^d
//    (and the sign of int8 0x80 for d = 7) is folded into the query weights.  The
//    query weights are 32-bit fixed point split into four int8 limbs; four heads times
//    four limbs fill the 16 MFMA rows.
//  * Values: D[bit, (head, limb)] = sum_tokens bit(token) * Plimb[token, (head, limb)],
//    with P = 2^(z - m) * alpha^V in 32-bit fixed point.  The tiles store one value bit
//    of 32 tokens per word, so the same one-AND expansion feeds the token dimension.
// Integer accumulation is exact; limbs are recombined in fp32 once per token (keys)
// or once per split (values).
//
// The query bit weights of a (sequence, KV head) are computed once, by the workgroup
// of split 0, and published in the workspace; the other splits poll a flag a bounded
// number of times while their cache loads are in flight, and compute the weights
// themselves if the flag does not appear.
// ---------------------------------------------------------------------------------------
constexpr int kMaxVT = 8;        // value-bit tiles of 16 per wave (<= 512 bits)
constexpr int kMaxTilesK = 8;    // 16-token key tiles per wave (S <= 512)
constexpr int kMaxLoads = 6;     // 16-byte loads per thread per cache region

__device__ inline v4i mfma_i8(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// Four balanced int8 limbs of a 32-bit value |x| < 2^30, packed in one dword (limb L in
// byte L, two's complement): x = sum_L limb_L 256^L.
__device__ inline uint32_t pack_limbs(int x) {
  return ((uint32_t)x + 0x80808080u) ^ 0x80808080u;
}

__device__ inline float limb_sum4(float v) {
  v += __shfl_xor(v, 1, 64);
  v += __shfl_xor(v, 2, 64);
  return v;
}

// Query bit weights in MFMA operand order (limb planes), their offsets C and exponents.
// scratch: >= 8 * NH * kD floats of LDS not otherwise in use.
template <int NH>
__device__ void query_planes(const HeadParams* hk, const void* q, int q_dtype, int64_t qbase,
                             int G, float scale, int BK, int NP, float (*qs)[kD],
                             float (*qp)[kD], float* scratch, uint8_t* ql, int (*cofs)[4],
                             int* fexp, unsigned* qmax_bits) {
  const int tid = threadIdx.x;
  for (int i = tid; i < NH * kD; i += kDecThreads) {
    const int h = i / kD;
    qs[h][i % kD] = (h < G) ? load_q(q, q_dtype, qbase + i) : 0.f;
  }
  for (int i = tid; i < 4 * NH * 2 * NP * 64 / 4; i += kDecThreads)
    reinterpret_cast<uint32_t*>(ql)[i] = 0u;
  if (tid < NH) qmax_bits[tid] = 0u;
  if (tid < NH * 4) cofs[tid / 4][tid % 4] = 0;
  __syncthreads();
  // q~ = T_K^T q: thread (rows 16 jq .. 16 jq + 15, columns 4 c4 .. 4 c4 + 3).
  {
    const int c4 = tid & 31, jq = tid >> 5;
    const v4f* t4 = reinterpret_cast<const v4f*>(hk->T);
    v4f acc[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) acc[h] = (v4f){0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int jj = 0; jj < 16; ++jj) {
      const int j = 16 * jq + jj;
      const v4f tr = t4[j * (kD / 4) + c4];
#pragma unroll
      for (int h = 0; h < NH; ++h) acc[h] += tr * qs[h][j];
    }
#pragma unroll
    for (int h = 0; h < NH; ++h)
      reinterpret_cast<v4f*>(scratch)[(jq * NH + h) * (kD / 4) + c4] = acc[h];
  }
  __syncthreads();
  for (int i = tid; i < NH * kD; i += kDecThreads) {
    const int h = i / kD, c = i % kD;
    float acc = 0.f;
#pragma unroll
    for (int jq = 0; jq < 8; ++jq) acc += scratch[(jq * NH + h) * kD + c];
    const int b = hk->bits[c];
    float qv = 0.f;
    if (h < G && b) {
      qv = acc * hk->s[c] * ldexpf(1.f, 1 - b) * scale * kLog2e;
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
    const int c = hk->virt_chan[v], k = hk->virt_bit[v];
    const int D = v >> 5, p = v & 31, j = p >> 3, d = p & 7;
    int fx = (int)rintf(ldexpf(qp[h][c], k - d + fexp[h]));
    if (d == 7) fx = -fx;
    const uint32_t limbs = pack_limbs(fx);
    const int s = 2 * (D >> 2) + (d >> 2);
    const int pos = ((D & 3) << 4) + ((d & 3) << 2) + j;
#pragma unroll
    for (int L = 0; L < 4; ++L)
      ql[((L * NH + h) * 2 * NP + s) * 64 + pos] = (uint8_t)(limbs >> (8 * L));
    if (k == hk->bits[c] - 1) {                 // offset C = sum_c Q(c, msb)
      const int bv = (d == 7) ? -128 : (1 << d);
#pragma unroll
      for (int L = 0; L < 4; ++L)
        atomicAdd(&cofs[h][L], (int)(int8_t)(limbs >> (8 * L)) * bv);
    }
  }
  __syncthreads();
}

template <int NT>
__global__ __launch_bounds__(kDecThreads, 2) void decode_mfma_kernel(
    const void* __restrict__ params_k, const void* __restrict__ params_v, int n_q_heads,
    int n_kv_heads, const void* __restrict__ q, int q_dtype,
    const uint8_t* __restrict__ k_codes, const uint16_t* __restrict__ k_alpha,
    const uint8_t* __restrict__ v_codes, const uint16_t* __restrict__ v_alpha,
    const int32_t* __restrict__ seq_len, int64_t cap, float scale, float* __restrict__ out,
    unsigned* __restrict__ counters, unsigned* __restrict__ flags,
    QPlanes* __restrict__ planes, Partial* __restrict__ partials, int n_splits, int S, int RK,
    int RV) {
  constexpr int NH = 4 * NT;                         // head slots (rows of 4 limbs each)
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ float qs[NH][kD];
  __shared__ float qp[NH][kD];
  __shared__ int cofs[NH][4];                        // key offset C per head and limb
  __shared__ int fexp[NH];                           // fixed-point exponent of Q per head
  __shared__ unsigned qmax_bits[NH];
  __shared__ unsigned amax_bits;
  __shared__ unsigned ready;
  __shared__ float red[kDecThreads / 64];
  __shared__ float wmax[4][NH], wsum[4][NH];
  __shared__ double wpa[4][NH];
  __shared__ float mh[NH], lh[NH];
  __shared__ double pah[NH];

  const int G = n_q_heads / n_kv_heads;
  const int split = blockIdx.x, kvh = blockIdx.y, seq = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lrow = lane & 15, lgrp = lane >> 4;
  const HeadParams* hk = head_params(params_k, kvh);
  const HeadParams* hv = head_params(params_v, kvh);
  const bool layout_ok = hk->record_bytes == RK && hv->record_bytes == RV;
  const int BK = hk->budget, BV = hv->budget;
  const int RWK = RK / 4;
  const int NP = (RWK + 3) / 4;
  const int NVT = (BV + 15) / 16;
  const int64_t kv_row = (int64_t)seq * n_kv_heads + kvh;
  const int len = (int)min<int64_t>(max(seq_len[seq], 0), cap);
  const int t0 = split * S;
  const int nt = max(0, min(S, len - t0));
  const int n_load = min(S, (nt + kTile - 1) / kTile * kTile);

  // Dynamic LDS: [key records | value tiles] (also prologue scratch) | alpha^K | alpha^V
  // | P limbs | Q limbs | O'.
  const int front = max(S * RK + 16 + S * RV, 8 * NH * kD * 4);
  uint8_t* kbuf = smem;
  uint8_t* vbuf = kbuf + S * RK + 16;
  uint16_t* akb = reinterpret_cast<uint16_t*>(smem + front);
  uint16_t* avb = akb + S;
  uint8_t* pb = reinterpret_cast<uint8_t*>(avb + S);            // [4][NH][S]
  uint8_t* ql = pb + 4 * NH * S;                                // [4][NH][2 NP][64]
  float* ob = reinterpret_cast<float*>(ql + 4 * NH * 2 * kMaxPairs * 64);   // [NH][BV]

  Partial* part = partials + (kv_row * n_splits + split) * G;
  if (nt == 0 || !layout_ok) {
    for (int i = tid; i < G * kD; i += kDecThreads) part[i / kD].o[i % kD] = 0.f;
    if (tid < G) {
      part[tid].m = layout_ok ? -INFINITY : NAN;
      part[tid].l = layout_ok ? 0.f : NAN;
    }
    merge_if_last(params_v, n_q_heads, kvh, seq, kv_row, G, out, counters, flags, partials,
                  n_splits, reinterpret_cast<float*>(smem), red);
    return;
  }

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

  // (2) Query bit weights while the loads are in flight: published by split 0.
  QPlanes* qpl = planes + kv_row;
  const int plane_vecs = 4 * NH * 2 * NP * 64 / 16;
  if (tid == 0) amax_bits = 0u;
  bool have = false;
  if (split != 0) {
    if (tid == 0) {
      unsigned ok = 0u;
      for (int it = 0; it < kSpinLimit; ++it) {
        if (__hip_atomic_load(&flags[kv_row], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT)) {
          ok = 1u;
          break;
        }
        __builtin_amdgcn_s_sleep(10);
      }
      ready = ok;
    }
    __syncthreads();
    have = ready != 0u;
    if (have) {
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      for (int i = tid; i < plane_vecs; i += kDecThreads)
        reinterpret_cast<v4i*>(ql)[i] = reinterpret_cast<const v4i*>(qpl->ql)[i];
      if (tid < NH * 4) cofs[tid / 4][tid % 4] = qpl->cofs[tid / 4][tid % 4];
      if (tid < NH) fexp[tid] = qpl->fexp[tid];
    }
  }
  if (!have) {
    query_planes<NH>(hk, q, q_dtype, ((int64_t)seq * n_q_heads + kvh * G) * kD, G, scale, BK,
                     NP, qs, qp, reinterpret_cast<float*>(smem), ql, cofs, fexp, qmax_bits);
    if (split == 0) {
      for (int i = tid; i < plane_vecs; i += kDecThreads)
        reinterpret_cast<v4i*>(qpl->ql)[i] = reinterpret_cast<const v4i*>(ql)[i];
      if (tid < NH * 4) qpl->cofs[tid / 4][tid % 4] = cofs[tid / 4][tid % 4];
      if (tid < NH) qpl->fexp[tid] = fexp[tid];
      __threadfence();
      __syncthreads();
      if (tid == 0)
        __hip_atomic_store(&flags[kv_row], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();

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
  if (tid < 128 && (tid & 63) < na16) {
    reinterpret_cast<v4i*>(tid < 64 ? akb : avb)[tid & 63] = ra;
    if (tid >= 64) {
      // max alpha^V over the valid tokens 8 idx .. 8 idx + 7 of this load
      const int first = 8 * (tid & 63);
      float m = 0.f;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t w = (uint32_t)ra[u];
        if (first + 2 * u < nt) m = fmaxf(m, fabsf(half_bits_to_float((uint16_t)(w & 0xffff))));
        if (first + 2 * u + 1 < nt) m = fmaxf(m, fabsf(half_bits_to_float((uint16_t)(w >> 16))));
      }
      atomicMax(&amax_bits, __float_as_uint(m));
    }
  }
  __syncthreads();

  // (4) Key scores: this wave's S/4 tokens in 16-token tiles.
  v4i aq[NT][2 * kMaxPairs];
#pragma unroll
  for (int rt = 0; rt < NT; ++rt)
#pragma unroll
    for (int s = 0; s < 2 * kMaxPairs; ++s)
      if (s < 2 * NP) {
        const int h = 4 * rt + (lrow >> 2), L = lrow & 3;
        aq[rt][s] = *reinterpret_cast<const v4i*>(ql + ((L * NH + h) * 2 * NP + s) * 64 + lgrp * 16);
      }
  const int ntile = S / 64;
  float zr[kMaxTilesK][NT];
#pragma unroll
  for (int tt = 0; tt < kMaxTilesK; ++tt) {
    if (tt < ntile) {
      const int tl = wave * (S / 4) + 16 * tt + lrow;
      const uint8_t* rec = kbuf + tl * RK;
      v4i acc[NT];
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) acc[rt] = (v4i){0, 0, 0, 0};
#pragma unroll
      for (int P = 0; P < kMaxPairs; ++P) {
        if (P < NP) {
          const int D = 4 * P + lgrp;
          const uint32_t w = (D < RWK) ? *reinterpret_cast<const uint32_t*>(rec + 4 * D) : 0u;
          const v4i b0 = {(int)(w & 0x01010101u), (int)(w & 0x02020202u),
                          (int)(w & 0x04040404u), (int)(w & 0x08080808u)};
          const v4i b1 = {(int)(w & 0x10101010u), (int)(w & 0x20202020u),
                          (int)(w & 0x40404040u), (int)(w & 0x80808080u)};
#pragma unroll
          for (int rt = 0; rt < NT; ++rt) {
            acc[rt] = mfma_i8(aq[rt][2 * P], b0, acc[rt]);
            acc[rt] = mfma_i8(aq[rt][2 * P + 1], b1, acc[rt]);
          }
        }
      }
      const float ak = half_bits_to_float(akb[tl]);
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) {
        const int h = 4 * rt + lgrp;
        const float f = ldexpf((float)(acc[rt][3] - cofs[h][3]), 24) +
                        ldexpf((float)(acc[rt][2] - cofs[h][2]), 16) +
                        ldexpf((float)(acc[rt][1] - cofs[h][1]), 8) +
                        (float)(acc[rt][0] - cofs[h][0]);
        zr[tt][rt] = (tl < nt && h < G) ? ak * ldexpf(f, -fexp[h]) : -INFINITY;
      }
    }
  }

  // (5) Split softmax statistics: m per head, then p = 2^(z - m).
#pragma unroll
  for (int rt = 0; rt < NT; ++rt) {
    float m = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < kMaxTilesK; ++tt)
      if (tt < ntile) m = fmaxf(m, zr[tt][rt]);
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    if (lrow == 0) wmax[wave][4 * rt + lgrp] = m;
  }
  __syncthreads();
  if (tid < NH) {
    mh[tid] = fmaxf(fmaxf(wmax[0][tid], wmax[1][tid]), fmaxf(wmax[2][tid], wmax[3][tid]));
  }
  {
    int e = 0;
    frexpf(__uint_as_float(amax_bits), &e);
    // P = 2^(z - m) alpha^V <= max alpha^V < 2^e, so P * 2^(30 - e) < 2^30.
    const int fv = amax_bits ? 30 - e : 0;
    __syncthreads();
#pragma unroll
    for (int rt = 0; rt < NT; ++rt) {
      const int h = 4 * rt + lgrp;
      const float m = mh[h];
      float lsum = 0.f;
      double pa = 0.0;
#pragma unroll
      for (int tt = 0; tt < kMaxTilesK; ++tt) {
        if (tt < ntile) {
          const int tl = wave * (S / 4) + 16 * tt + lrow;
          const float p = (zr[tt][rt] == -INFINITY) ? 0.f : exp2f(zr[tt][rt] - m);
          lsum += p;
          const float pv = (tl < nt) ? p * half_bits_to_float(avb[tl]) : 0.f;
          const int qq = tl & 127, r = qq & 31, j = r >> 3, d = r & 7;
          int fx = (int)rintf(ldexpf(pv, fv - d));
          pa += ldexp((double)fx, d);
          if (d == 7) fx = -fx;
          const uint32_t limbs = pack_limbs(fx);
          const int pos = (tl & ~127) + ((qq >> 5) << 5) + ((d >> 2) << 4) + ((d & 3) << 2) + j;
#pragma unroll
          for (int L = 0; L < 4; ++L) pb[(L * NH + h) * S + pos] = (uint8_t)(limbs >> (8 * L));
        }
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        lsum += __shfl_xor(lsum, o, 64);
        pa += __shfl_xor(pa, o, 64);
      }
      if (lrow == 0) {
        wsum[wave][h] = lsum;
        wpa[wave][h] = pa;
      }
    }
    __syncthreads();
    if (tid < NH) {
      lh[tid] = wsum[0][tid] + wsum[1][tid] + wsum[2][tid] + wsum[3][tid];
      pah[tid] = ldexp(wpa[0][tid] + wpa[1][tid] + wpa[2][tid] + wpa[3][tid], -fv);
    }

    // (6) Value bits x P limbs.
    v4i accv[kMaxVT][NT];
#pragma unroll
    for (int k = 0; k < kMaxVT; ++k)
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) accv[k][rt] = (v4i){0, 0, 0, 0};
    const int nchunk = (nt + 127) / 128;
    for (int ch = 0; ch < nchunk; ++ch) {
      v4i pb0[NT], pb1[NT];
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) {
        const int h = 4 * rt + (lrow >> 2), L = lrow & 3;
        const uint8_t* src = pb + (L * NH + h) * S + ch * 128 + lgrp * 32;
        pb0[rt] = *reinterpret_cast<const v4i*>(src);
        pb1[rt] = *reinterpret_cast<const v4i*>(src + 16);
      }
      const uint8_t* tile = vbuf + (2 * ch + (lgrp >> 1)) * (kTile * RV);
#pragma unroll
      for (int k = 0; k < kMaxVT; ++k) {
        const int vt = wave + 4 * k;
        if (vt < NVT) {
          const int v = 16 * vt + lrow;
          const uint32_t w = *reinterpret_cast<const uint32_t*>(tile + (2 * v + (lgrp & 1)) * 4);
          const v4i a0 = {(int)(w & 0x01010101u), (int)(w & 0x02020202u),
                          (int)(w & 0x04040404u), (int)(w & 0x08080808u)};
          const v4i a1 = {(int)(w & 0x10101010u), (int)(w & 0x20202020u),
                          (int)(w & 0x40404040u), (int)(w & 0x80808080u)};
#pragma unroll
          for (int rt = 0; rt < NT; ++rt) {
            accv[k][rt] = mfma_i8(a0, pb0[rt], accv[k][rt]);
            accv[k][rt] = mfma_i8(a1, pb1[rt], accv[k][rt]);
          }
        }
      }
    }
    // Recombine limbs (columns 4 h + L) and store O'[h][v] = sum_t P_t bit_v(t).
#pragma unroll
    for (int k = 0; k < kMaxVT; ++k) {
      const int vt = wave + 4 * k;
      if (vt < NVT) {
#pragma unroll
        for (int rt = 0; rt < NT; ++rt) {
          const int h = 4 * rt + (lrow >> 2), L = lrow & 3;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float s = limb_sum4(ldexpf((float)accv[k][rt][i], 8 * L));
            const int v = 16 * vt + 4 * lgrp + i;
            if (L == 0 && v < BV) ob[h * BV + v] = ldexpf(s, -fv);
          }
        }
      }
    }
  }
  __syncthreads();

  // (7) Partial o~_c = s_c 2^(1-b_c) (sum_k 2^k O'(c,k) - 2^(b_c-1) sum_t P_t).
  for (int i = tid; i < G * kD; i += kDecThreads) {
    const int h = i / kD, c = i % kD;
    const int b = hv->bits[c];
    float o = 0.f;
    if (b) {
      const int off = hv->bit_off[c];
      float acc = 0.f;
      for (int k = 0; k < b; ++k) acc += ldexpf(ob[h * BV + off + k], k);
      o = hv->s[c] * ldexpf(1.f, 1 - b) * (acc - (float)ldexp(pah[h], b - 1));
    }
    part[h].o[c] = o;
  }
  if (tid < G) {
    part[tid].m = mh[tid];
    part[tid].l = lh[tid];
  }
  merge_if_last(params_v, n_q_heads, kvh, seq, kv_row, G, out, counters, flags, partials,
                n_splits, reinterpret_cast<float*>(smem), red);
}

}  // namespace

size_t decode_workspace_bytes(int batch, int n_q_heads, int n_kv_heads, int64_t cap) {
  return ws_layout(batch, n_q_heads, n_kv_heads, cap).total;
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
  const size_t merge_lds = (4 * kDecThreads + (size_t)G * kD) * sizeof(float);
  const bool fast = G <= kMaxNH && rk <= 64 && rv <= 64;
  if (fast) {
    const int S = (rk <= 48 && rv <= 48) ? 512 : 256;
    const int NT = G <= 4 ? 1 : 2, NH = 4 * NT;
    const int n_splits = (int)((cap + S - 1) / S);
    const size_t front = std::max((size_t)S * (rk + rv) + 16, (size_t)8 * NH * kD * 4);
    size_t lds = front + 4 * (size_t)S + 4 * (size_t)NH * S +
                 4 * (size_t)NH * 2 * kMaxPairs * 64 + (size_t)NH * 512 * sizeof(float);
    lds = std::max(lds, merge_lds);
    if (lds > 160 * 1024 - 24 * 1024) return AATC_E_UNSUPPORTED;
    dim3 grid((unsigned)n_splits, (unsigned)n_kv_heads, (unsigned)batch);
    const void* fn = NT == 1 ? (const void*)decode_mfma_kernel<1> : (const void*)decode_mfma_kernel<2>;
    static size_t set_lds[3] = {0, 0, 0};
    if (lds > set_lds[NT]) {
      if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
          hipSuccess)
        return AATC_E_DEVICE;
      set_lds[NT] = lds;
    }
    if (NT == 1)
      hipLaunchKernelGGL(decode_mfma_kernel<1>, grid, dim3(kDecThreads), lds, st, params_k,
                         params_v, n_q_heads, n_kv_heads, q, (int)q_dtype,
                         static_cast<const uint8_t*>(k_codes), k_alpha,
                         static_cast<const uint8_t*>(v_codes), v_alpha, seq_len, cap,
                         softmax_scale, out, ctr, flg, pln, parts, n_splits, S, rk, rv);
    else
      hipLaunchKernelGGL(decode_mfma_kernel<2>, grid, dim3(kDecThreads), lds, st, params_k,
                         params_v, n_q_heads, n_kv_heads, q, (int)q_dtype,
                         static_cast<const uint8_t*>(k_codes), k_alpha,
                         static_cast<const uint8_t*>(v_codes), v_alpha, seq_len, cap,
                         softmax_scale, out, ctr, flg, pln, parts, n_splits, S, rk, rv);
    return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
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
