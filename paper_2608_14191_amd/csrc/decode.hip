// AATC decode attention on gfx950 (Algorithm 1, inference part, evaluated in the
// transformed domain of App. B: q~ = T_K^T q; the inverse transform T_V is applied once
// to each output).
//
// Grid: (token split, KV head, sequence).  Each workgroup scores its split's tokens
// for the G query heads of its KV head, runs a split-local softmax and accumulates
// the value codes; the last workgroup of each (sequence, KV head) merges the split
// partials (m, l, o~) and applies T_V.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "launch.h"
#include "params.h"

namespace aatc {
namespace {

constexpr int kDecThreads = 256;
constexpr int kSplit = 512;                      // tokens per workgroup split
constexpr float kLog2e = 1.4426950408889634f;

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

struct Partial {         // per (sequence, KV head, split, head-in-group)
  float m;               // split max of the log2-domain logits
  float l;               // sum of 2^(z - m)
  float o[kD];           // sum of 2^(z - m) * h^V (transformed domain, storage channels)
};

__global__ __launch_bounds__(kDecThreads) void decode_split_kernel(
    const void* __restrict__ params_k, const void* __restrict__ params_v, int n_q_heads,
    int n_kv_heads, const void* __restrict__ q, int q_dtype,
    const uint8_t* __restrict__ k_codes, const uint16_t* __restrict__ k_alpha,
    const uint8_t* __restrict__ v_codes, const uint16_t* __restrict__ v_alpha,
    const int32_t* __restrict__ seq_len, int64_t cap, float scale, float* __restrict__ out,
    unsigned* __restrict__ counters, Partial* __restrict__ partials, int n_splits) {
  extern __shared__ float dyn[];
  __shared__ float qs[kMaxGroup][kD];
  __shared__ float qp[kMaxGroup][kD];
  __shared__ float cterm[kMaxGroup];
  __shared__ float red[kDecThreads / 64];
  __shared__ float mh[kMaxGroup], lh[kMaxGroup], pah[kMaxGroup];
  __shared__ unsigned last_flag;

  const int split = blockIdx.x, kvh = blockIdx.y, seq = blockIdx.z;
  const int G = n_q_heads / n_kv_heads;
  const int tid = threadIdx.x;
  const HeadParams* hk = head_params(params_k, kvh);
  const HeadParams* hv = head_params(params_v, kvh);
  const int rk = hk->record_bytes, rv = hv->record_bytes;
  const int bk = hk->budget, bv = hv->budget;
  float* sc = dyn;                                  // [G][kSplit] logits, then weights
  float* vq = dyn + G * kSplit;                     // [G][kMaxBudget] per-bit weights / sums

  const int len = (int)min<int64_t>(max(seq_len[seq], 0), cap);   // out-of-range lengths clamp
  const int t0 = split * kSplit;
  const int nt = max(0, min(kSplit, len - t0));

  // Queries of the group, then q'_c = (T_K^T q)_c * s_c * 2^(1-b_c) * scale * log2(e).
  for (int i = tid; i < G * kD; i += kDecThreads)
    qs[i / kD][i % kD] = load_q(q, q_dtype, ((int64_t)seq * n_q_heads + kvh * G) * kD + i);
  __syncthreads();
  for (int i = tid; i < G * kD; i += kDecThreads) {
    const int h = i / kD, c = i % kD;
    float acc = 0.f;
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
    part[tid].m = (nt > 0) ? mh[tid] : -INFINITY;
    part[tid].l = (nt > 0) ? lh[tid] : 0.f;
  }

  // Last workgroup of this (sequence, KV head) merges the splits.
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const unsigned prev = atomicAdd(&counters[kv_row], 1u);
    last_flag = (prev == (unsigned)n_splits - 1u) ? 1u : 0u;
  }
  __syncthreads();
  if (!last_flag) return;
  __threadfence();

  const Partial* all = partials + kv_row * n_splits * G;
  float* wts = dyn;                                 // [G][n_splits] merge weights
  float* ot = dyn + G * n_splits;                   // [G][kD] merged o~
  for (int h = 0; h < G; ++h) {
    float m = -INFINITY;
    for (int s = tid; s < n_splits; s += kDecThreads) m = fmaxf(m, all[s * G + h].m);
    m = block_reduce(m, true, red);
    float l = 0.f;
    for (int s = tid; s < n_splits; s += kDecThreads) {
      const float ms = all[s * G + h].m;
      const float w = (ms == -INFINITY) ? 0.f : exp2f(ms - m);
      wts[h * n_splits + s] = w;
      l += w * all[s * G + h].l;
    }
    l = block_reduce(l, false, red);
    if (tid == 0) lh[h] = l;
  }
  __syncthreads();
  for (int i = tid; i < G * kD; i += kDecThreads) {
    const int h = i / kD, c = i % kD;
    float acc = 0.f;
    for (int s = 0; s < n_splits; ++s) acc += wts[h * n_splits + s] * all[s * G + h].o[c];
    ot[h * kD + c] = (lh[h] > 0.f) ? acc / lh[h] : 0.f;
  }
  __syncthreads();
  for (int i = tid; i < G * kD; i += kDecThreads) {
    const int h = i / kD, j = i % kD;
    float acc = 0.f;
    for (int c = 0; c < kD; ++c) acc += hv->T[j * kD + c] * ot[h * kD + c];
    out[((int64_t)seq * n_q_heads + kvh * G + h) * kD + j] = acc;
  }
  if (tid == 0) counters[kv_row] = 0u;
}

}  // namespace

static int n_splits_for(int64_t cap) { return (int)((cap + kSplit - 1) / kSplit); }

size_t decode_workspace_bytes(int batch, int n_q_heads, int n_kv_heads, int64_t cap) {
  const size_t counters = ((size_t)batch * n_kv_heads * sizeof(unsigned) + 255) / 256 * 256;
  const size_t parts = (size_t)batch * n_q_heads * n_splits_for(cap) * sizeof(Partial);
  return counters + parts;
}

aatc_status launch_decode(const void* params_k, const void* params_v, int batch,
                          int n_q_heads, int n_kv_heads, const void* q, aatc_dtype q_dtype,
                          const void* k_codes, const uint16_t* k_alpha, const void* v_codes,
                          const uint16_t* v_alpha, const int32_t* seq_len, int64_t cap,
                          float softmax_scale, float* out, void* workspace, void* stream) {
  const int G = n_q_heads / n_kv_heads;
  const int n_splits = n_splits_for(cap);
  const size_t counters = ((size_t)batch * n_kv_heads * sizeof(unsigned) + 255) / 256 * 256;
  auto* ctr = static_cast<unsigned*>(workspace);
  auto* parts = reinterpret_cast<Partial*>(static_cast<char*>(workspace) + counters);
  size_t lds = (size_t)G * (kSplit + kMaxBudget) * sizeof(float);
  const size_t lds_merge = (size_t)G * (n_splits + kD) * sizeof(float);
  if (lds_merge > lds) lds = lds_merge;
  if (lds > 160 * 1024 - 16 * 1024) return AATC_E_UNSUPPORTED;
  if (hipFuncSetAttribute((const void*)decode_split_kernel,
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return AATC_E_DEVICE;
  dim3 grid((unsigned)n_splits, (unsigned)n_kv_heads, (unsigned)batch);
  hipLaunchKernelGGL(decode_split_kernel, grid, dim3(kDecThreads), lds, (hipStream_t)stream,
                     params_k, params_v, n_q_heads, n_kv_heads, q, (int)q_dtype,
                     static_cast<const uint8_t*>(k_codes), k_alpha,
                     static_cast<const uint8_t*>(v_codes), v_alpha, seq_len, cap,
                     softmax_scale, out, ctr, parts, n_splits);
  return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
}

}  // namespace aatc
