// AATC under head-group transforms (Sec. 5.1, the remark on head groups; Sec. 5.2, one
// token scale per head group; Sec. 6: G = 2 groups for Llama's 8 KV heads, 1 for Qwen's 4).
//
// A group is gkv consecutive KV heads; its token is the concatenation of their vectors
// (d = 128 gkv elements, KV head kk of the group at [128 kk, 128 kk + 128)).  Encode and
// decode follow Alg. 1 on those d-element vectors with the group's transform:
//   - group_encode_kernel: h = T^T x exactly rounded (the exact one-wave routine of the
//     per-head path, over d elements), one alpha per (token, group), codes packed into
//     one token-major record per (token, group);
//   - group_query_kernel: per query head, the channel weights W_c = q~_c s_c 2^(1-b_c)
//     scale log2(e) of q~ = T[block]^T q (App. B's effective query; the query of KV head k
//     lives in block k % gkv of its group);
//   - group_split_mfma_kernel: per (sequence, group, 256-token split) the scores of every
//     query head of the group, the split's softmax and the transformed-domain value sums,
//     on the matrix cores (fp16 operands) with the records staged in LDS; the VALU kernels
//     group_split_wide_kernel and group_split_kernel (64-token chunks, an online softmax)
//     take more query heads per group, wider codes, or records too long for LDS;
//   - group_merge_sum_kernel, group_merge_apply_kernel: per (sequence, query head) the merge
//     of the split partials (by 64-channel chunks) and the inverse transform o = T[block] o~
//     (by 32-row chunks).
#include <algorithm>
#include <atomic>

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "encode_core.h"
#include "group.h"
#include "group_launch.h"

namespace aatc {
namespace {

constexpr int kGThreads = 256;
constexpr int kGQThreads = 1024;                  // query kernel: sixteen waves of 8 rows
constexpr int kGChunk = 64;                       // tokens staged per chunk (one per lane)

__device__ inline void group_wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

__device__ inline float g_wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ inline float g_wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// The signed code of a channel at record bit `off`, width b (1..16), from the record's
// dwords in LDS (the row has one padding dword after the record).
__device__ inline int record_code(const uint32_t* row, int off, int b) {
  const uint32_t w0 = row[off >> 5], w1 = row[(off >> 5) + 1];
  const uint32_t v = __builtin_amdgcn_alignbit(w1, w0, (uint32_t)(off & 31));   // (w1:w0) >> off
  return __builtin_amdgcn_sbfe((int)v, 0, b);                                   // sign-extended
}

// ---------------------------------------------------------------------------------------
// Encode: one wave per (token, group); lane l holds elements and channels l + 64 i.
// h_c = fl32(sum_j x_j T_jc) exactly: fp64 sums of the exact products x_j T_jc, exact while
// |x|_1 stays below 2^(31 + g) (every product is a multiple of 2^(g - 22), g the lowest set
// bit of the token's elements, and |T| <= 1); otherwise an interval test, and the exact
// accumulator where the interval straddles an fp32 rounding boundary.
// ---------------------------------------------------------------------------------------
constexpr int kGTokensPerWave = 2;              // tokens sharing each row of T in a wave
template <int NC>
__global__ __launch_bounds__(kGThreads) void group_encode_kernel(
    const void* __restrict__ params, const void* __restrict__ x, int dtype, int64_t n_tok,
    int64_t x_stride, uint8_t* __restrict__ codes, uint16_t* __restrict__ alpha, int64_t cap,
    int64_t pos) {
  constexpr int D = 64 * NC;
  constexpr int TPW = kGTokensPerWave;
  constexpr int kRow = D * kMaxBits / 32 + 1;
  __shared__ uint32_t rec[kGThreads / 64][kRow];
  const int g = blockIdx.y, lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t t0 = ((int64_t)blockIdx.x * (kGThreads / 64) + wave) * TPW;
  if (t0 >= n_tok) return;                          // (whole wave; no barrier follows)
  const int nv = (int)min((int64_t)TPW, n_tok - t0);   // this wave's tokens
  const GroupParams* gp = group_params(params, g);
  const int rw = gp->record_bytes >> 2;
  uint32_t* row = rec[wave];
  const size_t esize = dtype == AATC_BF16 ? 2 : 4;
  const void* xrow[TPW];
  float xl[TPW][NC];
#pragma unroll
  for (int u = 0; u < TPW; ++u) {
    xrow[u] = static_cast<const char*>(x) + ((t0 + min(u, nv - 1)) * x_stride + (int64_t)g * D) * esize;
#pragma unroll
    for (int i = 0; i < NC; ++i) xl[u][i] = u < nv ? load_elem(xrow[u], dtype, lane + 64 * i) : 0.f;
  }
  double s[TPW][NC];
#pragma unroll
  for (int u = 0; u < TPW; ++u)
#pragma unroll
    for (int k = 0; k < NC; ++k) s[u][k] = 0.0;
  // Row j of T (fp32, exact multiples of 2^-22): lane l reads channels l + 64 k, one
  // coalesced row per element, used for the wave's TPW tokens; products are exact in fp64.
  const float* trow = gp->T + lane;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
#pragma unroll 2
    for (int jj = 0; jj < 64; ++jj) {
      const float* tr = trow + (size_t)(64 * i + jj) * D;
      double tv[NC];
#pragma unroll
      for (int k = 0; k < NC; ++k) tv[k] = (double)tr[64 * k];
#pragma unroll
      for (int u = 0; u < TPW; ++u) {
        const double xd =
            (double)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(xl[u][i]), jj));
#pragma unroll
        for (int k = 0; k < NC; ++k) s[u][k] = fma(xd, tv[k], s[u][k]);
      }
    }
  }
#pragma unroll
  for (int u = 0; u < TPW; ++u) {
    if (u >= nv) break;                             // (uniform)
    const int64_t t = t0 + u;
    // Lowest set bit over the token's nonzero elements (4096 for a zero token), and |x|_1,
    // which bounds sum_j |x_j T_jc| for every channel (|T| <= 1).
    int glsb = 4096;
    float l1 = 0.f;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const uint32_t bv = __float_as_uint(xl[u][i]) & 0x7fffffffu;
      l1 += fabsf(xl[u][i]);
      if (bv != 0u) {
        const int ef = (int)(bv >> 23), m = (int)(bv & 0x7fffffu);
        glsb = min(glsb, ef ? ef - 150 + __builtin_ctz((uint32_t)m | 0x800000u)
                            : -149 + __builtin_ctz((uint32_t)m));
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) glsb = min(glsb, __shfl_xor(glsb, o, 64));
    l1 = g_wave_sum(l1);
    // Every product, hence every partial sum, is a multiple of 2^(g - 22); below
    // 2^(53 + g - 22) in magnitude they are all fp64 numbers and s is exact.  The float sum
    // l1 is within 2^-14 relative of |x|_1.
    const double l1d = (double)l1 * (1.0 + 0x1p-14);
    const bool exact = l1d < ldexp(1.0, 31 + min(glsb, 900));
    float r[NC];
    float m = 0.f;
#pragma unroll
    for (int k = 0; k < NC; ++k) {
      const int c = lane + 64 * k;
      const double sv = s[u][k];
      float h;
      if (exact) {
        h = (float)sv;
      } else {
        // fp64 sum of D exact products: |error| <= D 2^-53 sum |p| <= D 2^-53 |x|_1
        const double bb = l1d * (D * 0x1p-52) + fabs(sv) * 0x1p-51 + 0x1p-1060;
        const float lo = (float)(sv - bb), hi = (float)(sv + bb);
        h = lo;
        if (lo != hi && gp->bits[c] > 0) {
          // (the exact accumulator holds any sum of up to 512 such products: each is below
          // 2^46 units of its lsb, so 512 of them stay below 2^137, inside its 320 bits)
          const int32_t* tc = gp->Tqt + (size_t)c * D;
          const void* xr = xrow[u];
          h = exact_dot_q22([&](int j) { return load_elem(xr, dtype, j); },
                            [&](int j) { return tc[j]; }, D);
        }
      }
      r[k] = h * gp->inv_s[c];
      m = fmaxf(m, gp->bits[c] > 0 ? fabsf(r[k]) : 0.f);
    }
    const __half a16 = token_alpha(g_wave_max(m));
    const float inv = inverse_alpha(a16);
    const bool midrise = gp->quantizer == AATC_QUANT_MIDRISE;
    for (int i = lane; i < rw + 1; i += 64) row[i] = 0u;
    group_wave_sync();                               // the cleared row before the ORs
#pragma unroll
    for (int k = 0; k < NC; ++k) {
      const int c = lane + 64 * k;
      const int b = gp->bits[c], off = gp->bit_off[c];
      if (b > 0) {
        const uint32_t q = quantize_code(r[k], inv, b, midrise);
        atomicOr(&row[off >> 5], q << (off & 31));
        if ((off & 31) + b > 32) atomicOr(&row[(off >> 5) + 1], q >> (32 - (off & 31)));
      }
    }
    group_wave_sync();                               // every OR before the read-out
    uint32_t* out = reinterpret_cast<uint32_t*>(codes + ((int64_t)g * cap + pos + t) * gp->record_bytes);
    for (int i = lane; i < rw; i += 64) out[i] = row[i];
    if (lane == 0) alpha[(int64_t)g * cap + pos + t] = __half_as_ushort(a16);
    group_wave_sync();                               // the read-out before the next clear
  }
}

// ---------------------------------------------------------------------------------------
// Decode.
// ---------------------------------------------------------------------------------------
struct GroupDecodeArgs {
  const void* params_k;
  const void* params_v;
  const void* q;
  int q_dtype;
  const uint8_t* k_codes;
  const uint16_t* k_alpha;
  const uint8_t* v_codes;
  const uint16_t* v_alpha;
  const int32_t* seq_len;
  int64_t cap;
  int n_q_heads, n_kv_heads, gkv, n_groups, heads;   // heads: query heads per group
  int n_splits;
  int rwk, rwv;                  // record dwords of the key and value caches
  float scale_log2e;
  float* w;                      // workspace regions
  float* cst;
  float* part;
  float* out;
  uint16_t* wop;                 // the weights as fp16 operands of the matrix-core split
  int32_t* wexp;                 //   and their per-head exponents (written when wops)
  int wops;
  float* otl;                    // merged o~ per (sequence, query head)
};

// One workgroup per (sequence, query head): W_c for the head's group channels.  Wave w of
// sixteen sums the query against rows 8 w .. 8 w + 7 of the head's block of T (lane l:
// channels l + 64 m, coalesced rows; every load of the wave in flight at once), and the
// sixteen partial sums meet in LDS.
template <int NC>
__global__ __launch_bounds__(kGQThreads) void group_query_kernel(GroupDecodeArgs a) {
  constexpr int D = 64 * NC;
  constexpr int NW = kGQThreads / 64;
  constexpr int RW = 128 / NW;                      // rows of the block per wave
  __shared__ float qs[128];
  __shared__ float part[NW][D];
  __shared__ float red[NW], redm[NW];
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, lane = tid & 63;
  const int wave = tid >> 6;
  const int gq = a.n_q_heads / a.n_kv_heads;
  const int k = h / gq, g = k / a.gkv, kk = k % a.gkv, hl = h - g * a.heads;
  const GroupParams* gp = group_params(a.params_k, g);
  if (tid < 128) qs[tid] = load_elem(a.q, a.q_dtype, ((int64_t)b * a.n_q_heads + h) * 128 + tid);
  __syncthreads();
  float acc[NC];
#pragma unroll
  for (int m = 0; m < NC; ++m) acc[m] = 0.f;
  const float* trow = gp->T + (size_t)(kk * 128 + RW * wave) * D + lane;
#pragma unroll
  for (int j = 0; j < RW; ++j) {
    const float qj = qs[RW * wave + j];
#pragma unroll
    for (int m = 0; m < NC; ++m) acc[m] = fmaf(qj, trow[(size_t)j * D + 64 * m], acc[m]);
  }
#pragma unroll
  for (int m = 0; m < NC; ++m) part[wave][lane + 64 * m] = acc[m];
  __syncthreads();
  const bool midrise = gp->quantizer == AATC_QUANT_MIDRISE;
  const size_t rowi = ((size_t)b * a.n_groups + g) * a.heads + hl;
  constexpr int CPT = (D + kGQThreads - 1) / kGQThreads;
  float wvs[CPT];
  float csum = 0.f, wmax = 0.f;
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = tid + kGQThreads * i;
    wvs[i] = 0.f;
    if (c < D) {
      float qt = part[0][c];
#pragma unroll
      for (int w = 1; w < NW; ++w) qt += part[w][c];
      const int bc = gp->bits[c];
      const float wv = bc > 0 ? ldexpf(qt * gp->s[c] * a.scale_log2e, 1 - bc) : 0.f;
      a.w[rowi * D + c] = wv;
      csum += midrise ? 0.5f * wv : 0.f;
      wvs[i] = wv;
      wmax = fmaxf(wmax, fabsf(wv));
    }
  }
  csum = g_wave_sum(csum);
  wmax = g_wave_max(wmax);
  if (lane == 0) {
    red[wave] = csum;
    redm[wave] = wmax;
  }
  __syncthreads();
  if (tid == 0) {
    float cs = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) cs += red[w];
    a.cst[rowi] = cs;
  }
  if (a.wops && hl < 16) {
    // The matrix-core split's operands: W 2^e (largest |W| in [2^14, 2^15)) as fp16
    // Wh + Wl, channel c of this head (slot hl) at block c / 32, lane 16 ((c % 32) / 8) + hl,
    // element c % 8.
    float m = redm[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) m = fmaxf(m, redm[w]);
    int e = 0;
    if (m > 0.f) (void)frexpf(m, &e);
    e = m > 0.f ? 15 - e : 0;
    const size_t gset = (size_t)b * a.n_groups + g;
    if (tid == 0) a.wexp[gset * 16 + hl] = e;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + kGQThreads * i;
      if (c < D) {
        const float w = ldexpf(wvs[i], e);
        const _Float16 wh = (_Float16)w, wl = (_Float16)(w - (float)wh);
        const int l = 16 * ((c & 31) >> 3) + hl;
        uint16_t* o = a.wop + (gset * (D / 32) + (c >> 5)) * (2 * 64 * 8);
        o[l * 8 + (c & 7)] = __builtin_bit_cast(uint16_t, wh);
        o[(64 + l) * 8 + (c & 7)] = __builtin_bit_cast(uint16_t, wl);
      }
    }
  }
}

// One workgroup per (sequence, group, split of kGSplit tokens).  NQ: query heads of a group
// rounded up to a multiple of 4 (the unused ones have zero weights and are not stored).
template <int NC, int NQ>
__global__ __launch_bounds__(kGThreads) void group_split_kernel(GroupDecodeArgs a) {
  constexpr int D = 64 * NC;
  constexpr int HW = NQ / 4;                        // heads scored by each wave
  constexpr int CPT = (D + kGThreads - 1) / kGThreads;   // value channels per thread
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ float ak[kGChunk], av[kGChunk];
  __shared__ float m_run[NQ], l_run[NQ], fac[NQ], cst[NQ];
  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int len = (int)min((int64_t)max(a.seq_len[b], 0), a.cap);
  const int s0 = split * kGSplit;
  if (s0 >= len) return;                            // (whole workgroup, before any barrier)
  const int s1 = min(len, s0 + kGSplit);
  const GroupParams* pk = group_params(a.params_k, g);
  const GroupParams* pv = group_params(a.params_v, g);
  // (partial rows are [(sequence, group)][split][head])
  float* pbase = a.part + ((((size_t)b * a.n_groups + g) * a.n_splits + split) * a.heads) * (D + kGPH);
  const int rwk = a.rwk, rwv = a.rwv;
  if (pk->record_bytes != 4 * rwk || pv->record_bytes != 4 * rwv || pk->d != D || pv->d != D) {
    // caches of another record size than the parameter blocks: NaN outputs
    if (tid < a.heads) pbase[(size_t)tid * (D + kGPH)] = NAN;
    return;
  }
  const int rsk = rwk + 1, rsv = rwv + 1;           // LDS row strides (one padding dword)
  float* wl = reinterpret_cast<float*>(smem);                    // [D][NQ]
  uint32_t* kc = reinterpret_cast<uint32_t*>(wl + D * NQ);       // [kGChunk][rsk]
  uint32_t* vc = kc + kGChunk * rsk;                             // [kGChunk][rsv]
  float* pl = reinterpret_cast<float*>(vc + kGChunk * rsv);      // [kGChunk][NQ]
  uint32_t* kdesc = reinterpret_cast<uint32_t*>(pl + kGChunk * NQ);   // [D]: off | b << 16
  const size_t row0 = ((size_t)b * a.n_groups + g) * a.heads;
  for (int c = tid; c < D; c += kGThreads)
    kdesc[c] = (uint32_t)pk->bit_off[c] | ((uint32_t)pk->bits[c] << 16);
  for (int i = tid; i < D * NQ; i += kGThreads) {
    const int c = i / NQ, h = i % NQ;
    wl[i] = h < a.heads ? a.w[(row0 + h) * D + c] : 0.f;
  }
  if (tid < NQ) {
    m_run[tid] = -INFINITY;
    l_run[tid] = 0.f;
    cst[tid] = tid < a.heads ? a.cst[row0 + tid] : 0.f;
  }
  const int dak = pk->d_active;
  const bool mr_v = pv->quantizer == AATC_QUANT_MIDRISE;
  // This thread's value channels.
  int vb[CPT], vo[CPT];
  float acc[NQ][CPT];
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = tid + kGThreads * i;
    vb[i] = c < D ? pv->bits[c] : 0;
    vo[i] = c < D ? pv->bit_off[c] : 0;
#pragma unroll
    for (int h = 0; h < NQ; ++h) acc[h][i] = 0.f;
  }
  const size_t tok0 = ((size_t)b * a.n_groups + g) * (size_t)a.cap;
  const uint32_t* kw = reinterpret_cast<const uint32_t*>(a.k_codes + tok0 * pk->record_bytes);
  const uint32_t* vw = reinterpret_cast<const uint32_t*>(a.v_codes + tok0 * pv->record_bytes);
  for (int c0 = s0; c0 < s1; c0 += kGChunk) {
    const int nc = min(kGChunk, s1 - c0);
    __syncthreads();                                // the previous chunk's LDS is consumed
    for (int i = tid; i < nc * rwk; i += kGThreads) {
      const int t = i / rwk, w = i - t * rwk;
      kc[t * rsk + w] = kw[(size_t)(c0 + t) * rwk + w];
    }
    for (int i = tid; i < nc * rwv; i += kGThreads) {
      const int t = i / rwv, w = i - t * rwv;
      vc[t * rsv + w] = vw[(size_t)(c0 + t) * rwv + w];
    }
    if (tid < kGChunk) {
      kc[tid * rsk + rwk] = 0u;
      vc[tid * rsv + rwv] = 0u;
      float fk = 0.f, fv = 0.f;
      if (tid < nc) {
        fk = __half2float(__ushort_as_half(a.k_alpha[tok0 + c0 + tid]));
        fv = __half2float(__ushort_as_half(a.v_alpha[tok0 + c0 + tid]));
      }
      ak[tid] = fk;
      av[tid] = fv;
    }
    __syncthreads();
    // Scores: lane = token of the chunk, wave w = heads w HW .. w HW + HW - 1.
    {
      const bool ok = lane < nc;
      const uint32_t* krow = kc + (ok ? lane : 0) * rsk;
      float z[HW];
#pragma unroll
      for (int m = 0; m < HW; ++m) z[m] = 0.f;
#pragma unroll 4
      for (int c = 0; c < dak; ++c) {
        const uint32_t dsc = kdesc[c];
        const float cf = (float)record_code(krow, (int)(dsc & 0xffffu), (int)(dsc >> 16));
        const float* wr = wl + c * NQ + wave * HW;
#pragma unroll
        for (int m = 0; m < HW; ++m) z[m] = fmaf(wr[m], cf, z[m]);
      }
#pragma unroll
      for (int m = 0; m < HW; ++m) {
        const int h = wave * HW + m;
        const float zf = ok ? ak[lane] * (z[m] + cst[h]) : -INFINITY;
        const float mold = m_run[h];
        const float mnew = fmaxf(mold, g_wave_max(zf));
        const bool any = mnew > -INFINITY;
        const float p = (ok && any) ? __builtin_amdgcn_exp2f(zf - mnew) : 0.f;
        const float f = (any && mold > -INFINITY) ? __builtin_amdgcn_exp2f(mold - mnew) : (any ? 0.f : 1.f);
        const float ps = g_wave_sum(p);
        pl[lane * NQ + h] = p * av[lane];
        if (lane == 0) {
          m_run[h] = mnew;
          l_run[h] = l_run[h] * f + ps;
          fac[h] = f;
        }
      }
    }
    __syncthreads();
    // Values: thread = value channels tid + 256 i; every token of the chunk.
#pragma unroll
    for (int h = 0; h < NQ; ++h) {
      const float f = fac[h];
#pragma unroll
      for (int i = 0; i < CPT; ++i) acc[h][i] *= f;
    }
#pragma unroll 1
    for (int t = 0; t < nc; ++t) {
      const uint32_t* vrow = vc + t * rsv;
      float cf[CPT];
#pragma unroll
      for (int i = 0; i < CPT; ++i)
        cf[i] = vb[i] > 0 ? (float)record_code(vrow, vo[i], vb[i]) + (mr_v ? 0.5f : 0.f) : 0.f;
      const float* pr = pl + t * NQ;
#pragma unroll
      for (int h = 0; h < NQ; ++h) {
        const float p = pr[h];
#pragma unroll
        for (int i = 0; i < CPT; ++i) acc[h][i] = fmaf(p, cf[i], acc[h][i]);
      }
    }
  }
  __syncthreads();
  // Partial: (m, l) per head, o~_c = s_c 2^(1-b_c) sum_i P_i alpha_i level_ic.
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = tid + kGThreads * i;
    if (c < D) {
      const float sc = vb[i] > 0 ? ldexpf(pv->s[c], 1 - vb[i]) : 0.f;
#pragma unroll
      for (int h = 0; h < NQ; ++h)
        if (h < a.heads) pbase[(size_t)h * (D + kGPH) + kGPH + c] = acc[h][i] * sc;
    }
  }
  if (tid < a.heads) {
    pbase[(size_t)tid * (D + kGPH)] = m_run[tid];
    pbase[(size_t)tid * (D + kGPH) + 1] = l_run[tid];
  }
}

// The same split with the records of all 256 tokens in LDS (key records first, then the
// value records in the same rows) and eight waves: lane = token, waves 0-3 score the first
// half of the group's query heads for tokens 0..255 and waves 4-7 the second half (each code
// feeds NQ / 2 independent products), and thread = value channel.  Used when its LDS fits.
constexpr int kGWideThreads = 512;
template <int NC, int NQ>
__device__ inline void group_split_wide_body(const GroupDecodeArgs& a) {
  constexpr int D = 64 * NC;
  constexpr int NT = kGWideThreads;
  constexpr int HH = NQ / 2;                        // heads scored by each half
  constexpr int CPT = (D + NT - 1) / NT;
  static_assert(kGSplit == 256, "four waves of tokens");
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ float ak[kGSplit], av[kGSplit];
  __shared__ float wred[4][NQ];
  __shared__ float mh[NQ], lh[NQ], cst[NQ];
  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tok = tid & (kGSplit - 1), half = wave >> 2;
  const int len = (int)min((int64_t)max(a.seq_len[b], 0), a.cap);
  const int s0 = split * kGSplit;
  if (s0 >= len) return;                            // (whole workgroup, before any barrier)
  const int nt = min(len, s0 + kGSplit) - s0;
  const GroupParams* pk = group_params(a.params_k, g);
  const GroupParams* pv = group_params(a.params_v, g);
  float* pbase = a.part + ((((size_t)b * a.n_groups + g) * a.n_splits + split) * a.heads) * (D + kGPH);
  const int rwk = a.rwk, rwv = a.rwv;
  if (pk->record_bytes != 4 * rwk || pv->record_bytes != 4 * rwv || pk->d != D || pv->d != D) {
    if (tid < a.heads) pbase[(size_t)tid * (D + kGPH)] = NAN;
    return;
  }
  const int rs = max(rwk, rwv) + 1;                 // LDS row stride (one padding dword)
  float* wl = reinterpret_cast<float*>(smem);                      // [D][NQ]
  uint32_t* rb = reinterpret_cast<uint32_t*>(wl + D * NQ);         // [kGSplit][rs]
  float* pl = reinterpret_cast<float*>(rb + kGSplit * rs);         // [kGSplit][NQ]
  uint32_t* kdesc = reinterpret_cast<uint32_t*>(pl + kGSplit * NQ);   // [D]: off | b << 16
  const size_t row0 = ((size_t)b * a.n_groups + g) * a.heads;
  for (int i = tid; i < D * NQ; i += NT) {
    const int c = i / NQ, h = i % NQ;
    wl[i] = h < a.heads ? a.w[(row0 + h) * D + c] : 0.f;
  }
  for (int c = tid; c < D; c += NT)
    kdesc[c] = (uint32_t)pk->bit_off[c] | ((uint32_t)pk->bits[c] << 16);
  if (tid < NQ) cst[tid] = tid < a.heads ? a.cst[row0 + tid] : 0.f;
  const size_t tok0 = ((size_t)b * a.n_groups + g) * (size_t)a.cap + s0;
  const uint32_t* kw = reinterpret_cast<const uint32_t*>(a.k_codes + tok0 * pk->record_bytes);
  const uint32_t* vw = reinterpret_cast<const uint32_t*>(a.v_codes + tok0 * pv->record_bytes);
  for (int i = tid; i < nt * rwk; i += NT) {
    const int t = i / rwk, w = i - t * rwk;
    rb[t * rs + w] = kw[i];
  }
  if (tid < kGSplit) {
    rb[tid * rs + rwk] = 0u;
    float fk = 0.f, fv = 0.f;
    if (tid < nt) {
      fk = __half2float(__ushort_as_half(a.k_alpha[tok0 + tid]));
      fv = __half2float(__ushort_as_half(a.v_alpha[tok0 + tid]));
    }
    ak[tid] = fk;
    av[tid] = fv;
  }
  __syncthreads();
  // Scores of token `tok` for heads half HH .. half HH + HH - 1.
  const bool ok = tok < nt;
  float z[HH];
  {
    const uint32_t* krow = rb + (ok ? tok : 0) * rs;
#pragma unroll
    for (int h = 0; h < HH; ++h) z[h] = 0.f;
    const int dak = pk->d_active;
    const float* wh = wl + half * HH;
#pragma unroll 2
    for (int c = 0; c < dak; ++c) {
      const uint32_t dsc = kdesc[c];
      const float cf = (float)record_code(krow, (int)(dsc & 0xffffu), (int)(dsc >> 16));
      const float* wc = wh + c * NQ;
      if constexpr (HH % 4 == 0) {
#pragma unroll
        for (int q = 0; q < HH / 4; ++q) {
          const float4 w4 = reinterpret_cast<const float4*>(wc)[q];
          z[4 * q] = fmaf(w4.x, cf, z[4 * q]);
          z[4 * q + 1] = fmaf(w4.y, cf, z[4 * q + 1]);
          z[4 * q + 2] = fmaf(w4.z, cf, z[4 * q + 2]);
          z[4 * q + 3] = fmaf(w4.w, cf, z[4 * q + 3]);
        }
      } else {
#pragma unroll
        for (int h = 0; h < HH; ++h) z[h] = fmaf(wc[h], cf, z[h]);
      }
    }
    const float akt = ak[tok];
#pragma unroll
    for (int i = 0; i < HH; ++i) {
      z[i] = ok ? akt * (z[i] + cst[half * HH + i]) : -INFINITY;
      const float m = g_wave_max(z[i]);
      if (lane == 0) wred[wave & 3][half * HH + i] = m;
    }
  }
  __syncthreads();                                  // (every key record read, maxima in)
  if (tid < NQ) mh[tid] = fmaxf(fmaxf(wred[0][tid], wred[1][tid]), fmaxf(wred[2][tid], wred[3][tid]));
  for (int i = tid; i < nt * rwv; i += NT) {
    const int t = i / rwv, w = i - t * rwv;
    rb[t * rs + w] = vw[i];
  }
  if (tid < kGSplit) rb[tid * rs + rwv] = 0u;
  __syncthreads();
  {
    const float avt = av[tok];
#pragma unroll
    for (int i = 0; i < HH; ++i) {
      const int h = half * HH + i;
      const float p = ok ? __builtin_amdgcn_exp2f(z[i] - mh[h]) : 0.f;
      pl[tok * NQ + h] = p * avt;
      const float ps = g_wave_sum(p);
      if (lane == 0) wred[wave & 3][h] = ps;
    }
  }
  __syncthreads();
  if (tid < NQ) lh[tid] = (wred[0][tid] + wred[1][tid]) + (wred[2][tid] + wred[3][tid]);
  // Values: thread = channels tid + 512 i, every token, every head.
  const bool mr_v = pv->quantizer == AATC_QUANT_MIDRISE;
  int vb[CPT], vo[CPT];
  float acc[NQ][CPT];
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = tid + NT * i;
    vb[i] = c < D ? pv->bits[c] : 0;
    vo[i] = c < D ? pv->bit_off[c] : 0;
#pragma unroll
    for (int h = 0; h < NQ; ++h) acc[h][i] = 0.f;
  }
  bool any = false;
#pragma unroll
  for (int i = 0; i < CPT; ++i) any = any || vb[i] > 0;
  if (any) {
#pragma unroll 2
    for (int t = 0; t < nt; ++t) {
      const uint32_t* vrow = rb + t * rs;
      float cf[CPT];
#pragma unroll
      for (int i = 0; i < CPT; ++i)
        cf[i] = vb[i] > 0 ? (float)record_code(vrow, vo[i], vb[i]) + (mr_v ? 0.5f : 0.f) : 0.f;
      const float4* pr = reinterpret_cast<const float4*>(pl + t * NQ);
#pragma unroll
      for (int q = 0; q < NQ / 4; ++q) {
        const float4 p4 = pr[q];
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
          acc[4 * q][i] = fmaf(p4.x, cf[i], acc[4 * q][i]);
          acc[4 * q + 1][i] = fmaf(p4.y, cf[i], acc[4 * q + 1][i]);
          acc[4 * q + 2][i] = fmaf(p4.z, cf[i], acc[4 * q + 2][i]);
          acc[4 * q + 3][i] = fmaf(p4.w, cf[i], acc[4 * q + 3][i]);
        }
      }
    }
  }
  __syncthreads();                                  // (mh, lh written)
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = tid + NT * i;
    if (c < D) {
      const float sc = vb[i] > 0 ? ldexpf(pv->s[c], 1 - vb[i]) : 0.f;
#pragma unroll
      for (int h = 0; h < NQ; ++h)
        if (h < a.heads) pbase[(size_t)h * (D + kGPH) + kGPH + c] = acc[h][i] * sc;
    }
  }
  if (tid < a.heads) {
    pbase[(size_t)tid * (D + kGPH)] = mh[tid];
    pbase[(size_t)tid * (D + kGPH) + 1] = lh[tid];
  }
}

template <int NC, int NQ>
__global__ __launch_bounds__(kGWideThreads) void group_split_wide_kernel(GroupDecodeArgs a) {
  group_split_wide_body<NC, NQ>(a);
}

// Loads of one staging pass: dwords i0 + u NT (u < kGStageU) of the records (the index past
// the end clamped to the last dword), all issued before any is used.
constexpr int kGStageU = 24;
template <int NT>
__device__ inline void stage_load(const uint32_t* src, int total, int i0, uint32_t (&v)[kGStageU]) {
#pragma unroll
  for (int u = 0; u < kGStageU; ++u) v[u] = src[min(i0 + u * NT, total - 1)];
}
// Their stores into LDS rows of rs dwords (token t = i / rw as the high half of
// i ceil(2^32 / rw): exact for i < 2^32 / rw).
template <int NT>
__device__ inline void stage_store(uint32_t* rb, int rs, int total, int rw, int i0,
                                   const uint32_t (&v)[kGStageU]) {
  const uint32_t mk = rw > 1 ? (uint32_t)((0x100000000ull + (uint32_t)rw - 1u) / (uint32_t)rw) : 0u;
#pragma unroll
  for (int u = 0; u < kGStageU; ++u) {
    const int i = i0 + u * NT;
    if (i < total) {
      const int t = rw > 1 ? (int)__umulhi((uint32_t)i, mk) : i;
      rb[t * rs + (i - t * rw)] = v[u];
    }
  }
}
// The records of tokens 0 .. nt-1 (rw dwords each, contiguous at src) into LDS rows, one
// round trip per pass of kGStageU dwords per thread.
template <int NT>
__device__ inline void stage_records(uint32_t* rb, int rs, const uint32_t* src, int nt, int rw) {
  const int total = nt * rw;
  for (int i0 = threadIdx.x; i0 < total; i0 += NT * kGStageU) {
    uint32_t v[kGStageU];
    stage_load<NT>(src, total, i0, v);
    stage_store<NT>(rb, rs, total, rw, i0, v);
  }
}

// The same with 16-byte loads (src 16-byte aligned, total >= 4): the whole uint4s of the
// records, the last total % 4 dwords by single loads; kGStage4 uint4 per thread and pass.
constexpr int kGStage4 = 6;
template <int NT>
__device__ inline void stage4_load(const uint32_t* src, int total, int j0, uint4 (&v)[kGStage4],
                                   uint32_t& tail) {
  const uint4* s4 = reinterpret_cast<const uint4*>(src);
  const int n4 = total >> 2;
#pragma unroll
  for (int u = 0; u < kGStage4; ++u) v[u] = s4[min(j0 + u * NT, n4 - 1)];   // (n4 >= 1)
  const int it = 4 * n4 + (int)threadIdx.x;
  tail = it < total ? src[it] : 0u;
}
template <int NT>
__device__ inline void stage4_store(uint32_t* rb, int rs, int total, int rw, int j0,
                                    const uint4 (&v)[kGStage4], uint32_t tail, bool first) {
  const uint32_t mk = rw > 1 ? (uint32_t)((0x100000000ull + (uint32_t)rw - 1u) / (uint32_t)rw) : 0u;
  auto put = [&](int i, uint32_t x) {
    const int t = rw > 1 ? (int)__umulhi((uint32_t)i, mk) : i;
    rb[t * rs + (i - t * rw)] = x;
  };
  const int n4 = total >> 2;
#pragma unroll
  for (int u = 0; u < kGStage4; ++u) {
    const int j = j0 + u * NT;
    if (j < n4) {
      put(4 * j, v[u].x);
      put(4 * j + 1, v[u].y);
      put(4 * j + 2, v[u].z);
      put(4 * j + 3, v[u].w);
    }
  }
  const int it = 4 * n4 + (int)threadIdx.x;
  if (first && it < total) put(it, tail);
}
// The records into LDS rows: 16-byte loads when src is aligned, one round trip per pass.
template <int NT>
__device__ inline void stage_records_any(uint32_t* rb, int rs, const uint32_t* src, int nt, int rw) {
  const int total = nt * rw;
  if (total <= 0) return;
  if ((reinterpret_cast<uintptr_t>(src) & 15u) == 0u && total >= 4) {
    // (every thread takes the first pass: it also carries the tail dwords)
    for (int j0 = threadIdx.x; j0 == (int)threadIdx.x || j0 < (total >> 2); j0 += NT * kGStage4) {
      uint4 v[kGStage4];
      uint32_t tail;
      stage4_load<NT>(src, total, j0, v, tail);
      stage4_store<NT>(rb, rs, total, rw, j0, v, tail, j0 == (int)threadIdx.x);
    }
  } else {
    stage_records<NT>(rb, rs, src, nt, rw);
  }
}

// The same split on the matrix cores (up to 16 query heads per group, codes of at most 12
// bits, which fp16 holds exactly): eight waves, the records of all 256 tokens in LDS.
//   - Scores: v_mfma_f32_16x16x32_f16 with A = the query weights (16 heads x 32 channels)
//     and B = the codes of 16 tokens (32 channels x 16 tokens).  Each head's weights come
//     scaled by a power of two (largest |W| in [2^14, 2^15)) and split into fp16 parts
//     W' = Wh + Wl (written by group_query_kernel), both multiplied with the same codes into
//     one fp32 sum (products exact, |W' - Wh - Wl| <= 2^-22 |W'|).
//   - Values: A = P (16 heads x 32 tokens), P = p alpha^V scaled by a power of two (largest
//     alpha^V of the split in [2^13, 2^14)) and split the same way, B = the codes of 16
//     channels over those 32 tokens.  The midrise half step is 1/2 sum_t P, added once.
// Operand layouts (lane 16 kg + n): A row n, k = 8 kg .. 8 kg + 7; B column n, the same k;
// the 16 x 16 result row 4 kg + i, column n in element i.
// DUAL: key and value records in LDS together, every load of the split issued at the start
// (P then reuses the key rows); otherwise the value records replace the key records after
// the scores.  A workgroup whose codes are wider takes the VALU body above (uniform).
typedef _Float16 gh8 __attribute__((ext_vector_type(8)));
typedef float gf4 __attribute__((ext_vector_type(4)));
constexpr int kGPRow = kGSplit + 8;              // halves per head row of P (rows 4 banks
                                                 // apart: conflict-free operand reads)
constexpr size_t kGPBytes = (size_t)2 * 16 * kGPRow * 2;
constexpr size_t kGMfmaLdsCap = 144 * 1024;       // dynamic LDS of the matrix-core split

template <int NC>
inline constexpr size_t group_mfma_lds(int rw_max, bool dual) {
  const size_t rows = (size_t)kGSplit * (rw_max + 1) * 4;
  return (size_t)(64 * NC / 32) * 2 * 64 * 16 +               // weight operands
         (size_t)2 * 64 * NC * 4 +                              // key and value descriptors
         (dual ? std::max(rows, kGPBytes) + rows : rows + kGPBytes);
}

template <int NC, bool DUAL>
__global__ __launch_bounds__(kGWideThreads) void group_split_mfma_kernel(GroupDecodeArgs a) {
  constexpr int D = 64 * NC;
  constexpr int NT = kGWideThreads;
  constexpr int NKB = D / 32;                       // channel blocks of the score products
  constexpr int NCB = D / 16;                       // channel blocks of the value products
  constexpr int W4 = NKB * 128 / NT;                // 16-byte operand loads per thread
  static_assert(kGSplit == 256, "eight waves of 32 tokens");
  static_assert(NKB * 128 % NT == 0, "whole operand loads");
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ float ak[kGSplit], av[kGSplit];
  __shared__ float wred[8][16], wred2[8][16];
  __shared__ float mh[16], lh[16], ph_sum[16], cst[16];
  __shared__ int wexp[16];
  __shared__ int pexp;
  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, n = lane & 15, kg = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int len = (int)min((int64_t)max(a.seq_len[b], 0), a.cap);
  const int s0 = split * kGSplit;
  if (s0 >= len) return;                            // (whole workgroup, before any barrier)
  const GroupParams* pk = group_params(a.params_k, g);
  const GroupParams* pv = group_params(a.params_v, g);
  if (pk->max_bits > 12 || pv->max_bits > 12) {
    group_split_wide_body<NC, 16>(a);
    return;
  }
  const int nt = min(len, s0 + kGSplit) - s0;
  float* pbase = a.part + ((((size_t)b * a.n_groups + g) * a.n_splits + split) * a.heads) * (D + kGPH);
  const int rwk = a.rwk, rwv = a.rwv;
  if (pk->record_bytes != 4 * rwk || pv->record_bytes != 4 * rwv || pk->d != D || pv->d != D) {
    if (tid < a.heads) pbase[(size_t)tid * (D + kGPH)] = NAN;
    return;
  }
  const int rs = max(rwk, rwv) + 1;                 // LDS row stride (one padding dword)
  const size_t rows_b = (size_t)kGSplit * rs * 4;
  gh8* wop = reinterpret_cast<gh8*>(smem);                                  // [NKB][2][64]
  uint32_t* kdesc = reinterpret_cast<uint32_t*>(wop + NKB * 2 * 64);        // [D]: off | b << 16
  uint32_t* vdesc = kdesc + D;
  uint32_t* rbk = vdesc + D;                                                // [kGSplit][rs]
  uint32_t* rbv = DUAL ? reinterpret_cast<uint32_t*>(reinterpret_cast<uint8_t*>(rbk) +
                                                     std::max(rows_b, kGPBytes))
                       : rbk;
  _Float16* pl = DUAL ? reinterpret_cast<_Float16*>(rbk)                    // [2][16][kGPRow]
                      : reinterpret_cast<_Float16*>(reinterpret_cast<uint8_t*>(rbk) + rows_b);
  const size_t gset = (size_t)b * a.n_groups + g;
  const size_t row0 = gset * a.heads;
  const size_t tok0 = gset * (size_t)a.cap + s0;
  const uint32_t* kw = reinterpret_cast<const uint32_t*>(a.k_codes + tok0 * pk->record_bytes);
  const uint32_t* vw = reinterpret_cast<const uint32_t*>(a.v_codes + tok0 * pv->record_bytes);
  // (1) Every load first: the weight operands, the records (the first pass of each, 16-byte
  //     loads where the records are aligned), the scales, descriptors and constants; then
  //     the stores.
  auto stage_all = [&]() {
    const uint4* wsrc = reinterpret_cast<const uint4*>(a.wop) + gset * (NKB * 128);
    uint4 wv4[W4];
    const int totk = nt * rwk, totv = nt * rwv;
    const bool vec = ((reinterpret_cast<uintptr_t>(kw) | reinterpret_cast<uintptr_t>(vw)) & 15u) == 0u &&
                     totk >= 4 && totv >= 4 && totk <= 4 * NT * kGStage4 && totv <= 4 * NT * kGStage4;
    if (DUAL && vec) {                              // (uniform; no branch among the loads)
      uint4 vk[kGStage4], vv[kGStage4];
      uint32_t tk, tv;
#pragma unroll
      for (int i = 0; i < W4; ++i) wv4[i] = wsrc[tid + NT * i];
      stage4_load<NT>(kw, totk, tid, vk, tk);
      stage4_load<NT>(vw, totv, tid, vv, tv);
#pragma unroll
      for (int i = 0; i < W4; ++i) reinterpret_cast<uint4*>(wop)[tid + NT * i] = wv4[i];
      stage4_store<NT>(rbk, rs, totk, rwk, tid, vk, tk, true);
      stage4_store<NT>(rbv, rs, totv, rwv, tid, vv, tv, true);
    } else {
#pragma unroll
      for (int i = 0; i < W4; ++i) wv4[i] = wsrc[tid + NT * i];
#pragma unroll
      for (int i = 0; i < W4; ++i) reinterpret_cast<uint4*>(wop)[tid + NT * i] = wv4[i];
      stage_records_any<NT>(rbk, rs, kw, nt, rwk);
      if constexpr (DUAL) stage_records_any<NT>(rbv, rs, vw, nt, rwv);
    }
  };
  {
    // (the small loads of step (1), issued before the records' and stored after them)
    constexpr int CPT = (D + NT - 1) / NT;
    uint32_t kbits[CPT], koff[CPT], vbits[CPT], voff[CPT];
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = min(tid + NT * i, D - 1);
      kbits[i] = pk->bits[c];
      koff[i] = pk->bit_off[c];
      vbits[i] = pv->bits[c];
      voff[i] = pv->bit_off[c];
    }
    const int ti = min(tid, nt - 1);
    const uint16_t ka16 = a.k_alpha[tok0 + ti], va16 = a.v_alpha[tok0 + ti];
    const int hi = min(tid & 15, a.heads - 1);
    const float cst_v = a.cst[row0 + hi];
    const int wexp_v = a.wexp[gset * 16 + hi];
    stage_all();
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + NT * i;
      // (a dropped channel: offset 0, width 0; its code is selected to 0)
      if (c < D) {
        kdesc[c] = kbits[i] ? koff[i] | (kbits[i] << 16) : 0u;
        vdesc[c] = vbits[i] ? voff[i] | (vbits[i] << 16) : 0u;
      }
    }
    if (tid < kGSplit) {
      rbk[tid * rs + rwk] = 0u;
      if constexpr (DUAL) rbv[tid * rs + rwv] = 0u;
      ak[tid] = tid < nt ? __half2float(__ushort_as_half(ka16)) : 0.f;
      av[tid] = tid < nt ? __half2float(__ushort_as_half(va16)) : 0.f;
    }
    if (tid < 16) {
      cst[tid] = tid < a.heads ? cst_v : 0.f;
      wexp[tid] = tid < a.heads ? wexp_v : 0;
    }
  }
  __syncthreads();
  if (tid < kGSplit) {
    // the largest value scale of the split, for the exponent of P's scaling
    const float m = g_wave_max(av[tid]);
    if (lane == 0) wred2[wave][0] = m;
  }
  // (2) Scores of tokens 32 wave + 16 tb + n, heads 4 kg + i (slots past the group's heads
  //     hold other data: their operand rows are zeroed).
  // (the extract is made for every channel and a dropped one, width 0, selected to 0:
  // no branch around the LDS reads)
  auto code_of = [&](const uint32_t* row, uint32_t dsc) -> _Float16 {
    const int bw = (int)(dsc >> 16);
    const int code = record_code(row, (int)(dsc & 0xffffu), bw);
    return (_Float16)(float)(bw ? code : 0);
  };
  const bool head_ok = n < a.heads;
  gf4 zs[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  {
    const uint32_t* krow[2] = {rbk + (32 * wave + n) * rs, rbk + (32 * wave + 16 + n) * rs};
    const gh8 zero8 = {};
#pragma unroll 2
    for (int kb = 0; kb < NKB; ++kb) {
      const gh8 whi = head_ok ? wop[(2 * kb) * 64 + lane] : zero8;
      const gh8 wlo = head_ok ? wop[(2 * kb + 1) * 64 + lane] : zero8;
      const int c0 = 32 * kb + 8 * kg;
      const uint4 d0 = *reinterpret_cast<const uint4*>(kdesc + c0);
      const uint4 d1 = *reinterpret_cast<const uint4*>(kdesc + c0 + 4);
      const uint32_t dk[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        gh8 cb;
#pragma unroll
        for (int e = 0; e < 8; ++e) cb[e] = code_of(krow[tb], dk[e]);
        zs[tb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(whi, cb, zs[tb], 0, 0, 0);
        zs[tb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(wlo, cb, zs[tb], 0, 0, 0);
      }
    }
  }
  float z[2][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int h = 4 * kg + i;
    float m = -INFINITY;
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      const int t = 32 * wave + 16 * tb + n;
      z[tb][i] = t < nt ? ak[t] * (ldexpf(zs[tb][i], -wexp[h]) + cst[h]) : -INFINITY;
      m = fmaxf(m, z[tb][i]);
    }
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    if (n == 0) wred[wave][h] = m;
  }
  __syncthreads();                                  // (every key record read, maxima in)
  if (tid < 16) {
    float m = wred[0][tid];
#pragma unroll
    for (int w = 1; w < 8; ++w) m = fmaxf(m, wred[w][tid]);
    mh[tid] = m;
  }
  if (tid == 0) {
    const float m = fmaxf(fmaxf(wred2[0][0], wred2[1][0]), fmaxf(wred2[2][0], wred2[3][0]));
    int e = 0;
    if (m > 0.f) (void)frexpf(m, &e);
    pexp = m > 0.f ? 14 - e : 0;                    // max alpha^V 2^pexp in [2^13, 2^14)
  }
  if constexpr (!DUAL) {
    stage_records_any<NT>(rbv, rs, vw, nt, rwv);
    if (tid < kGSplit) rbv[tid * rs + rwv] = 0u;
  }
  __syncthreads();
  // (3) p = 2^(z - m), P = p alpha^V: the sums of p (the softmax denominator) and of P (the
  //     midrise half step), and P 2^pexp as fp16 parts in [head][token] rows.
  {
    const int pe = pexp;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * kg + i;
      float ps = 0.f, qs = 0.f;
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        const int t = 32 * wave + 16 * tb + n;
        const float p = t < nt ? __builtin_amdgcn_exp2f(z[tb][i] - mh[h]) : 0.f;
        const float pv_ = p * av[t];
        ps += p;
        qs += pv_;
        const float sp = ldexpf(pv_, pe);
        const _Float16 hh = (_Float16)sp;
        pl[h * kGPRow + t] = hh;
        pl[(16 + h) * kGPRow + t] = (_Float16)(sp - (float)hh);
      }
#pragma unroll
      for (int o = 8; o >= 1; o >>= 1) {
        ps += __shfl_xor(ps, o, 64);
        qs += __shfl_xor(qs, o, 64);
      }
      if (n == 0) {
        wred[wave][h] = ps;
        wred2[wave][h] = qs;
      }
    }
  }
  __syncthreads();
  if (tid < 16) {
    float ps = 0.f, qs = 0.f;
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      ps += wred[w][tid];
      qs += wred2[w][tid];
    }
    lh[tid] = ps;
    ph_sum[tid] = qs;
  }
  __syncthreads();
  // (4) Values: wave w takes channel blocks w, w + 8, ...; lane 16 kg + n ends with heads
  //     4 kg + i of channel 16 cb + n.
  const bool mr_v = pv->quantizer == AATC_QUANT_MIDRISE;
  const int pe = pexp;
  for (int cb = wave; cb < NCB; cb += 8) {
    const int c = 16 * cb + n;
    const uint32_t dsc = vdesc[c];
    gf4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 2
    for (int tk = 0; tk < kGSplit / 32; ++tk) {
      const int t0 = 32 * tk + 8 * kg;
      const gh8 phi = *reinterpret_cast<const gh8*>(pl + n * kGPRow + t0);
      const gh8 plo = *reinterpret_cast<const gh8*>(pl + (16 + n) * kGPRow + t0);
      gh8 cv;
#pragma unroll
      for (int e = 0; e < 8; ++e) cv[e] = code_of(rbv + (t0 + e) * rs, dsc);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(phi, cv, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(plo, cv, acc, 0, 0, 0);
    }
    const int bc = (int)(dsc >> 16);
    const float sc = bc > 0 ? ldexpf(pv->s[c], 1 - bc) : 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * kg + i;
      if (h < a.heads) {
        const float o = ldexpf(acc[i], -pe) + (mr_v ? 0.5f * ph_sum[h] : 0.f);
        pbase[(size_t)h * (D + kGPH) + kGPH + c] = o * sc;
      }
    }
  }
  if (tid < a.heads) {
    pbase[(size_t)tid * (D + kGPH)] = mh[tid];
    pbase[(size_t)tid * (D + kGPH) + 1] = lh[tid];
  }
}

// The merge in two launches, spread over (query head, channel chunk) and (query head,
// output rows) so that every CU reads a share of the split partials and of T_V.
// group_merge_sum_kernel: one workgroup per (sequence, query head, 64 channels of o~): the
// splits' maximum M and weights 2^(m_s - M) (recomputed by every chunk: a few hundred
// floats), thread (range, channel) sums one quarter of the splits with eight loads in
// flight, and o~ = sum_s w_s o~_s / sum_s w_s l_s goes to the workspace (NaN if a split
// reported mismatched records, 0 for an empty sequence).
constexpr int kGMergeThreads = 256;
constexpr int kGMergeSplits = 1024;              // splits weighted per pass
template <int NC>
__global__ __launch_bounds__(kGMergeThreads) void group_merge_sum_kernel(GroupDecodeArgs a) {
  constexpr int D = 64 * NC;
  constexpr int NT = kGMergeThreads;
  constexpr int NSUB = NT / 64;                    // split ranges per channel
  constexpr int NW = NT / 64;
  __shared__ float ot[NSUB][64];
  __shared__ float wsp[kGMergeSplits];
  __shared__ float red[NW];
  const int h = blockIdx.x / NC, ci = blockIdx.x % NC, b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int gq = a.n_q_heads / a.n_kv_heads;
  const int k = h / gq, g = k / a.gkv, hl = h - g * a.heads;
  float* otw = a.otl + ((size_t)b * a.n_q_heads + h) * D + 64 * ci;
  const int len = (int)min((int64_t)max(a.seq_len[b], 0), a.cap);
  if (len == 0) {
    if (tid < 64) otw[tid] = 0.f;
    return;
  }
  const int ns = (len + kGSplit - 1) / kGSplit;
  const float* pb = a.part + ((((size_t)b * a.n_groups + g) * a.n_splits) * a.heads + hl) * (D + kGPH);
  const size_t sstride = (size_t)a.heads * (D + kGPH);
  float mx = -INFINITY;
  for (int s = tid; s < ns; s += NT) {
    const float ms = pb[s * sstride];
    mx = ms != ms ? ms : fmaxf(mx, ms);             // (a NaN mark is kept)
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float y = __shfl_xor(mx, o, 64);
    mx = (mx != mx || y != y) ? NAN : fmaxf(mx, y);
  }
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  float M = red[0];
  for (int w = 1; w < NW; ++w) M = (M != M || red[w] != red[w]) ? NAN : fmaxf(M, red[w]);
  if (M != M) {
    if (tid < 64) otw[tid] = NAN;
    return;
  }
  const int c = tid & 63, sub = tid >> 6;
  float L = 0.f, acc = 0.f;
  for (int s0 = 0; s0 < ns; s0 += kGMergeSplits) {
    const int n = min(kGMergeSplits, ns - s0);
    __syncthreads();                                // (the previous pass's weights are read)
    float lsum = 0.f;
    for (int s = tid; s < n; s += NT) {
      const float* p = pb + (size_t)(s0 + s) * sstride;
      const float w = __builtin_amdgcn_exp2f(p[0] - M);
      wsp[s] = w;
      lsum = fmaf(w, p[1], lsum);
    }
    lsum = g_wave_sum(lsum);
    __syncthreads();
    if (lane == 0) red[wave] = lsum;
    __syncthreads();
    for (int w = 0; w < NW; ++w) L += red[w];
    const int lo = n * sub / NSUB, hi = n * (sub + 1) / NSUB;
    const float* p = pb + kGPH + 64 * ci + c + (size_t)s0 * sstride;
    float a0 = 0.f, a1 = 0.f;
    int s = lo;
    for (; s + 8 <= hi; s += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = p[(size_t)(s + u) * sstride];
#pragma unroll
      for (int u = 0; u < 8; u += 2) {
        a0 = fmaf(wsp[s + u], v[u], a0);
        a1 = fmaf(wsp[s + u + 1], v[u + 1], a1);
      }
    }
    for (; s < hi; ++s) a0 = fmaf(wsp[s], p[(size_t)s * sstride], a0);
    acc += a0 + a1;
  }
  ot[sub][c] = acc;
  __syncthreads();
  if (tid < 64) {
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < NSUB; ++u) v += ot[u][tid];
    otw[tid] = v * (L > 0.f ? 1.f / L : 0.f);
  }
}

// group_merge_apply_kernel: one workgroup per (sequence, query head, 32 output rows):
// o_j = sum_c T_V[128 kk + j][c] o~_c, thread (row, part) over D / 8 consecutive channels
// (every load of its slice in flight at once), the eight parts met by shuffles.
constexpr int kGApplyRows = 32;
template <int NC>
__global__ __launch_bounds__(256) void group_merge_apply_kernel(GroupDecodeArgs a) {
  constexpr int D = 64 * NC;
  constexpr int PC = D / 8;                         // channels per part (a multiple of 16)
  const int h = blockIdx.x / (128 / kGApplyRows), jq = blockIdx.x % (128 / kGApplyRows);
  const int b = blockIdx.y, tid = threadIdx.x;
  const int gq = a.n_q_heads / a.n_kv_heads;
  const int k = h / gq, g = k / a.gkv, kk = k % a.gkv;
  const int j = kGApplyRows * jq + (tid >> 3), part = tid & 7;
  const GroupParams* pv = group_params(a.params_v, g);
  const float4* trow = reinterpret_cast<const float4*>(pv->T + (size_t)(kk * 128 + j) * D + part * PC);
  const float4* ov = reinterpret_cast<const float4*>(a.otl + ((size_t)b * a.n_q_heads + h) * D + part * PC);
  float4 tv[PC / 4], o4[PC / 4];
#pragma unroll
  for (int q = 0; q < PC / 4; ++q) {
    tv[q] = trow[q];
    o4[q] = ov[q];
  }
  float v = 0.f;
#pragma unroll
  for (int q = 0; q < PC / 4; ++q) {
    v = fmaf(tv[q].x, o4[q].x, v);
    v = fmaf(tv[q].y, o4[q].y, v);
    v = fmaf(tv[q].z, o4[q].z, v);
    v = fmaf(tv[q].w, o4[q].w, v);
  }
#pragma unroll
  for (int o = 4; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  if (part == 0) a.out[((int64_t)b * a.n_q_heads + h) * 128 + j] = v;
}

// The dynamic LDS limit of one kernel on the current device, raised once per device when a
// launch first needs more (an idempotent attribute call; the recorded limit only grows).
struct GroupLds {
  std::atomic<size_t> set[64] = {};
  bool ensure(const void* kernel, size_t lds) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return false;
    if (dev < 0 || dev >= 64)
      return hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)lds) == hipSuccess;
    size_t cur = set[dev].load(std::memory_order_acquire);
    if (lds <= cur) return true;
    if (hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
        hipSuccess)
      return false;
    while (cur < lds && !set[dev].compare_exchange_weak(cur, lds, std::memory_order_acq_rel)) {
    }
    return true;
  }
};

// Whether the matrix-core split fits (its LDS, and that of the VALU body it falls back to
// for codes over 12 bits, with 16 head slots); *lds gets the size, and the result is true
// when both record sets fit at once (DUAL).
template <int NC>
bool group_mfma_fit(int rwk, int rwv, size_t* lds) {
  constexpr int D = 64 * NC;
  const int rwm = std::max(rwk, rwv);
  const size_t w16 = sizeof(float) * (size_t)D * 16 + sizeof(uint32_t) * (size_t)kGSplit * (rwm + 1) +
                     sizeof(float) * (size_t)kGSplit * 16 + sizeof(uint32_t) * D;
  const size_t m2 = std::max(w16, group_mfma_lds<NC>(rwm, true));
  const size_t m1 = std::max(w16, group_mfma_lds<NC>(rwm, false));
  *lds = m2 <= kGMfmaLdsCap ? m2 : m1 <= kGMfmaLdsCap ? m1 : 0;
  return m2 <= kGMfmaLdsCap;
}

template <int NC, int NQ>
aatc_status launch_split(const GroupDecodeArgs& a, int batch, int rwk, int rwv,
                         hipStream_t st) {
  constexpr int D = 64 * NC;
  const size_t lds_wide = sizeof(float) * (size_t)D * NQ +
                          sizeof(uint32_t) * (size_t)kGSplit * (std::max(rwk, rwv) + 1) +
                          sizeof(float) * (size_t)kGSplit * NQ + sizeof(uint32_t) * D;
  const dim3 grid((unsigned)a.n_splits, (unsigned)a.n_groups, (unsigned)batch);
  if constexpr (NQ <= 16) {
    if (a.wops) {
      size_t lds = 0;
      const bool dual = group_mfma_fit<NC>(rwk, rwv, &lds);
      if (dual) {
        static GroupLds limit_m2;
        if (!limit_m2.ensure((const void*)group_split_mfma_kernel<NC, true>, lds))
          return AATC_E_DEVICE;
        hipLaunchKernelGGL((group_split_mfma_kernel<NC, true>), grid, dim3(kGWideThreads), lds,
                           st, a);
      } else {
        static GroupLds limit_m1;
        if (!limit_m1.ensure((const void*)group_split_mfma_kernel<NC, false>, lds))
          return AATC_E_DEVICE;
        hipLaunchKernelGGL((group_split_mfma_kernel<NC, false>), grid, dim3(kGWideThreads), lds,
                           st, a);
      }
      return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
    }
  }
  if (lds_wide <= 144 * 1024) {
    static GroupLds limit_wide;
    if (!limit_wide.ensure((const void*)group_split_wide_kernel<NC, NQ>, lds_wide))
      return AATC_E_DEVICE;
    hipLaunchKernelGGL((group_split_wide_kernel<NC, NQ>), grid, dim3(kGWideThreads), lds_wide,
                       st, a);
    return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
  }
  const size_t lds = sizeof(float) * (size_t)D * NQ +
                     sizeof(uint32_t) * (size_t)kGChunk * (rwk + 1 + rwv + 1) +
                     sizeof(float) * (size_t)kGChunk * NQ + sizeof(uint32_t) * D;
  if (lds > 150 * 1024) return AATC_E_UNSUPPORTED;
  static GroupLds limit;
  if (!limit.ensure((const void*)group_split_kernel<NC, NQ>, lds)) return AATC_E_DEVICE;
  hipLaunchKernelGGL((group_split_kernel<NC, NQ>),
                     dim3((unsigned)a.n_splits, (unsigned)a.n_groups, (unsigned)batch),
                     dim3(kGThreads), lds, st, a);
  return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
}

template <int NC>
aatc_status launch_decode_nc(GroupDecodeArgs a, int batch, int rwk, int rwv, hipStream_t st) {
  size_t lds_m = 0;
  (void)group_mfma_fit<NC>(rwk, rwv, &lds_m);
  a.wops = a.heads <= 16 && lds_m > 0 ? 1 : 0;      // the query kernel writes the operands
  hipLaunchKernelGGL((group_query_kernel<NC>), dim3((unsigned)a.n_q_heads, (unsigned)batch),
                     dim3(kGQThreads), 0, st, a);
  if (hipGetLastError() != hipSuccess) return AATC_E_DEVICE;
  aatc_status s;
  if (a.heads <= 4) s = launch_split<NC, 4>(a, batch, rwk, rwv, st);
  else if (a.heads <= 8) s = launch_split<NC, 8>(a, batch, rwk, rwv, st);
  else if (a.heads <= 16) s = launch_split<NC, 16>(a, batch, rwk, rwv, st);
  else s = launch_split<NC, 32>(a, batch, rwk, rwv, st);
  if (s != AATC_OK) return s;
  hipLaunchKernelGGL((group_merge_sum_kernel<NC>),
                     dim3((unsigned)(a.n_q_heads * NC), (unsigned)batch), dim3(kGMergeThreads), 0,
                     st, a);
  if (hipGetLastError() != hipSuccess) return AATC_E_DEVICE;
  hipLaunchKernelGGL((group_merge_apply_kernel<NC>),
                     dim3((unsigned)(a.n_q_heads * (128 / kGApplyRows)), (unsigned)batch),
                     dim3(256), 0, st, a);
  return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
}

}  // namespace

aatc_status launch_group_encode(const void* params, int n_groups, int gkv, const void* x,
                                aatc_dtype x_dtype, int64_t n_tok, int64_t x_tok_stride,
                                void* codes, uint16_t* alpha, int64_t cap, int64_t pos,
                                void* stream) {
  if (n_tok == 0) return AATC_OK;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t per_block = (int64_t)(kGThreads / 64) * kGTokensPerWave;
  const int64_t blocks = (n_tok + per_block - 1) / per_block;
  if (blocks > 0x7fffffff) return AATC_E_UNSUPPORTED;
  const dim3 grid((unsigned)blocks, (unsigned)n_groups);
  auto* c8 = static_cast<uint8_t*>(codes);
#define AATC_GENC(NC)                                                                     \
  hipLaunchKernelGGL(group_encode_kernel<NC>, grid, dim3(kGThreads), 0, st, params, x,   \
                     (int)x_dtype, n_tok, x_tok_stride, c8, alpha, cap, pos)
  switch (gkv) {
    case 1: AATC_GENC(2); break;
    case 2: AATC_GENC(4); break;
    case 3: AATC_GENC(6); break;
    case 4: AATC_GENC(8); break;
    default: return AATC_E_UNSUPPORTED;
  }
#undef AATC_GENC
  return hipGetLastError() == hipSuccess ? AATC_OK : AATC_E_DEVICE;
}

size_t group_decode_workspace_bytes(int batch, int n_q_heads, int n_kv_heads, int gkv,
                                    int64_t cap) {
  const int n_groups = n_kv_heads / gkv;
  const int heads = n_q_heads / n_groups;
  return group_ws_layout(batch, n_groups, heads, 128 * gkv, cap).total;
}

aatc_status launch_group_decode(const void* params_k, const void* params_v, int batch,
                                int n_q_heads, int n_kv_heads, int gkv, const void* q,
                                aatc_dtype q_dtype, const void* k_codes,
                                const uint16_t* k_alpha, const void* v_codes,
                                const uint16_t* v_alpha, const int32_t* seq_len, int64_t cap,
                                int k_record_bytes, int v_record_bytes, float softmax_scale,
                                float* out, void* workspace, void* stream) {
  const hipStream_t st = static_cast<hipStream_t>(stream);
  GroupDecodeArgs a{};
  a.params_k = params_k;
  a.params_v = params_v;
  a.q = q;
  a.q_dtype = (int)q_dtype;
  a.k_codes = static_cast<const uint8_t*>(k_codes);
  a.k_alpha = k_alpha;
  a.v_codes = static_cast<const uint8_t*>(v_codes);
  a.v_alpha = v_alpha;
  a.seq_len = seq_len;
  a.cap = cap;
  a.n_q_heads = n_q_heads;
  a.n_kv_heads = n_kv_heads;
  a.gkv = gkv;
  a.n_groups = n_kv_heads / gkv;
  a.heads = n_q_heads / a.n_groups;
  a.scale_log2e = softmax_scale * 1.4426950408889634f;
  const GroupWs l = group_ws_layout(batch, a.n_groups, a.heads, 128 * gkv, cap);
  a.n_splits = l.n_splits;
  if ((int64_t)l.n_splits > 0xffff || batch > 0xffff) return AATC_E_UNSUPPORTED;
  char* ws = static_cast<char*>(workspace);
  a.w = reinterpret_cast<float*>(ws + l.w);
  a.cst = reinterpret_cast<float*>(ws + l.c);
  a.part = reinterpret_cast<float*>(ws + l.partials);
  a.wop = reinterpret_cast<uint16_t*>(ws + l.wop);
  a.wexp = reinterpret_cast<int32_t*>(ws + l.wexp);
  a.otl = reinterpret_cast<float*>(ws + l.ot);
  a.out = out;
  const int rwk = k_record_bytes / 4, rwv = v_record_bytes / 4;
  a.rwk = rwk;
  a.rwv = rwv;
  switch (gkv) {
    case 1: return launch_decode_nc<2>(a, batch, rwk, rwv, st);
    case 2: return launch_decode_nc<4>(a, batch, rwk, rwv, st);
    case 3: return launch_decode_nc<6>(a, batch, rwk, rwv, st);
    case 4: return launch_decode_nc<8>(a, batch, rwk, rwv, st);
  }
  return AATC_E_UNSUPPORTED;
}

}  // namespace aatc
