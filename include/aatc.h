/*
 * aatc.h -- C ABI of the Attention-Aware Transform Coding (AATC) hot path on MI355X.
 *
 * AATC ("KV Cache Compression Through the Lens of Transform Coding") stores each key
 * and value vector of a KV head in a calibrated decorrelated basis, quantizing every
 * transformed channel with its own bit width (0 bits drops the channel), and runs
 * decode attention directly on the packed cache.
 *
 * Conventions shared by every entry point:
 *   - Head dimension d is 128; other values return AATC_E_UNSUPPORTED.  The head-group
 *     entry points (aatc_*group*, at the end) take groups of 128 gkv channels, gkv <= 4.
 *   - Channel widths are 0..16 bits (b_max <= 16; App. E allows 0 to 16 bits).
 *   - "Device" pointers are HIP device memory owned by the caller; "host" pointers are
 *     ordinary host memory.  Device buffers are 16-byte aligned unless stated
 *     otherwise.  The library allocates no device memory, never frees
 *     caller memory and never synchronizes a stream.
 *   - Every call validates its arguments on the host and returns AATC_E_INVALID
 *     (or AATC_E_UNSUPPORTED) before launching anything.  Launch failures return
 *     AATC_E_DEVICE.  No C++ exception crosses this interface.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Kernels are enqueued on
 *     it and run asynchronously.
 *   - The library is stateless and thread-safe.
 *
 * Cache layouts (per sequence; B_b = sum of a tensor's channel widths, the "budget",
 * R = 4 * ceil(B_b / 32) bytes per token):
 *   - Codes are stored as b_c-bit two's complement patterns.
 *   - RECORDS (used for keys): [n_kv_heads][cap][R] bytes.  Token t's codes are one
 *     LSB-first bit string: storage channel c occupies bits [o_c, o_c + b_c), o_c the
 *     sum of the earlier widths; bit i is bit (i % 8) of byte (i / 8); zero padded.
 *   - TILES (used for values): [n_kv_heads][cap / 64][64 * R] bytes.  Tile j holds
 *     tokens 64 j .. 64 j + 63 bit-transposed: record bit v of token 64 j + t, with
 *     t = 16 d + 4 g + i (d, g, i in 0..3), is bit 8 i + 2 g + (d mod 2) of the
 *     little-endian 32-bit word 2 v + d / 2 of the tile.  cap must be a multiple of
 *     64.  (This order makes the decode kernel's value operands line up with its
 *     score outputs.)
 *   - Token scales alpha: [n_kv_heads][cap] fp16 bit patterns, for either layout.
 */
#ifndef AATC_H_
#define AATC_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define AATC_HEAD_DIM 128
#define AATC_MAX_BITS 16
#define AATC_TILE_TOKENS 64

typedef enum {
  AATC_OK = 0,
  AATC_E_INVALID = 1,      /* bad pointer, size, alignment or combination */
  AATC_E_UNSUPPORTED = 2,  /* valid request outside what v1 implements (d != 128) */
  AATC_E_NUMERIC = 3,      /* non-finite input or eigensolver failure */
  AATC_E_DEVICE = 4,       /* a HIP call or kernel launch failed */
  AATC_E_WORKSPACE = 5     /* workspace too small */
} aatc_status;

typedef enum { AATC_F32 = 0, AATC_BF16 = 1, AATC_F16 = 2 } aatc_dtype;

typedef enum { AATC_LAYOUT_RECORDS = 0, AATC_LAYOUT_TILES = 1 } aatc_layout;

/*
 * The two readings of the Sec. 5.2 quantizer (Delta = 2 alpha s_c / 2^b_c; codes stored
 * as b-bit two's complement either way):
 *   AATC_QUANT_MIDTREAD  the printed formula: code = clamp(floor(h / Delta + 1/2),
 *                        -2^(b-1), 2^(b-1) - 1), level code * Delta;
 *   AATC_QUANT_MIDRISE   the symmetric quantizer of Sec. 4's remark and App. B's noise
 *                        model: code = clamp(floor(h / Delta), -2^(b-1), 2^(b-1) - 1),
 *                        level (code + 1/2) Delta (error at most Delta / 2 everywhere).
 */
typedef enum { AATC_QUANT_MIDTREAD = 0, AATC_QUANT_MIDRISE = 1 } aatc_quantizer;

/*
 * Calibration artifact of one (KV head, tensor), channels in storage order (widest
 * first; eigen order breaks ties, so zero-bit channels form a suffix).
 */
typedef struct {
  int32_t d;                    /* head dimension (128) */
  int32_t budget_bits;          /* B = sum of bits */
  int32_t record_bytes;         /* R = 4 * ceil(B / 32) */
  int32_t d_active;             /* channels with >= 1 bit */
  int32_t quantizer;            /* aatc_quantizer: AATC_QUANT_MIDTREAD from the calibrate
                                   entry points; set it before aatc_params_pack for the
                                   midrise reading (widths and scales do not depend on it) */
  float transform[AATC_HEAD_DIM * AATC_HEAD_DIM]; /* row-major [j][c] = T_jc: column c
                                   is the unit eigenvector of storage channel c, stored
                                   on the 2^-22 grid (every entry a multiple of 2^-22,
                                   |T_jc| <= 1, so exactly an fp32 number) */
  uint8_t bits[AATC_HEAD_DIM];  /* width of storage channel c, non-increasing */
  uint16_t scale_f16[AATC_HEAD_DIM]; /* s_c as fp16 bits (0 for dropped channels) */
  int32_t perm[AATC_HEAD_DIM];  /* eigen index (by decreasing eigenvalue) of channel c */
  double sigma2[AATC_HEAD_DIM]; /* eigenvalues, decreasing (eigen order) */
  double weight[AATC_HEAD_DIM]; /* attention-aware channel weights w (eigen order) */
  uint8_t bits_eig[AATC_HEAD_DIM]; /* widths in eigen order */
} aatc_calibration;

/*
 * aatc_calibrate -- offline calibration of one (KV head, tensor) on the host.
 *
 * Follows Algorithm 1 (calibration part) with Sec. 5.1 (decorrelating transform) and
 * Sec. 5.2 (attention-aware reverse water-filling, "The right scaling"):
 *   Sigma = X^T X / n (uncentered, fp64); eigenvectors by decreasing eigenvalue, each
 *   signed so its largest-magnitude entry is positive (the PCA form of the whitening
 *   SVD, App. D); weights w_c = (1/T) sum over the group's query heads and tokens of
 *   (P_c^T q)^2 when q_calib is given (eq. waterfilling-keys and its GQA remark,
 *   App. B), w_c = ||P_c^T W_O||^2 when w_o is given (value weights, Sec. 5.2), else 1
 *   ("var-only", Sec. 6); integer widths minimizing sum_c w_c sigma_c^2 2^(-2 b_c)
 *   with sum_c b_c = round(avg_bits * d) and 0 <= b_c <= b_max, by exact greedy
 *   marginal allocation (ties to the lower eigen index); s_c = fp16 of the
 *   `percentile` quantile (linear interpolation) of |h_c| over the calibration tokens.
 *   The transform is stored with each entry rounded to the nearest multiple of 2^-22.
 *
 * x_calib  host [n_calib][d] fp32 calibration samples of this head (n_calib >= 2).
 * q_calib  host [n_q][d] fp32 calibration queries of the q_group query heads that
 *          share this KV head, stacked (n_q a multiple of q_group), or NULL.
 * w_o      host [d][d_out] fp32 rows of W_O that read this head's values, or NULL.
 *          At most one of q_calib / w_o may be non-NULL.
 * avg_bits average bits per channel, 0 < avg_bits * d <= d * b_max.
 * b_max    1..16.
 * percentile in (0, 1], 0.99 in the paper.
 * out      host, caller-allocated, fully written on success.
 * Errors: AATC_E_INVALID for NULL/size/range problems, AATC_E_UNSUPPORTED for
 * d != 128, AATC_E_NUMERIC for non-finite inputs or no eigensolver convergence.
 */
aatc_status aatc_calibrate(const float* x_calib, int64_t n_calib, int32_t d,
                           const float* q_calib, int64_t n_q, int32_t q_group,
                           const float* w_o, int32_t d_out,
                           double avg_bits, int32_t b_max, double percentile,
                           aatc_calibration* out);

/*
 * aatc_calibrate_whitened -- aatc_calibrate from the layer's input activations and its
 * projection, in the paper's form (Sec. 5.1 Step 1, eq. AB-factorization; App. D).
 *
 * Sigma_X = X^T X / T (fp64, uncentered); its Cholesky factor L (Sigma_X = L L^T); the
 * whitened weight W~ = L^T W; the right singular vectors P of W~ (the eigenvectors of
 * W~^T W~, by decreasing singular value, signed like aatc_calibrate's) form the basis, with
 * channel variances S_c^2 of K = X W in that basis.  The cache stores K P: it differs from
 * the paper's H = X A (A = L^-T U sqrt(S)) by a per-channel scale only, which changes no
 * code.  Weights, allocation, storage order and scales then follow aatc_calibrate, on the
 * samples K = X W (fp64).  With the same samples this is the calibration aatc_calibrate
 * returns for K (the two forms span the same channels, App. D).
 *
 * x_in     host [n_calib][d_model] fp32 input activations of the layer (n_calib >= 2;
 *          Sigma_X must be positive definite, so n_calib >= d_model in practice).
 * w_proj   host [d_model][d] fp32 key or value projection of this KV head.
 * q_calib, n_q, q_group, w_o, d_out, avg_bits, b_max, percentile, out: as in aatc_calibrate.
 * Errors: as aatc_calibrate; AATC_E_NUMERIC also when Sigma_X is not positive definite.
 */
aatc_status aatc_calibrate_whitened(const float* x_in, int64_t n_calib, int32_t d_model,
                                    const float* w_proj, int32_t d,
                                    const float* q_calib, int64_t n_q, int32_t q_group,
                                    const float* w_o, int32_t d_out, double avg_bits,
                                    int32_t b_max, double percentile, aatc_calibration* out);

/*
 * aatc_calibrate_bits -- aatc_calibrate with the widths given instead of allocated.
 *
 * For widths that come from one budget over several heads or layers (aatc_allocate_global,
 * Sec. 5.2 and Alg. 1 "allocate bits globally"): the same covariance, transform, weights,
 * storage order and scales as aatc_calibrate, with b_c = bits_eig[c] for the channel of
 * the c-th largest eigenvalue.
 *
 * bits_eig      host [d] widths in eigen order (decreasing eigenvalue), each 0..16, sum >= 1.
 * record_bytes  0 for the smallest record 4 * ceil(B / 32), else the record size to use
 *               (a multiple of 4, at least that, at most 256): the heads of one tensor
 *               whose budgets differ share the record size of the widest this way.
 * Other arguments and errors as in aatc_calibrate (avg_bits and b_max are not taken).
 */
aatc_status aatc_calibrate_bits(const float* x_calib, int64_t n_calib, int32_t d,
                                const float* q_calib, int64_t n_q, int32_t q_group,
                                const float* w_o, int32_t d_out, const uint8_t* bits_eig,
                                int32_t record_bytes, double percentile,
                                aatc_calibration* out);

/*
 * aatc_allocate_global -- integer widths of one tensor (keys or values) over all layers
 * under a single budget (host only).
 *
 * Sec. 5.2 states the water-filling problem summed over layers with one budget per
 * tensor; App. E divides each layer's variances (and the key weights) by that layer's
 * own 95th percentile, and protects the first layers with a fixed budget (the average
 * width for values, one bit more for keys).  Readings: the total is round(avg_bits m L)
 * bits; each protected layer takes round((avg_bits + protect_extra) m) and allocates it
 * over its own channels; the other layers share the rest; every allocation is the greedy
 * of aatc_calibrate (largest W_c 4^-b_c first, lowest (layer, channel) on ties) on
 * W = w' sigma2', the percentile interpolating linearly and a zero percentile leaving
 * the layer unscaled.
 *
 * sigma2   host, [n_layers][m] channel variances (eigenvalues, any channel order), >= 0.
 * weight   host, [n_layers][m] channel weights >= 0, or NULL for all ones.
 * m        channels per layer (all KV heads of the layer together).
 * b_max    1..8; n_protect >= 0 (3 in the paper; more than n_layers protects all).
 * protect_extra     bits above the average for protected layers (1 keys, 0 values).
 * normalize_weight  nonzero: the weights are scaled per layer as well (keys).
 * bits     host, caller-allocated [n_layers][m], fully written on success.
 * Errors: AATC_E_INVALID for NULL pointers, sizes or ranges, negative or non-finite
 * inputs, and budgets that no allocation in [0, b_max] meets.  A layer's heads may end with
 * different totals: aatc_calibrate_bits gives each its widths, padded to one record size
 * for the tensor (the largest 4 * ceil(B_h / 32) of the layer), which one parameter block
 * and one decode call take.
 */
aatc_status aatc_allocate_global(const double* sigma2, const double* weight,
                                 int32_t n_layers, int32_t m, double avg_bits,
                                 int32_t b_max, int32_t n_protect, int32_t protect_extra,
                                 int32_t normalize_weight, uint8_t* bits);

/*
 * aatc_params_bytes / aatc_params_pack -- build the device parameter block of one
 * tensor (K or V) for n_kv_heads heads from their calibrations (host only).
 *
 * The block holds, per head, the transform (fp32 and as the integers T * 2^22), widths,
 * bit offsets, fp16 scales and their fp32 reciprocals, and bit-to-channel tables for the
 * decoder.  All heads of a tensor must have the same record size; their budgets may
 * differ (each head's bits beyond its budget are zero padding).
 * The caller copies the `bytes` written to `host_buf` into device memory (16-byte
 * aligned) and passes that device pointer to aatc_encode / aatc_decode_attention.
 * Errors: AATC_E_INVALID (NULL, n_kv_heads < 1, bytes too small, record sizes differ,
 * malformed calibration, a transform entry off the 2^-22 grid or above 1 in magnitude).
 */
size_t aatc_params_bytes(int32_t n_kv_heads);
aatc_status aatc_params_pack(const aatc_calibration* per_head, int32_t n_kv_heads,
                             void* host_buf, size_t bytes);

/*
 * aatc_encode -- append n_tok tokens of one sequence to a compressed cache.
 *
 * Algorithm 1 (inference part: project and append quantized codes) with Sec. 5.2:
 * per token and head, h = T^T x (eq. transformed-cache) with h_c the exact value of
 * sum_j x_j T_jc rounded once to fp32 (nearest, ties to even); r_c = fl32(h_c * (1/s_c));
 * alpha = fp16(max over stored channels of |r_c|); code_c = clamp(floor(r_c * (1/alpha) *
 * 2^(b_c - 1) + 1/2), -2^(b_c-1), 2^(b_c-1) - 1) (the product rounded to fp32, the floor
 * exact) stored as its b_c-bit two's complement pattern, packed in `layout`.
 *
 * dev_params   device block from aatc_params_pack (this tensor, n_kv_heads heads).
 * x            device [n_tok] tokens, token t at x + t * x_tok_stride elements, each
 *              [n_kv_heads][d] contiguous, of type x_dtype (F32 or BF16).
 * codes        device cache of this sequence in `layout` (see top of file).
 * alpha        device [n_kv_heads][cap] fp16 token scales.
 * cap, pos     cache capacity in tokens and first token written; pos + n_tok <= cap.
 *              TILES needs cap % 64 == 0; tokens of a partly written tile that lie
 *              outside [pos, pos + n_tok) keep their bits.
 * n_tok == 0 is a no-op.  Errors: AATC_E_INVALID.
 * Speed: more than 16 tokens with 16-byte aligned token rows (x and x_tok_stride times
 * the element size) run on the matrix cores; other layouts take a slower kernel that
 * writes the same codes.
 */
aatc_status aatc_encode(const void* dev_params, int32_t n_kv_heads, int32_t d,
                        const void* x, aatc_dtype x_dtype, int64_t n_tok,
                        int64_t x_tok_stride, aatc_layout layout, void* codes,
                        uint16_t* alpha, int64_t cap, int64_t pos, void* stream);

/*
 * aatc_decode_attention -- one decode step of attention over packed caches.
 *
 * Algorithm 1 (inference: reconstruct, softmax, output) evaluated in the transformed
 * domain (App. B: effective query q~ = T_K^T q): for query head j of sequence b,
 * reading KV head j / (n_q_heads / n_kv_heads),
 *   o = T_V * sum_i softmax_i(scale * q~ . h^K_i) h^V_i,
 * with h^_c = alpha_i s_c 2^(1-b_c) code_ic and no mask inside
 * [0, seq_len[b]).  Online softmax over token splits; the inverse transform T_V is
 * applied once to each output.
 *
 * dev_params_k / _v  device parameter blocks of the key and value tensors.
 * q          device [batch][n_q_heads][d], q_dtype F32 or BF16.
 * k_codes    device RECORDS layout, [batch][n_kv_heads][cap][R_K].
 * k_alpha    device [batch][n_kv_heads][cap] fp16, 16-byte aligned (as v_alpha).
 * v_codes    device TILES layout, [batch][n_kv_heads][cap / 64][64 * R_V].
 * v_alpha    device [batch][n_kv_heads][cap] fp16.
 * seq_len    device [batch] int32, 0 <= seq_len[b] <= cap (0 gives a zero output;
 *            values outside [0, cap] are clamped).
 * cap        tokens per sequence in the caches, a multiple of 64.
 * k_record_bytes, v_record_bytes  R of the key and value tensors, as in their
 *            calibrations (the sizes the caches were allocated with).  If they differ
 *            from the parameter blocks, the outputs are NaN.
 * softmax_scale  logit scale, 1/sqrt(d) for standard attention.
 * out        device [batch][n_q_heads][d] fp32.
 * workspace  device scratch of at least aatc_decode_workspace_bytes(...) bytes,
 *            zero-filled once after allocation; every call leaves it reusable.
 * Errors: AATC_E_INVALID, AATC_E_WORKSPACE, AATC_E_DEVICE.
 */
size_t aatc_decode_workspace_bytes(int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                   int64_t cap);
aatc_status aatc_decode_attention(const void* dev_params_k, const void* dev_params_v,
                                  int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                  int32_t d, const void* q, aatc_dtype q_dtype,
                                  const void* k_codes, const uint16_t* k_alpha,
                                  const void* v_codes, const uint16_t* v_alpha,
                                  const int32_t* seq_len, int64_t cap,
                                  int32_t k_record_bytes, int32_t v_record_bytes,
                                  float softmax_scale, float* out, void* workspace,
                                  size_t ws_bytes, void* stream);

/*
 * aatc_append_decode_attention -- one decode step that also appends the step's new token.
 *
 * Equivalent to aatc_encode of x_k into (k_codes, k_alpha) and of x_v into (v_codes,
 * v_alpha) at position seq_len[b] - 1 of every sequence b (Alg. 1: the new key and value
 * are projected, quantized and appended), followed by aatc_decode_attention with the
 * same arguments; codes, scales and outputs are identical to that sequence of calls.
 * Sequences with seq_len[b] = 0 append nothing.  With G <= 8 and records of at most
 * 64 bytes it is one launch: every workgroup of a (sequence, KV head) computes a share
 * of the new token's exact transform coefficients into the workspace, and the
 * workgroup that merges the splits quantizes and stores the token and adds its term to
 * the attention.  Other shapes run the per-token encode before the decode launch.
 *
 * x_k, x_v   device [batch][n_kv_heads][d] new key / value token of each sequence,
 *            x_dtype F32 or BF16.
 * k_codes, k_alpha, v_codes, v_alpha  as in aatc_decode_attention; written at the new
 *            token's position.
 * Other arguments and errors as in aatc_decode_attention.
 */
aatc_status aatc_append_decode_attention(const void* dev_params_k, const void* dev_params_v,
                                         int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                         int32_t d, const void* q, aatc_dtype q_dtype,
                                         const void* x_k, const void* x_v, aatc_dtype x_dtype,
                                         void* k_codes, uint16_t* k_alpha, void* v_codes,
                                         uint16_t* v_alpha, const int32_t* seq_len, int64_t cap,
                                         int32_t k_record_bytes, int32_t v_record_bytes,
                                         float softmax_scale, float* out, void* workspace,
                                         size_t ws_bytes, void* stream);

/*
 * aatc_decode_attention_segmented -- decode attention over a compressed cache plus a
 * segment of tokens kept at input precision.
 *
 * The paper's inference path (Sec. 6, experimental setup; App. E, "AATC") keeps the first
 * s tokens and the most recent w tokens of each sequence at full precision and quantizes
 * the rest (aatc_segment_counts gives the split).  The result is exact softmax attention
 * of each query head over the union of the seq_len[b] tokens of the compressed caches (as
 * in aatc_decode_attention) and the seg_len[b] segment tokens, whose order does not matter:
 *   o = sum_i softmax_i(scale q . k_i) v_i,  k_i, v_i dequantized or as stored.
 * The segment is one more softmax partial: a small kernel computes it (in the original
 * domain, then T_V^T into the transformed domain of the merge) before the decode launch.
 *
 * seg_k, seg_v  device [batch][n_kv_heads][seg_cap][d] segment keys and values, seg_dtype
 *               F32 or BF16 (2- or 4-byte aligned).
 * seg_len       device [batch] int32 tokens in the segment (clamped to [0, seg_cap]).
 * seg_cap       1..256.
 * Other arguments, the workspace and errors as in aatc_decode_attention.
 */
aatc_status aatc_decode_attention_segmented(
    const void* dev_params_k, const void* dev_params_v, int32_t batch, int32_t n_q_heads,
    int32_t n_kv_heads, int32_t d, const void* q, aatc_dtype q_dtype, const void* k_codes,
    const uint16_t* k_alpha, const void* v_codes, const uint16_t* v_alpha,
    const int32_t* seq_len, int64_t cap, int32_t k_record_bytes, int32_t v_record_bytes,
    float softmax_scale, const void* seg_k, const void* seg_v, aatc_dtype seg_dtype,
    const int32_t* seg_len, int32_t seg_cap, float* out, void* workspace, size_t ws_bytes,
    void* stream);

/*
 * aatc_segment_counts -- the split of a sequence of n_tokens tokens under the paper's
 * full-precision policy (Sec. 6 experimental setup; App. E, "AATC": s = 4, w = 128,
 * step 16): the first `sink` tokens and a recent window stay at input precision; each
 * time the window holds `window` tokens, its oldest `step` tokens are quantized into the
 * compressed cache.  With m = max(n_tokens - sink, 0) tokens after the sink,
 * n_compressed = 0 if m < window, else step * (floor((m - window) / step) + 1): tokens
 * sink .. sink + n_compressed - 1 are compressed, the other n_segment tokens (the sink
 * and the window, which then holds window - step .. window - 1 tokens) are not.
 * Host only.  Errors: AATC_E_INVALID (NULL outputs, n_tokens < 0, sink < 0, window < 1,
 * step outside [1, window]).
 */
aatc_status aatc_segment_counts(int64_t n_tokens, int32_t sink, int32_t window, int32_t step,
                                int64_t* n_compressed, int32_t* n_segment);

/*
 * aatc_append_decode_attention_noalloc -- aatc_append_decode_attention without a caller
 * workspace, for callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).
 *
 * The same step and results as aatc_append_decode_attention with the same arguments; the
 * workspace is the library's own static device array (32 MiB, one per GPU the library
 * runs on, held until the process ends; no allocation at any call).  Its limit: at most
 * 256 (sequence, KV head) rows (batch * n_kv_heads), and aatc_decode_workspace_bytes of
 * the call plus a fixed 64 KiB counter region within 32 MiB (about batch * n_q_heads *
 * cap / 512 * 528 bytes of partials: e.g. batch 4, 32 query heads, 131072 tokens).  Larger
 * requests return AATC_E_WORKSPACE before anything is launched.  Calls that overlap on one
 * GPU share the array and race: order them on one stream.
 * Errors: as aatc_append_decode_attention; AATC_E_DEVICE if the array's address cannot be
 * obtained.
 */
aatc_status aatc_append_decode_attention_noalloc(
    const void* dev_params_k, const void* dev_params_v, int32_t batch, int32_t n_q_heads,
    int32_t n_kv_heads, int32_t d, const void* q, aatc_dtype q_dtype, const void* x_k,
    const void* x_v, aatc_dtype x_dtype, void* k_codes, uint16_t* k_alpha, void* v_codes,
    uint16_t* v_alpha, const int32_t* seq_len, int64_t cap, int32_t k_record_bytes,
    int32_t v_record_bytes, float softmax_scale, float* out, void* stream);

/*
 * Head-group transforms (Sec. 5.1, the remark on head groups: heads are merged into G
 * groups, each with its own transform block; Sec. 5.2: the token scale is taken per head
 * group; Sec. 6: G = 2 groups for Llama-3.1-8B's 8 KV heads, G = 1 for Qwen-2.5-7B's 4).
 *
 * A group is gkv consecutive KV heads (1 <= gkv <= 4): group g holds KV heads
 * g gkv .. g gkv + gkv - 1, and its token is the concatenation of their vectors,
 * d = 128 gkv elements with KV head kk of the group at elements [128 kk, 128 kk + 128).
 * Everything per KV head above becomes per group: one transform (d x d), one allocation of
 * round(avg_bits d) bits, per-channel scales, one token scale alpha per (token, group) and
 * one record per (token, group).  Both tensors use the RECORDS layout:
 *   codes [n_groups][cap][R] bytes (per sequence), alpha [n_groups][cap] fp16.
 * Query head j reads KV head k = j / (n_q_heads / n_kv_heads): block k % gkv of group
 * k / gkv, i.e. q~ = T[block]^T q has d transformed coordinates and o = T_V[block] o~.
 */
#define AATC_GROUP_MAX_DIM 512

/* Calibration artifact of one (head group, tensor): aatc_calibration with d up to 512;
 * transform is [j][c] with row stride d (the first d * d entries are used). */
typedef struct {
  int32_t d;                    /* 128 gkv */
  int32_t budget_bits;
  int32_t record_bytes;
  int32_t d_active;
  int32_t quantizer;
  float transform[AATC_GROUP_MAX_DIM * AATC_GROUP_MAX_DIM];
  uint8_t bits[AATC_GROUP_MAX_DIM];
  uint16_t scale_f16[AATC_GROUP_MAX_DIM];
  int32_t perm[AATC_GROUP_MAX_DIM];
  double sigma2[AATC_GROUP_MAX_DIM];
  double weight[AATC_GROUP_MAX_DIM];
  uint8_t bits_eig[AATC_GROUP_MAX_DIM];
} aatc_group_calibration;

/*
 * aatc_calibrate_group -- aatc_calibrate for one head group: x_calib is [n_calib][d] (the
 * group's concatenated tokens, d = 128 gkv), q_calib [n_q][d] the group's calibration
 * queries, each placed in its KV head's block and zero elsewhere (q_group = the group's
 * query heads: the weights average over tokens and sum over those heads), w_o [d][d_out]
 * the rows of W_O that read the group's values.  Same steps, arguments and errors as
 * aatc_calibrate; d must be 128, 256, 384 or 512.
 */
aatc_status aatc_calibrate_group(const float* x_calib, int64_t n_calib, int32_t d,
                                 const float* q_calib, int64_t n_q, int32_t q_group,
                                 const float* w_o, int32_t d_out, double avg_bits,
                                 int32_t b_max, double percentile, aatc_group_calibration* out);

/* Bytes of the device parameter block of n_groups groups (about 2 MiB per group), and
 * its host-side packing (every group must have the same d, record size and quantizer;
 * the caller copies host_buf to the device).  Errors: AATC_E_INVALID. */
size_t aatc_group_params_bytes(int32_t n_groups);
aatc_status aatc_group_params_pack(const aatc_group_calibration* per_group, int32_t n_groups,
                                   void* host_buf, size_t bytes);

/*
 * aatc_group_encode -- aatc_encode for head groups: tokens [n_tok] at x + t * x_tok_stride
 * elements, each [n_groups * d] contiguous (= [n_kv_heads][128]), F32 or BF16; group g's
 * codes go to codes + (g * cap + pos + t) * R, its scale to alpha[g * cap + pos + t].
 * h is the exact product with the stored transform rounded once to fp32, as in
 * aatc_encode.  gkv = d / 128.  Errors: AATC_E_INVALID.
 */
aatc_status aatc_group_encode(const void* dev_params, int32_t n_groups, int32_t gkv,
                              const void* x, aatc_dtype x_dtype, int64_t n_tok,
                              int64_t x_tok_stride, void* codes, uint16_t* alpha, int64_t cap,
                              int64_t pos, void* stream);

/*
 * aatc_group_decode_attention -- aatc_decode_attention over group-compressed caches:
 * k_codes / v_codes [batch][n_groups][cap][R] (RECORDS), k_alpha / v_alpha
 * [batch][n_groups][cap] fp16, q [batch][n_q_heads][128], out [batch][n_q_heads][128]
 * fp32.  Query heads per group (n_q_heads / n_groups) at most 32; records at most 512
 * bytes.  Four launches on `stream` (query weights, 256-token splits, the merge of the
 * splits, the inverse transform); workspace of aatc_group_decode_workspace_bytes bytes, every value
 * used written earlier in the same call (no zero fill needed).  Errors: AATC_E_INVALID, AATC_E_UNSUPPORTED,
 * AATC_E_WORKSPACE, AATC_E_DEVICE.
 */
size_t aatc_group_decode_workspace_bytes(int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                         int32_t gkv, int64_t cap);
aatc_status aatc_group_decode_attention(const void* dev_params_k, const void* dev_params_v,
                                        int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                        int32_t gkv, const void* q, aatc_dtype q_dtype,
                                        const void* k_codes, const uint16_t* k_alpha,
                                        const void* v_codes, const uint16_t* v_alpha,
                                        const int32_t* seq_len, int64_t cap,
                                        int32_t k_record_bytes, int32_t v_record_bytes,
                                        float softmax_scale, float* out, void* workspace,
                                        size_t ws_bytes, void* stream);

/* Human-readable name of a status code (static string). */
const char* aatc_status_string(aatc_status s);

#ifdef __cplusplus
}
#endif

#endif /* AATC_H_ */
