/*
 * offq.h -- C ABI of the MI355X (gfx950) OffQ W4A4KV4 online path.
 *
 * OffQ ("Taming Structured Outliers in LLM Quantization by Offsetting")
 * concentrates the structured activation outliers into the first channel of
 * each channel group (top-1 PCA rotation and grouping permutation, fused into
 * the weights offline), then applies an online Hadamard rotation whose first
 * row is all ones, so that this channel becomes a constant offset of the group
 * (sec. 3.2, Eq. 4 and Eq. 5), and absorbs that offset into the integer
 * zero-point of a per-group asymmetric 4-bit quantizer (sec. 3, Eq. 1).  All
 * matrix products then run on 4-bit integer codes.
 *
 * This library implements the online part only: the fused rotate + quantize
 * of activations, the int4 x int4 GEMM (and its decode-shape GEMV) with the
 * dequantising epilogue, the KV-cache quantizer, and an offline helper that
 * packs weights into the operand format the GEMM reads.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All data pointers are DEVICE pointers, allocated and freed by the caller;
 *   the library allocates nothing and keeps no per-call state.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *   Every call only enqueues work on `stream` and returns without
 *   synchronising; device faults surface at the caller's next sync.
 * - Arguments are validated on the host before anything is enqueued; a call
 *   that returns an error has enqueued nothing.  `offq_last_error()` gives a
 *   message for the last failing call of the calling thread.
 * - bf16 and fp16 tensors are passed as uint16_t bit patterns.
 * - Packed 4-bit codes: two per byte, channel 2j in the low nibble of byte j,
 *   channel 2j+1 in the high nibble.  Activation codes are unsigned 0..15;
 *   weight codes are 4-bit two's complement -8..7.
 * - Numerics: inputs are assumed finite.  NaN/Inf inputs give unspecified
 *   codes and outputs but never an out-of-bounds access.
 * - M == 0 (or rows == 0) is valid and enqueues nothing; the data pointers
 *   may then be NULL.
 *
 * The quantizer (sec. 3, Eq. 1, with 16-bit scale and 16-bit zero-point as in
 * sec. 3.4), for every group y[0..g) of fp32 values:
 *     mx = max y, mn = min y
 *     s  = fl32(fl32(mx - mn) / 15); if mx == mn: s = |mn| (1 if mn == 0)
 *     s16 = fp16_rne(clamp(s, 2^-24, 65504)),  sq = (float)s16,  r = fl32(1/sq)
 *     z  = clamp(rne(-mn * r), -32768, 32767)         (exact product)
 *     q  = clamp(rne(y * r) + z, 0, 15)               (exact product)
 * and x_hat = sq * (q - z) reconstructs y.
 */
#ifndef OFFQ_H
#define OFFQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  OFFQ_OK = 0,
  OFFQ_ERR_INVALID = 1,      /* bad pointer, size, stride or alignment        */
  OFFQ_ERR_UNSUPPORTED = 2,  /* valid but unsupported: g out of range, not gfx950 */
  OFFQ_ERR_HIP = 3           /* the HIP runtime reported an error at launch     */
} offq_status_t;

/* Version of this ABI; bumped on any incompatible change. */
#define OFFQ_ABI_VERSION 1
int offq_abi_version(void);

/* Static, human-readable name of a status code. */
const char* offq_status_string(offq_status_t status);

/* Message describing the last failing call made by the calling thread
 * (empty string if none).  Valid until the next call on that thread. */
const char* offq_last_error(void);

/*
 * offq_rotate_quantize -- fused online block-Hadamard rotation + per-group
 * 4-bit quantization of activations (sec. 3.2 Eq. 4 and group-wise offsetting;
 * sec. 3 Eq. 1; sec. 3.3 step 2(4) for the online group-wise H4).
 *
 *   For every row m and group b (channels [b*g, (b+1)*g)):
 *     y = x[m, group b] * H_g * c   if apply_hadamard   (H_g Sylvester, c = fl32(1/sqrt(g)))
 *     y = x[m, group b]             otherwise
 *   then the quantizer above on y.  The first channel of each group becomes
 *   the group's constant offset, which the zero-point absorbs.
 *
 *   x        bf16 [M, K], row stride ldx elements (ldx >= K, ldx % 8 == 0),
 *            16-byte aligned.
 *   M, K     rows (tokens) and channels; K % g == 0.
 *   g        group = Hadamard block size, power of two, 16 <= g <= 8192
 *            (g == K: one group per token).
 *   apply_hadamard  1 = rotate then quantize, 0 = quantize only (inputs whose
 *            rotation is already fused into the producing weights).
 *   codes    uint8 [M, K/2] packed unsigned codes, contiguous, 4-byte aligned.
 *   scale    fp16  [M, K/g] scales sq, contiguous.
 *   zero     int16 [M, K/g] zero-points z, contiguous.
 *   y_debug  nullable fp32 [M, K] contiguous, 16-byte aligned: if non-NULL,
 *            receives exactly the fp32 values that were quantized.
 */
offq_status_t offq_rotate_quantize(const uint16_t* x, int64_t M, int64_t K, int64_t ldx,
                         int32_t g, int32_t apply_hadamard,
                         uint8_t* codes, uint16_t* scale, int16_t* zero,
                         float* y_debug, void* stream);

/*
 * offq_w4a4_gemm -- int4 x int4 GEMM with int32 accumulation and the
 * dequantising epilogue that follows from Eq. 1 (x_hat = s (q_a - z),
 * w_hat = sw q_w):
 *
 *   acc_b[m, n] = sum_{k in group b} q_a[m, k] * q_w[n, k]           (int32)
 *   Y[m, n]     = sw[n] * sum_b s[m, b] * (acc_b[m, n] - z[m, b] * colsum[b, n])
 *
 *   The z * colsum term is the zero-point (offset) correction through
 *   per-column weight sums.  Y is rounded to bf16 (nearest even).  Shapes with
 *   M <= 16 (decode) take a weight-streaming GEMV path; larger M the MFMA
 *   GEMM path.  Results are identical up to fp32 summation order.
 *
 *   a_codes  uint8 [M, K/2] (from offq_rotate_quantize), 16-byte aligned.
 *   a_scale  fp16  [M, K/g];  a_zero int16 [M, K/g].
 *   w_codes  two's-complement int4 codes in the blocked layout written by
 *            offq_pack_weights (offq_weight_codes_bytes(N, K) bytes),
 *            16-byte aligned.
 *   w_scale  fp16  [N] per-output-channel symmetric scale sw.
 *   w_colsum int32 [K/g, N]: colsum[b, n] = sum_{k in group b} q_w[n, k].
 *   M, N, K  K % g == 0; g power of two, 64 <= g <= 8192.
 *   y        bf16 [M, N], row stride ldy >= N elements.
 *   acc_debug nullable int32 [K/g, M, N] contiguous: if non-NULL, receives
 *            every per-group integer accumulator acc_b.
 */
offq_status_t offq_w4a4_gemm(const uint8_t* a_codes, const uint16_t* a_scale,
                   const int16_t* a_zero, const uint8_t* w_codes,
                   const uint16_t* w_scale, const int32_t* w_colsum,
                   int64_t M, int64_t N, int64_t K, int32_t g,
                   uint16_t* y, int64_t ldy, int32_t* acc_debug, void* stream);

/*
 * offq_kv_quantize -- 4-bit KV-cache quantization: one row = one (batch,
 * head, position); group = head_dim (sec. 4.2, "Number of Groups").  With
 * apply_hadamard = 1 the row first receives the per-head online Hadamard H3
 * (sec. 3.3 step 2(3), keys after RoPE); values, whose rotation R2 is fused
 * offline (sec. 3.3 step 2(2)), use apply_hadamard = 0.
 *
 *   kv        bf16 [rows, head_dim], row stride row_stride elements
 *             (>= head_dim, % 8 == 0), 16-byte aligned.
 *   head_dim  power of two, 16 <= head_dim <= 8192 (128 for Llama-class).
 *   codes     uint8 [rows, head_dim/2]; scale fp16 [rows]; zero int16 [rows].
 *   y_debug   nullable fp32 [rows, head_dim].
 */
offq_status_t offq_kv_quantize(const uint16_t* kv, int64_t rows, int32_t head_dim,
                     int64_t row_stride, int32_t apply_hadamard,
                     uint8_t* codes, uint16_t* scale, int16_t* zero,
                     float* y_debug, void* stream);

/*
 * offq_pack_weights -- offline helper: per-output-channel symmetric 4-bit
 * weight quantization (sec. 4, implementation: per-channel symmetric weights)
 * into the operand format of offq_w4a4_gemm.
 *
 *   sw[n]  = fp16_rne(clamp(max_k |w[n,k]| / 7, 2^-24, 65504))  (1 for a zero row)
 *   q[n,k] = clamp(rne(w[n,k] / sw[n]), -8, 7)                   (exact quotient)
 *   colsum[b, n] = sum_{k in group b} q[n, k]
 *
 *   w        fp32 [N, K] contiguous, 16-byte aligned.
 *   g        group size the activations will use (power of two, 64..8192, K % g == 0).
 *   w_codes  offq_weight_codes_bytes(N, K) bytes, 16-byte aligned, in the
 *            blocked layout below; w_scale fp16 [N]; w_colsum int32 [K/g, N].
 *
 *   Blocked layout of w_codes: the codes of 16 output rows x 128 k form a
 *   1 KB block, 16 rows of 64 bytes (byte j of a block row holds k = 2j in
 *   its low nibble and k = 2j + 1 in its high nibble); the blocks of a band of
 *   16 rows follow in k order, the bands in row order.  Byte kk of row n sits
 *   at ((n / 16) * KB + kk / 64) * 1024 + (n % 16) * 64 + kk % 64 with
 *   KB = ceil(K / 128).  Rows past N up to a multiple of 16 and k past K up
 *   to a multiple of 128 hold zero codes.  (One wave's 16-byte-per-lane load
 *   of a block then reads 1 KB of contiguous memory in the decode GEMV.)
 */
offq_status_t offq_pack_weights(const float* w, int64_t N, int64_t K, int32_t g,
                      uint8_t* w_codes, uint16_t* w_scale, int32_t* w_colsum,
                      void* stream);

/*
 * offq_weight_codes_bytes -- size of w_codes for an [N, K] weight:
 * ceil(N / 16) * ceil(K / 128) * 1024 bytes; 0 for N or K outside
 * [1, 2^30].
 */
int64_t offq_weight_codes_bytes(int64_t N, int64_t K);

/*
 * offq_kv_attention_decode -- one decode step of attention over the 4-bit KV
 * cache written by offq_kv_quantize (sec. 3.3 step 2(2)/(3), sec. 4.2): keys
 * rotated by the per-head Hadamard H3 before quantization (apply_hadamard = 1),
 * values either rotated offline by R2 (apply_hadamard = 0; the output then
 * stays in that basis, which the output projection undoes) or by H3
 * (v_hadamard = 1: the output is rotated back).  For every (b, h), with
 * c = fl32(1/sqrt(128)) and H the 128-point Sylvester Hadamard matrix:
 *
 *     q_r[d] = bf16_rne(c * sum_i q[i] H[i][d])      (fp32 sum)
 *     s_j    = sm_scale * sk_j * sum_d q_r[d] (ck_j[d] - zk_j)     0 <= j < seq_len
 *     p      = softmax(s)
 *     o[d]   = sum_j p_j * sv_j * (cv_j[d] - zv_j);  if v_hadamard: o = c H o
 *     out    = bf16_rne(o)
 *
 *   q            bf16 [B, H, 128] contiguous (the query after RoPE).
 *   k_codes      uint8 [B, H, s_cap, 64], 16-byte aligned; k_scale fp16 and
 *                k_zero int16 [B, H, s_cap] (rows (b, h, j) of offq_kv_quantize
 *                with head_dim = 128).  v_codes (16-byte aligned), v_scale,
 *                v_zero likewise.
 *   seq_len      positions in use, 1 <= seq_len <= s_cap.
 *   sm_scale     score scale (1/sqrt(128) for standard attention).
 *   out          bf16 [B, H, 128].
 *   workspace    caller-owned device buffer of at least
 *                offq_kv_attention_workspace_bytes(B, H, seq_len) bytes,
 *                4-byte aligned; its contents are scratch.  Calls that share
 *                a workspace must be ordered on one stream.
 * head_dim is 128; other sizes return OFFQ_ERR_UNSUPPORTED.
 */
offq_status_t offq_kv_attention_decode(const uint16_t* q, const uint8_t* k_codes, const uint16_t* k_scale,
                             const int16_t* k_zero, const uint8_t* v_codes,
                             const uint16_t* v_scale, const int16_t* v_zero, int64_t B,
                             int64_t H, int64_t s_cap, int64_t seq_len, int32_t head_dim,
                             float sm_scale, int32_t v_hadamard, uint16_t* out, void* workspace,
                             int64_t workspace_bytes, void* stream);

/* Bytes of workspace offq_kv_attention_decode needs (0 for invalid sizes):
 * 130 floats per query head and chunk of up to 512 positions; H is the number
 * of query heads. */
int64_t offq_kv_attention_workspace_bytes(int64_t B, int64_t H, int64_t seq_len);

/*
 * offq_kv_attention_decode_gqa -- the same step with grouped-query attention
 * (the key/value heads of Llama 3 style models): Hq query heads share Hkv
 * key/value heads, query head h of batch b reading the cache rows of
 * key/value head h / (Hq / Hkv).  q and out are [B, Hq, 128]; the cache
 * arrays are [B, Hkv, s_cap, ...]; the workspace is sized by
 * offq_kv_attention_workspace_bytes(B, Hq, seq_len).  Hq must be a multiple
 * of Hkv (OFFQ_ERR_INVALID otherwise).  offq_kv_attention_decode is this call
 * with Hkv = Hq.
 */
offq_status_t offq_kv_attention_decode_gqa(const uint16_t* q, const uint8_t* k_codes,
                                 const uint16_t* k_scale, const int16_t* k_zero,
                                 const uint8_t* v_codes, const uint16_t* v_scale,
                                 const int16_t* v_zero, int64_t B, int64_t Hq, int64_t Hkv,
                                 int64_t s_cap, int64_t seq_len, int32_t head_dim, float sm_scale,
                                 int32_t v_hadamard, uint16_t* out, void* workspace,
                                 int64_t workspace_bytes, void* stream);

/*
 * offq_kv_attention_decode_quantize -- offq_kv_attention_decode_gqa whose
 * output rows also come out quantized for the next linear layer (the
 * O-projection, whose input is quantized without an online rotation, its
 * rotation being fused into the weights offline: sec. 3.3 step 2(1)).  Each
 * head's 128 outputs, rounded to bf16, form one group of the quantizer of
 * Eq. 1: out_codes [B, Hq * 64] bytes (two codes per byte, element 2k in the
 * low nibble), out_scale [B, Hq] fp16 bits, out_zero [B, Hq] int16 -- exactly
 * what offq_rotate_quantize(out, g = 128, hadamard = 0) writes for the bf16
 * output [B, Hq * 128].  out (bf16 [B, Hq, 128]) may be NULL; out_codes,
 * out_scale and out_zero may not.  Other arguments, the workspace and the
 * errors as for offq_kv_attention_decode_gqa.
 */
offq_status_t offq_kv_attention_decode_quantize(const uint16_t* q, const uint8_t* k_codes,
                                      const uint16_t* k_scale, const int16_t* k_zero,
                                      const uint8_t* v_codes, const uint16_t* v_scale,
                                      const int16_t* v_zero, int64_t B, int64_t Hq, int64_t Hkv,
                                      int64_t s_cap, int64_t seq_len, int32_t head_dim,
                                      float sm_scale, int32_t v_hadamard, uint16_t* out,
                                      uint8_t* out_codes, uint16_t* out_scale, int16_t* out_zero,
                                      void* workspace, int64_t workspace_bytes, void* stream);

/*
 * offq_kv_attention_decode_noalloc -- offq_kv_attention_decode_gqa for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops that must not call hipMalloc): the same kernels and results,
 * with the per-chunk records kept in a static device array of the library
 * instead of a caller-owned workspace.  The call itself allocates nothing;
 * the caller passes every input and the output.
 *
 *   Arguments as for offq_kv_attention_decode_gqa, without workspace.
 *   Limit: the records need offq_kv_attention_workspace_bytes(B, Hq, seq_len)
 *   bytes, at most 16 MiB (B * Hq * ceil(seq_len / 512) <= 32263, e.g.
 *   B = 8, Hq = 32, seq_len = 32768 uses half); larger sizes return
 *   OFFQ_ERR_UNSUPPORTED before anything is enqueued.
 *   Each device holds its own 16 MiB array from the first call until the
 *   process ends.  All calls on one device share that array: calls that can
 *   overlap on one device (different streams, or host threads without
 *   ordering) race and must be serialised by the caller.
 */
offq_status_t offq_kv_attention_decode_noalloc(const uint16_t* q, const uint8_t* k_codes,
                                               const uint16_t* k_scale, const int16_t* k_zero,
                                               const uint8_t* v_codes, const uint16_t* v_scale,
                                               const int16_t* v_zero, int64_t B, int64_t Hq,
                                               int64_t Hkv, int64_t s_cap, int64_t seq_len,
                                               int32_t head_dim, float sm_scale,
                                               int32_t v_hadamard, uint16_t* out, void* stream);

/* ---------------------------------------------------------------------------
 * Decoder-layer steps around the quantized linear layers (one decode step,
 * one new token per sequence), following the pipeline of sec. 3.3 / Fig. 2.
 * All tensors are bf16 unless stated; rows are contiguous in their last
 * dimension with the given row strides (in elements).
 * ------------------------------------------------------------------------- */

/*
 * offq_add_rmsnorm -- the residual stream and its RMSNorm (the norm's scale is
 * fused into the next weights offline, so none is applied here):
 *     h = bf16(fl32(x + res))          (h = x when res is NULL)
 *     y = bf16(h * fl32(1 / sqrt(mean_k h^2 + eps)))
 *   x [M, D] (ldx), res [M, D] (ldr) or NULL, h_out [M, D] (ldh) or NULL,
 *   y_out [M, D] (ldy) or NULL (at least one output).  D a multiple of 8,
 *   strides multiples of 8, pointers 16-byte aligned.  M = 0 is a no-op.
 */
offq_status_t offq_add_rmsnorm(const uint16_t* x, int64_t ldx, const uint16_t* res, int64_t ldr, int64_t M,
                     int64_t D, float eps, uint16_t* h_out, int64_t ldh, uint16_t* y_out,
                     int64_t ldy, void* stream);

/*
 * offq_swiglu -- out[m, f] = bf16(fl32(silu(g) * u)), silu(g) = g / (1 + e^-g)
 * in fp32, with g = gu[m, f] and u = gu[m, F + f]: the up/gate projection
 * writes gate in columns [0, F) and up in [F, 2F) (the grouping permutation
 * P4 of sec. 3.3 step 2(4) is fused into those weights offline).
 *   gu [M, 2F] (ldg >= 2F), out [M, F] (ldo >= F); F, ldg, ldo multiples of
 *   8; pointers 16-byte aligned.
 */
offq_status_t offq_swiglu(const uint16_t* gu, int64_t ldg, int64_t M, int64_t F, uint16_t* out, int64_t ldo,
                void* stream);

/*
 * offq_add_rmsnorm_quantize -- offq_add_rmsnorm followed by the quantizer of
 * offq_rotate_quantize with apply_hadamard = 0 on y (the QKV and up/gate
 * inputs, whose rotations are fused into the weights offline), in one pass:
 * h_out (nullable) as offq_add_rmsnorm; codes uint8 [M, D/2], scale fp16 and
 * zero int16 [M, D/g] as offq_rotate_quantize; y_debug bf16 [M, D] (row
 * stride ldy) or NULL: the normalized rows that were quantized.
 * D / 256 in {8, 16, 32, 64} (D = 2048 ... 16384); g a power of two with
 * D/256 <= g <= D/4 dividing D.
 */
offq_status_t offq_add_rmsnorm_quantize(const uint16_t* x, int64_t ldx, const uint16_t* res, int64_t ldr,
                              int64_t M, int64_t D, float eps, int32_t g, uint16_t* h_out,
                              int64_t ldh, uint8_t* codes, uint16_t* scale, int16_t* zero,
                              uint16_t* y_debug, int64_t ldy, void* stream);

/*
 * offq_swiglu_rotate_quantize -- offq_swiglu followed by the online
 * 128-point Hadamard H4 and the quantizer (offq_rotate_quantize with g = 128,
 * apply_hadamard = 1) on the bf16 SwiGLU output, in one pass (the
 * down-projection input, sec. 3.3 step 2(4)): codes uint8 [M, F/2], scale fp16
 * and zero int16 [M, F/128]; y_debug fp32 [M, F] or NULL: the rotated rows
 * that were quantized.  F a multiple of 128; ldg >= 2F, a multiple of 8.
 */
offq_status_t offq_swiglu_rotate_quantize(const uint16_t* gu, int64_t ldg, int64_t M, int64_t F,
                                uint8_t* codes, uint16_t* scale, int16_t* zero, float* y_debug,
                                void* stream);

/*
 * offq_rope_kv_append -- RoPE on the new token's query and key heads, the
 * per-head online Hadamard H3 on the key (sec. 3.3 step 2(3)) and the KV4
 * quantizer (as offq_kv_quantize, group = head dim) writing position
 * positions[m] of sequence m into the cache:
 *   qkv [M, (Hq + 2 Hkv) * 128] (ldq >= that, a multiple of 8; qkv 16-byte
 *     aligned): query heads, then key heads, then value heads of the QKV
 *     projection of token m;
 *   positions int32 [M] (device): the position of token m in its sequence;
 *     a position outside [0, s_cap) writes nothing to the cache;
 *   rope_base: RoPE's base (theta); dims (i, i + 64) rotate by angle
 *     fl32(pos * fl32(base^(-2i/128))), computed in fp32;
 *   k_hadamard / v_hadamard (0 or 1): c H on the key (after RoPE and a bf16
 *     rounding) / on the value before quantization (paper: 1 / 0);
 *   q_out [M, Hq, 128] (16-byte aligned): the query after RoPE;
 *   k_codes, v_codes uint8 [M, Hkv, s_cap, 64]; k_scale, v_scale fp16 and
 *     k_zero, v_zero int16 [M, Hkv, s_cap] (the layout the decode attention
 *     reads);
 *   k_y_debug, v_y_debug fp32 [M, Hkv, 128] (16-byte aligned) or NULL: the
 *     rows that were quantized.
 * head_dim must be 128.
 */
offq_status_t offq_rope_kv_append(const uint16_t* qkv, int64_t ldq, int64_t M, int64_t Hq, int64_t Hkv,
                        int32_t head_dim, const int32_t* positions, double rope_base,
                        int32_t k_hadamard, int32_t v_hadamard, uint16_t* q_out,
                        uint8_t* k_codes, uint16_t* k_scale, int16_t* k_zero, uint8_t* v_codes,
                        uint16_t* v_scale, int16_t* v_zero, int64_t s_cap, float* k_y_debug,
                        float* v_y_debug, void* stream);

/*
 * offq_rope_kv_prefill -- offq_rope_kv_append for the prefill of T tokens per
 * sequence (sec. 3.3 step 2(3), Fig. 2): row b T + t of qkv is token t of
 * sequence b, written at position positions[b T + t] of that sequence's
 * cache, which is [B, Hkv, s_cap, 64] (codes) and [B, Hkv, s_cap] (scales,
 * zero-points).  q_out [B T, Hq, 128]; debug rows [B T, Hkv, 128] or NULL.
 * T >= 1; the other arguments, the arithmetic and the errors are those of
 * offq_rope_kv_append, which is this call with T = 1.
 */
offq_status_t offq_rope_kv_prefill(const uint16_t* qkv, int64_t ldq, int64_t B, int64_t T,
                        int64_t Hq, int64_t Hkv, int32_t head_dim, const int32_t* positions,
                        double rope_base, int32_t k_hadamard, int32_t v_hadamard,
                        uint16_t* q_out, uint8_t* k_codes, uint16_t* k_scale, int16_t* k_zero,
                        uint8_t* v_codes, uint16_t* v_scale, int16_t* v_zero, int64_t s_cap,
                        float* k_y_debug, float* v_y_debug, void* stream);

/*
 * offq_kv_attention_prefill -- causal attention of T new tokens per sequence
 * over the 4-bit KV cache (sec. 3.3 step 2(3); the per-row arithmetic of
 * offq_kv_attention_decode_gqa): query t of sequence b sits at position
 * past + t and attends to cache positions 0 .. past + t.
 *   q        bf16 [B, T, Hq, 128] (device): the queries after RoPE (the
 *            q_out of offq_rope_kv_prefill), rotated by c H inside;
 *   k_codes, v_codes uint8 [B, Hkv, s_cap, 64]; k_scale, v_scale fp16 and
 *            k_zero, v_zero int16 [B, Hkv, s_cap]: the cache, holding the
 *            past + T positions read (later positions are never read);
 *   Hq a multiple of Hkv with Hq / Hkv in {1, 2, 4, 8}; past >= 0,
 *            past + T <= s_cap;
 *   sm_scale score scale; v_hadamard 0 or 1 as for the decode call;
 *   out      bf16 [B, T, Hq, 128] (row b T + t, the input of the output
 *            projection); it may not overlap q.
 * B = 0 or T = 0 does nothing (the pointers may then be NULL).
 * No workspace.  Errors: OFFQ_ERR_INVALID for bad sizes, pointers or
 * alignment (16 bytes for q and out), OFFQ_ERR_UNSUPPORTED for head_dim !=
 * 128 or another group size.
 */
offq_status_t offq_kv_attention_prefill(const uint16_t* q, int64_t B, int64_t T, int64_t Hq,
                        int64_t Hkv, int32_t head_dim, int64_t past, const uint8_t* k_codes,
                        const uint16_t* k_scale, const int16_t* k_zero, const uint8_t* v_codes,
                        const uint16_t* v_scale, const int16_t* v_zero, int64_t s_cap,
                        float sm_scale, int32_t v_hadamard, uint16_t* out, void* stream);

/* ---------------------------------------------------------------------------
 * Offline calibration (sec. 3.1 top-1 PCA, sec. 3.2 group-wise offsetting,
 * sec. 3.3 steps 1-2): from calibration activations to the fused, permuted
 * and rotated fp32 weights that offq_pack_weights then quantizes.  These run
 * once per model, not in the online path; offq_eigh blocks the calling thread
 * (it reads the convergence measure back after every sweep).
 * ------------------------------------------------------------------------- */

/* Bytes of workspace offq_top1_select needs: one float per token. */
int64_t offq_top1_workspace_bytes(int64_t n_seq, int64_t seq_len);

/*
 * offq_top1_select -- per calibration sequence, the token whose row has the
 * largest L-infinity norm (the first such token on ties), copied as fp32:
 *   x bf16: token t of sequence s at x + s*ld_seq + t*ld_tok, D channels
 *     (D, ld_tok, ld_seq multiples of 8; x 16-byte aligned);
 *   idx int32 [n_seq] (the selected token), X fp32 [n_seq, D] (row stride ldX).
 * Inputs must be finite.
 */
offq_status_t offq_top1_select(const uint16_t* x, int64_t n_seq, int64_t seq_len, int64_t D, int64_t ld_tok,
                     int64_t ld_seq, int32_t* idx, float* X, int64_t ldX, void* workspace,
                     int64_t workspace_bytes, void* stream);

/* offq_channel_absmax -- out fp64 [D] = max over rows of |x[r, c]| (bf16 x
 * [rows, D], row stride ldx): the statistic that picks the outlier channels of
 * the down-projection input (sec. 3.3 step 2(4)). */
offq_status_t offq_channel_absmax(const uint16_t* x, int64_t rows, int64_t D, int64_t ldx, double* out,
                        void* stream);

/* offq_gram -- C fp64 [D, D] (row stride ldC) = X^T X / N for X fp32 [N, D]
 * (row stride ldX), accumulated in fp64 (Eq. 2; zero-mean assumed, as there).
 * C is exactly symmetric. */
offq_status_t offq_gram(const float* X, int64_t N, int64_t D, int64_t ldX, double* C, int64_t ldC,
              void* stream);

/* Bytes of workspace offq_eigh needs (about 32 D^2). */
int64_t offq_eigh_workspace_bytes(int64_t D);

/*
 * offq_eigh -- C = U diag(evals) U^T for symmetric C fp64 [D, D] (row stride
 * ldC; read only), D even, 2 <= D <= 8192: evals fp64 [D] descending, U fp64
 * [D, D] (row stride ldU) with eigenvector k in column k, its entry of largest
 * magnitude positive.  Parallel cyclic Jacobi in fp64 until the off-diagonal
 * Frobenius norm is at most tol times the whole norm, or max_sweeps sweeps;
 * *sweeps and *rel_off (nullable) report what was reached.  workspace: at least
 * offq_eigh_workspace_bytes(D), 16-byte aligned.
 */
offq_status_t offq_eigh(const double* C, int64_t D, int64_t ldC, double* evals, double* U, int64_t ldU,
              void* workspace, int64_t workspace_bytes, int32_t max_sweeps, double tol,
              int32_t* sweeps, double* rel_off, void* stream);

/*
 * offq_group_permutation -- the sorted grouping of sec. 3.2 / sec. 4.3 for D
 * channels in groups of g (D a multiple of g): with G = D / g, the G channels
 * of largest key lead the groups in descending order (perm[b g] = the b-th
 * largest), the others fill slots 1..g-1 of the groups in ascending key order
 * (ties by channel index).  perm int32 [D]: new slot -> original channel.
 * workspace: D int32.
 */
offq_status_t offq_group_permutation(const double* key, int64_t D, int32_t g, int32_t* perm,
                           void* workspace, int64_t workspace_bytes, void* stream);

/*
 * offq_build_rotation -- R fp32 [D, D] (row stride ldR) = U P B, with U fp64
 * [D, D] (NULL: identity), P the permutation matrix of perm (NULL: identity;
 * column s of U P is column perm[s] of U) and B = blockdiag(H_g / sqrt(g)) on
 * consecutive groups of g columns when apply_hadamard (else identity); the
 * product is formed in fp64.  D <= 8192, D a multiple of g (power of two).
 */
offq_status_t offq_build_rotation(const double* U, int64_t ldU, int64_t D, const int32_t* perm, int32_t g,
                        int32_t apply_hadamard, float* R, int64_t ldR, void* stream);

/* offq_fuse_weights -- W_out fp32 [N, K] = W R for W fp32 [N, K] and R fp32
 * [K, K] (the rotation a linear layer's input receives, fused into its
 * weights: y = x W^T = (x R)(W R)^T). */
offq_status_t offq_fuse_weights(const float* W, int64_t ldW, int64_t N, int64_t K, const float* R,
                      int64_t ldR, float* W_out, int64_t ldo, void* stream);

/* offq_permute_rows -- W_out[s, :] = W[perm[s], :] (fp32 [N, K]): an output-
 * channel permutation fused into the producing weights (P4 into up/gate). */
offq_status_t offq_permute_rows(const float* W, int64_t ldW, int64_t N, int64_t K, const int32_t* perm,
                      float* W_out, int64_t ldo, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* OFFQ_H */
