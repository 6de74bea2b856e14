// Shared device/host helpers of the OffQ HIP library (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace offq {

// Weight operand layout (written by offq_pack_weights, read by the GEMM and
// GEMV kernels): the packed codes of 16 output rows x 128 k form a 1 KB block
// (16 rows of 64 bytes); the blocks of a band of 16 rows follow in k order and
// the bands in row order.  Rows past N up to a multiple of 16, and k past K up
// to a multiple of 128, hold zero codes.  A wave that loads 16 bytes per lane
// of one block reads 1 KB of contiguous memory.
__host__ __device__ constexpr int64_t wblk_kblocks(int64_t K) { return (K + 127) >> 7; }
__host__ __device__ constexpr int64_t wblk_bytes(int64_t N, int64_t K) {
  return ((N + 15) >> 4) * wblk_kblocks(K) * 1024;
}
// byte offset of code byte kk (codes 2 kk, 2 kk + 1) of row n; KB = wblk_kblocks(K)
__host__ __device__ inline int64_t wblk_off(int64_t n, int64_t kk, int64_t KB) {
  return ((((n >> 4) * KB + (kk >> 6)) << 10) | ((n & 15) << 6) | (kk & 63));
}

// bf16 bit pattern -> fp32 (exact).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bit pattern, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// two fp32 -> packed bf16 (lo = a, hi = b), round to nearest even
// (v_cvt_pk_bf16_f32 on gfx950).
typedef __bf16 offq_bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2_rne(float a, float b) {
  const offq_bf16x2 r = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ float fp16_bits_to_f32(uint16_t h) {
  _Float16 v = __builtin_bit_cast(_Float16, h);
  return (float)v;
}

// Per-group quantizer parameters of Eq. 1 (sec. 3) with a 16-bit scale and a
// 16-bit integer zero-point (sec. 3.4), from the group's max and min:
//   s = fl32(fl32(mx - mn) / 15)  (degenerate mx == mn: s = |mn|, or 1)
//   s16 = fp16_rne(clamp(s, 2^-24, 65504)), r = fl32(1 / f32(s16))
//   z = clamp(rne(-mn * r), -32768, 32767), the product taken exactly.
// Codes are then q = clamp(rne(y * r) + z, 0, 15) with the exact product,
// evaluated as described at quant_code().
struct QParams {
  float r;          // 1 / sq
  float lo;         // MAGIC - z       (exact integer in [2^23, 2^24))
  float hi;         // MAGIC - z + 15
  uint16_t s16;     // stored scale (fp16 bits)
  int16_t z;        // stored zero-point
};

// 1.5 * 2^23: fma(y, r, MAGIC) = MAGIC + rne(y * r) exactly when |y r| < 2^22,
// because every float in [2^23, 2^24) is an integer and MAGIC is even.
#define OFFQ_MAGIC 12582912.0f

// fl32(d / 15) without a division: q0 = fl(d * fl(1/15)), then one
// correction with the exact remainder fma(-q0, 15, d) (Markstein's method for
// a known divisor).  Equal to the IEEE quotient for every d with d / 15 in
// [2^-25, 2^17] (checked exhaustively on the GPU by
// tests/gpu_checks/fast_division.hip); outside that range both lie on the same
// side of the clamp to [2^-24, 65504] in quant_params (for finite d), so the
// clamped scale is the same.
__device__ __forceinline__ float div15_rn(float d) {
  const float R = 1.0f / 15.0f;
  const float q0 = d * R;
  const float rem = __builtin_fmaf(-q0, 15.0f, d);
  return __builtin_fmaf(rem, R, q0);
}

// fl32(1 / s) for s an fp16 value: the hardware reciprocal refined by one
// Newton step with fma.  Equal to the IEEE quotient for every positive finite
// fp16 value (checked exhaustively by the same GPU test).
__device__ __forceinline__ float rcp_fp16_rn(float s) {
  const float r0 = __builtin_amdgcn_rcpf(s);
  const float e = __builtin_fmaf(-s, r0, 1.0f);
  return __builtin_fmaf(e, r0, r0);
}

// z = clamp(rne(-mn * r), -32768, 32767) of the exact product, in fp32:
// pr = fl(-mn r) and its error er = fma(-mn, r, -pr) (exact; pr + er = -mn r).
// Below 2^23 every half-integer is a float, so rounding the product cannot
// cross one and rint(pr) is the answer, except when pr is itself a
// half-integer: then the sign of er decides (er = 0: the tie, to even).  Past
// the int16 range the clamp decides.  (Equal to the fp64 rounding: checked
// on the GPU for every fp16 scale against products near every 16th
// half-integer of the range and random operands.)
__device__ __forceinline__ int zero_point_rn(float mn, float r) {
#pragma clang fp contract(off)
  const float pr = -mn * r;
  const float er = __builtin_fmaf(-mn, r, -pr);
  float zf = __builtin_rintf(pr);
  if (fabsf(pr - zf) == 0.5f && er != 0.0f) zf = er > 0.0f ? __builtin_ceilf(pr) : __builtin_floorf(pr);
  zf = fminf(fmaxf(zf, -32768.0f), 32767.0f);
  return (int)zf;
}

__device__ __forceinline__ QParams quant_params(float mx, float mn) {
#pragma clang fp contract(off)
  float s;
  if (mx > mn) {
    // (an overflowed range is taken as the largest float: the scale clamps
    // to 65504 either way)
    s = div15_rn(fminf(mx - mn, 0x1.fffffep127f));
  } else {
    s = (mn != 0.0f) ? fabsf(mn) : 1.0f;
  }
  s = fminf(fmaxf(s, 0x1p-24f), 65504.0f);
  _Float16 h = (_Float16)s;            // round to nearest even
  float sq = (float)h;
  float r = rcp_fp16_rn(sq);           // = the IEEE fp32 quotient 1 / sq
  const int z = zero_point_rn(mn, r);
  QParams p;
  p.r = r;
  p.lo = OFFQ_MAGIC - (float)z;
  p.hi = p.lo + 15.0f;
  p.s16 = __builtin_bit_cast(uint16_t, h);
  p.z = (int16_t)z;
  return p;
}

// Returns bits(clamp(MAGIC + rne(y r), lo, hi)); subtracting bits(lo) gives the
// code clamp(rne(y r) + z, 0, 15).  Correct for every finite y: when
// |y r| >= 2^22 the fma result lies outside [lo, hi] on the correct side, and
// the clamp to [lo, hi] then yields code 0 or 15 exactly as the definition.
__device__ __forceinline__ uint32_t quant_bits(float y, const QParams& p) {
  float u = __builtin_fmaf(y, p.r, OFFQ_MAGIC);
  u = __builtin_amdgcn_fmed3f(u, p.lo, p.hi);
  return __float_as_uint(u);
}

}  // namespace offq
