// Offline weight packing: per-output-channel symmetric 4-bit quantization
// (sec. 4, implementation: weights per-channel symmetric) into the operand
// format of the W4A4 GEMM, plus the per-group column sums the epilogue uses
// for the zero-point correction.  The codes go to the blocked operand layout
// (1 KB blocks of 16 rows x 128 k; padding rows and k written as zero codes).
//
//   sw[n]   = fp16_rne(clamp(max_k |w[n,k]| / 7, 2^-24, 65504))   (1 for a zero row)
//   q[n,k]  = clamp(rne(w[n,k] / sw[n]), -8, 7)       (quotient evaluated in fp64;
//             for these operand widths its rounding never crosses a half-integer)
//   colsum[b,n] = sum_{k in group b} q[n,k]
#include "common.h"
#include "internal.h"

namespace offq {
namespace {

constexpr int PW_THREADS = 256;
constexpr int PW_MAX_GROUPS = 512;  // K / g <= 512 (g >= 64, K <= 32768)

__global__ __launch_bounds__(PW_THREADS) void pack_weights_kernel(
    const float* __restrict__ w, int64_t N, int64_t K, int log2g,
    uint8_t* __restrict__ wc, uint16_t* __restrict__ ws, int32_t* __restrict__ cs) {
  __shared__ float red[PW_THREADS / 64];
  __shared__ int gsum[PW_MAX_GROUPS];
  const int64_t n = blockIdx.x;
  const int tid = threadIdx.x;
  const int64_t KB = wblk_kblocks(K);
  if (n >= N) {  // padding rows of the last band: zero codes
    for (int64_t kk = tid * 4; kk < KB * 64; kk += PW_THREADS * 4)
      *reinterpret_cast<uint32_t*>(wc + wblk_off(n, kk, KB)) = 0u;
    return;
  }
  // padding k of the row's last block
  for (int64_t kk = (K >> 1) + tid * 4; kk < KB * 64; kk += PW_THREADS * 4)
    *reinterpret_cast<uint32_t*>(wc + wblk_off(n, kk, KB)) = 0u;
  const float* row = w + n * K;
  const int G = (int)(K >> log2g);

  for (int b = tid; b < G; b += PW_THREADS) gsum[b] = 0;

  float amax = 0.0f;
  for (int64_t k = tid * 4; k < K; k += PW_THREADS * 4) {
    const float4 v = *reinterpret_cast<const float4*>(row + k);
    amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v.x), fabsf(v.y)), fmaxf(fabsf(v.z), fabsf(v.w))));
  }
  for (int off = 32; off >= 1; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  if ((tid & 63) == 0) red[tid >> 6] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));

  float s;
  {
#pragma clang fp contract(off)
    s = (amax == 0.0f) ? 1.0f : amax / 7.0f;
  }
  s = fminf(fmaxf(s, 0x1p-24f), 65504.0f);
  const _Float16 h = (_Float16)s;
  const double sq = (double)(float)h;
  if (tid == 0) ws[n] = __builtin_bit_cast(uint16_t, h);

  // 8 weights -> 4 bytes per step
  for (int64_t k = tid * 8; k < K; k += PW_THREADS * 8) {
    const float4 v0 = *reinterpret_cast<const float4*>(row + k);
    const float4 v1 = *reinterpret_cast<const float4*>(row + k + 4);
    const float f[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
    uint32_t packed = 0;
    int sum = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      double q = __builtin_rint((double)f[j] / sq);
      q = fmin(fmax(q, -8.0), 7.0);
      const int qi = (int)q;
      sum += qi;
      packed |= ((uint32_t)qi & 0xfu) << (4 * j);
    }
    *reinterpret_cast<uint32_t*>(wc + wblk_off(n, k >> 1, KB)) = packed;
    atomicAdd(&gsum[(int)(k >> log2g)], sum);
  }
  __syncthreads();
  for (int b = tid; b < G; b += PW_THREADS) cs[(int64_t)b * N + n] = gsum[b];
}

}  // namespace

hipError_t launch_pack_weights(const float* w, int64_t N, int64_t K, int log2g,
                               uint8_t* w_codes, uint16_t* w_scale,
                               int32_t* w_colsum, hipStream_t stream) {
  if ((K >> log2g) > PW_MAX_GROUPS) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pack_weights_kernel, dim3((unsigned)((N + 15) / 16 * 16)), dim3(PW_THREADS), 0, stream, w,
                     N, K, log2g, w_codes, w_scale, w_colsum);
  return hipGetLastError();
}

}  // namespace offq
