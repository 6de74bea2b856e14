// Exhaustive GPU check of the division-free quotients used by the quantizer
// (paper_2606_07116_amd/csrc/common.h) against IEEE fp32 division:
//   div15_rn(d)    for every float d with d / 15 in [2^-25, 2^17]
//   rcp_fp16_rn(s) for every positive finite fp16 value s
// and of its fp32 zero-point rounding zero_point_rn(mn, r) against the fp64
// rounding of the exact product, for r = 1 / s of every such s with -mn r
// at, one ulp either side of, and one ulp of mn either side of every 16th
// half-integer of [-32768, 32768] (and past it), plus random operand bits.
// Prints the mismatch counts; exit status 0 when all are zero.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>

#include "../../paper_2606_07116_amd/csrc/common.h"

__global__ void check_div15(uint32_t lo_bits, uint32_t n, unsigned long long* bad) {
#pragma clang fp contract(off)
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float d = __uint_as_float(lo_bits + i);
  if (__float_as_uint(d / 15.0f) != __float_as_uint(offq::div15_rn(d))) atomicAdd(bad, 1ull);
}

__global__ void check_rcp(unsigned long long* bad) {
#pragma clang fp contract(off)
  const uint32_t h = blockIdx.x * blockDim.x + threadIdx.x;  // fp16 bit pattern
  if (h == 0 || h >= 0x7c00u) return;                       // positive, finite
  const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)h);
  if (__float_as_uint(1.0f / s) != __float_as_uint(offq::rcp_fp16_rn(s))) atomicAdd(bad, 1ull);
}

__device__ int zero_point_f64(float mn, float r) {
  double zd = __builtin_rint(-(double)mn * (double)r);
  zd = fmin(fmax(zd, -32768.0), 32767.0);
  return (int)zd;
}

__global__ void check_zero(unsigned long long* bad) {
#pragma clang fp contract(off)
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  const uint32_t h = 1 + (i >> 12), j = i & 4095;  // fp16 scale bits, case
  if (h >= 0x7c00u) return;
  const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)h);
  const float r = offq::rcp_fp16_rn(s);
  const float t = (float)((int)(j >> 1) - 1026) * 32.0f + 16.5f;  // a half-integer
  uint32_t k = (i * 2654435761u) ^ (i >> 13);
  k ^= k << 7;
  float mn[5] = {-t / r, -t * s, 0.0f, 0.0f, __uint_as_float(k)};
  mn[2] = __uint_as_float(__float_as_uint(mn[0]) + ((j & 1) ? 1u : -1u));  // one ulp in magnitude
  mn[3] = __uint_as_float(__float_as_uint(mn[1]) + ((j & 2) ? 1u : -1u));
  int nb = 0;
  for (int q = 0; q < 5; ++q) {
    if (!__builtin_isfinite(mn[q])) continue;
    nb += offq::zero_point_rn(mn[q], r) != zero_point_f64(mn[q], r);
  }
  if (nb) atomicAdd(bad, (unsigned long long)nb);
}

int main() {
  unsigned long long* bad = nullptr;
  if (hipMalloc(&bad, 3 * sizeof(unsigned long long)) != hipSuccess) return 2;
  (void)hipMemset(bad, 0, 3 * sizeof(unsigned long long));
  const uint32_t lo = __builtin_bit_cast(uint32_t, 15.0f * 0x1p-25f);
  const uint32_t hi = __builtin_bit_cast(uint32_t, 15.0f * 0x1p17f);
  const uint32_t n = hi - lo + 1;
  hipLaunchKernelGGL(check_div15, dim3((n + 255) / 256), dim3(256), 0, 0, lo, n, bad);
  hipLaunchKernelGGL(check_rcp, dim3(0x7c00 / 256), dim3(256), 0, 0, bad + 1);
  hipLaunchKernelGGL(check_zero, dim3((0x7bffu << 12) / 256), dim3(256), 0, 0, bad + 2);
  unsigned long long h[3] = {1, 1, 1};
  const hipError_t e = hipDeviceSynchronize();
  (void)hipMemcpy(h, bad, sizeof(h), hipMemcpyDeviceToHost);
  printf("div15_rn: %u inputs, %llu mismatches\n", n, h[0]);
  printf("rcp_fp16_rn: %u inputs, %llu mismatches\n", 0x7c00u - 1, h[1]);
  printf("zero_point_rn: %u scales x 4096 cases, %llu mismatches\n", 0x7bffu, h[2]);
  (void)hipFree(bad);
  return (e == hipSuccess && h[0] == 0 && h[1] == 0 && h[2] == 0) ? 0 : 1;
}
