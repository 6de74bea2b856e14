// Exhaustive GPU check of the division-free quotients used by the quantizer
// (paper_2606_07116_amd/csrc/common.h) against IEEE fp32 division:
//   div15_rn(d)    for every float d with d / 15 in [2^-25, 2^17]
//   rcp_fp16_rn(s) for every positive finite fp16 value s
// Prints the mismatch counts; exit status 0 when both are zero.
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

int main() {
  unsigned long long* bad = nullptr;
  if (hipMalloc(&bad, 2 * sizeof(unsigned long long)) != hipSuccess) return 2;
  (void)hipMemset(bad, 0, 2 * sizeof(unsigned long long));
  const uint32_t lo = __builtin_bit_cast(uint32_t, 15.0f * 0x1p-25f);
  const uint32_t hi = __builtin_bit_cast(uint32_t, 15.0f * 0x1p17f);
  const uint32_t n = hi - lo + 1;
  hipLaunchKernelGGL(check_div15, dim3((n + 255) / 256), dim3(256), 0, 0, lo, n, bad);
  hipLaunchKernelGGL(check_rcp, dim3(0x7c00 / 256), dim3(256), 0, 0, bad + 1);
  unsigned long long h[2] = {1, 1};
  const hipError_t e = hipDeviceSynchronize();
  (void)hipMemcpy(h, bad, sizeof(h), hipMemcpyDeviceToHost);
  printf("div15_rn: %u inputs, %llu mismatches\n", n, h[0]);
  printf("rcp_fp16_rn: %u inputs, %llu mismatches\n", 0x7c00u - 1, h[1]);
  (void)hipFree(bad);
  return (e == hipSuccess && h[0] == 0 && h[1] == 0) ? 0 : 1;
}
