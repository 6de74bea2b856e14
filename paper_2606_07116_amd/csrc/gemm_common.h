// Device helpers shared by the MFMA GEMM kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace offq {
namespace gemm {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

template <int NC>
__device__ __forceinline__ int swz(int row, int c) {
  if constexpr (NC == 4) return c ^ ((row >> 1) & 3);
  else return c ^ (row & 7);
}

__device__ __forceinline__ v4i act_lo(uint4 d) {
  return v4i{(int)(d.x & 0x0f0f0f0fu), (int)(d.y & 0x0f0f0f0fu), (int)(d.z & 0x0f0f0f0fu),
             (int)(d.w & 0x0f0f0f0fu)};
}
__device__ __forceinline__ v4i act_hi(uint4 d) {
  return v4i{(int)((d.x >> 4) & 0x0f0f0f0fu), (int)((d.y >> 4) & 0x0f0f0f0fu),
             (int)((d.z >> 4) & 0x0f0f0f0fu), (int)((d.w >> 4) & 0x0f0f0f0fu)};
}
__device__ __forceinline__ v4i wgt_lo16(uint4 d) {
  return v4i{(int)((d.x << 4) & 0xf0f0f0f0u), (int)((d.y << 4) & 0xf0f0f0f0u),
             (int)((d.z << 4) & 0xf0f0f0f0u), (int)((d.w << 4) & 0xf0f0f0f0u)};
}
__device__ __forceinline__ v4i wgt_hi16(uint4 d) {
  return v4i{(int)(d.x & 0xf0f0f0f0u), (int)(d.y & 0xf0f0f0f0u), (int)(d.z & 0xf0f0f0f0u),
             (int)(d.w & 0xf0f0f0f0u)};
}

// Workgroup barrier whose fence covers LDS only: outstanding global loads
// (the register prefetch of later stages) are not waited for.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Linear workgroup id -> (tile row, tile column): per-XCD regrouping, then
// groups of 4 tile rows walked column by column.
__device__ __forceinline__ void tile_of(int bid, int nwg, int tiles_m, int tiles_n, int& ti,
                                        int& tj) {
  int L = bid;
  if ((nwg & 7) == 0) L = (bid & 7) * (nwg >> 3) + (bid >> 3);
  constexpr int GM = 4;
  const int per_group = GM * tiles_n;
  const int grp = L / per_group;
  const int first = grp * GM;
  const int gm = min(tiles_m - first, GM);
  const int r = L - grp * per_group;
  ti = first + r % gm;
  tj = r / gm;
}

}  // namespace gemm
}  // namespace offq
