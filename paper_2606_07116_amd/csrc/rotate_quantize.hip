// Fused online block-Hadamard rotation + per-group 4-bit quantization (gfx950).
//
// Computes, for every group of g channels of a bf16 activation row,
//   y = x_group * H_g * c   (Sylvester H_g, c = fl32(1/sqrt(g)); sec. 3.2, Eq. 4,
//                            applied group-wise as in "Group-Wise Offsetting")
// and quantizes y with the per-group asymmetric quantizer of Eq. 1 (sec. 3),
// fp16 scale and int16 zero-point (sec. 3.4).  The first channel of each group
// becomes the group's constant offset (Eq. 5), absorbed by the zero-point.
//
// Work decomposition: one wavefront owns a tile of T = 64 * E consecutive
// elements (E = 64 registers per lane; E = 128 for g = 8192), i.e. T / g whole
// groups.  Tile element i sits in
//   layout A: lane i[8:3], register i[2:0] | i[high:9] << 3   (16-byte chunks:
//             coalesced bf16 loads, packed code stores)
//   layout B: lane i[2:0] | i[11:9] << 3, register i[8:3] | i[12] << 6
// The Walsh-Hadamard butterflies for index bits held in registers run in
// registers: bits {0,1,2,9,..} in layout A, bits {3..8} in layout B.  The
// two layouts are exchanged through a swizzled LDS buffer (no cross-lane
// arithmetic, no workgroup barrier beyond the wave itself).  Group max/min use
// in-register max/min plus xor-shuffles over the lanes of a group; the codes
// are produced with one fma + one med3 per element and packed 8 per dword.
#include "common.h"
#include "internal.h"

namespace offq {
namespace {

// LDS word for tile element i: xor-swizzle so that both the layout-A 16-byte
// accesses and the layout-B 4-byte accesses are free of bank conflicts.
__device__ __forceinline__ int lds_index(int i) {
  return i ^ (((i >> 9) & 7) << 3) ^ (((i >> 5) & 1) << 2);
}

__device__ __forceinline__ int elem_B(int lane, int r) {
  return (lane & 7) | ((r & 63) << 3) | (((lane >> 3) & 7) << 9) | ((r >> 6) << 12);
}

template <int E, int RB>
__device__ __forceinline__ void butterfly(float* v) {
#pragma unroll
  for (int r = 0; r < E; ++r) {
    if (!(r & (1 << RB))) {
      const float a = v[r], b = v[r | (1 << RB)];
      v[r] = a + b;
      v[r | (1 << RB)] = a - b;
    }
  }
}

// Butterflies over the index bits held in registers in layout A.
template <int LOGE, int LOGG>
__device__ __forceinline__ void stages_A(float* v) {
  constexpr int E = 1 << LOGE;
  if constexpr (LOGG > 0) butterfly<E, 0>(v);
  if constexpr (LOGG > 1) butterfly<E, 1>(v);
  if constexpr (LOGG > 2) butterfly<E, 2>(v);
  if constexpr (LOGG > 9) butterfly<E, 3>(v);   // index bit 9
  if constexpr (LOGG > 10) butterfly<E, 4>(v);  // index bit 10
  if constexpr (LOGG > 11) butterfly<E, 5>(v);  // index bit 11
  if constexpr (LOGG > 12) {                    // index bit 12
    static_assert(LOGE >= 7, "g = 8192 needs 128 registers per lane");
    butterfly<E, 6>(v);
  }
}

// Butterflies over index bits 3..8, held in registers 0..5 of layout B.
template <int LOGE, int LOGG>
__device__ __forceinline__ void stages_B(float* v) {
  constexpr int E = 1 << LOGE;
  if constexpr (LOGG > 3) butterfly<E, 0>(v);
  if constexpr (LOGG > 4) butterfly<E, 1>(v);
  if constexpr (LOGG > 5) butterfly<E, 2>(v);
  if constexpr (LOGG > 6) butterfly<E, 3>(v);
  if constexpr (LOGG > 7) butterfly<E, 4>(v);
  if constexpr (LOGG > 8) butterfly<E, 5>(v);
}

template <int LOGE, int LOGG, bool HAD, bool DBG>
__global__ __launch_bounds__(64) void rotate_quantize_kernel(
    const uint16_t* __restrict__ x, int64_t n_groups, int G, int64_t ldx,
    uint8_t* __restrict__ codes, int64_t ldc, uint16_t* __restrict__ scale,
    int16_t* __restrict__ zero, float* __restrict__ ydbg, int64_t ldy,
    float cnorm) {
  constexpr int E = 1 << LOGE;
  constexpr int T = 64 * E;
  constexpr int NCH = E / 8;
  constexpr int GPT = T >> LOGG;  // groups per tile (>= 1)
  static_assert(GPT >= 1, "tile smaller than a group");
  __shared__ __attribute__((aligned(16))) float lds[T];

  const int lane = threadIdx.x;
  const int64_t gbase = (int64_t)blockIdx.x * GPT;

  float v[E];

  // ---- load (layout A): chunk ch of lane = 8 consecutive bf16 -------------
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    const int i = (ch << 9) | (lane << 3);
    const int64_t q = gbase + (i >> LOGG);
    uint4 d = make_uint4(0u, 0u, 0u, 0u);
    if (q < n_groups) {
      const int64_t row = q / G;
      const int64_t col = ((q - row * G) << LOGG) + (i & ((1 << LOGG) - 1));
      d = *reinterpret_cast<const uint4*>(x + row * ldx + col);
    }
    v[ch * 8 + 0] = bf16_lo(d.x);
    v[ch * 8 + 1] = bf16_hi(d.x);
    v[ch * 8 + 2] = bf16_lo(d.y);
    v[ch * 8 + 3] = bf16_hi(d.y);
    v[ch * 8 + 4] = bf16_lo(d.z);
    v[ch * 8 + 5] = bf16_hi(d.z);
    v[ch * 8 + 6] = bf16_lo(d.w);
    v[ch * 8 + 7] = bf16_hi(d.w);
  }

  if constexpr (HAD) {
    stages_A<LOGE, LOGG>(v);
    // A -> B through LDS
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      const int i0 = (ch << 9) | (lane << 3);
      *reinterpret_cast<float4*>(&lds[lds_index(i0)]) =
          make_float4(v[ch * 8 + 0], v[ch * 8 + 1], v[ch * 8 + 2], v[ch * 8 + 3]);
      *reinterpret_cast<float4*>(&lds[lds_index(i0 | 4)]) =
          make_float4(v[ch * 8 + 4], v[ch * 8 + 5], v[ch * 8 + 6], v[ch * 8 + 7]);
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < E; ++r) v[r] = lds[lds_index(elem_B(lane, r))];
    __syncthreads();
    stages_B<LOGE, LOGG>(v);
    // B -> A
#pragma unroll
    for (int r = 0; r < E; ++r) lds[lds_index(elem_B(lane, r))] = v[r];
    __syncthreads();
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      const int i0 = (ch << 9) | (lane << 3);
      const float4 a = *reinterpret_cast<const float4*>(&lds[lds_index(i0)]);
      const float4 b = *reinterpret_cast<const float4*>(&lds[lds_index(i0 | 4)]);
      v[ch * 8 + 0] = a.x * cnorm;
      v[ch * 8 + 1] = a.y * cnorm;
      v[ch * 8 + 2] = a.z * cnorm;
      v[ch * 8 + 3] = a.w * cnorm;
      v[ch * 8 + 4] = b.x * cnorm;
      v[ch * 8 + 5] = b.y * cnorm;
      v[ch * 8 + 6] = b.z * cnorm;
      v[ch * 8 + 7] = b.w * cnorm;
    }
  }

  // ---- group max / min ---------------------------------------------------
  float cmx[NCH], cmn[NCH];
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    float a = v[ch * 8], b = v[ch * 8];
#pragma unroll
    for (int j = 1; j < 8; ++j) {
      a = fmaxf(a, v[ch * 8 + j]);
      b = fminf(b, v[ch * 8 + j]);
    }
    cmx[ch] = a;
    cmn[ch] = b;
  }
  if constexpr (LOGG >= 9) {
    constexpr int S = 1 << (LOGG - 9);  // chunks per group within a lane
#pragma unroll
    for (int ch = 0; ch < NCH; ch += S) {
#pragma unroll
      for (int j = 1; j < S; ++j) {
        cmx[ch] = fmaxf(cmx[ch], cmx[ch + j]);
        cmn[ch] = fminf(cmn[ch], cmn[ch + j]);
      }
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        cmx[ch] = fmaxf(cmx[ch], __shfl_xor(cmx[ch], off));
        cmn[ch] = fminf(cmn[ch], __shfl_xor(cmn[ch], off));
      }
#pragma unroll
      for (int j = 1; j < S; ++j) {
        cmx[ch + j] = cmx[ch];
        cmn[ch + j] = cmn[ch];
      }
    }
  } else {
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
#pragma unroll
      for (int off = 1; off < (1 << (LOGG - 3)); off <<= 1) {
        cmx[ch] = fmaxf(cmx[ch], __shfl_xor(cmx[ch], off));
        cmn[ch] = fminf(cmn[ch], __shfl_xor(cmn[ch], off));
      }
    }
  }

  // ---- parameters, codes, stores ------------------------------------------
  constexpr int SP = LOGG >= 9 ? (1 << (LOGG - 9)) : 1;
#pragma unroll
  for (int cg = 0; cg < NCH; cg += SP) {
    const QParams P = quant_params(cmx[cg], cmn[cg]);
    const uint32_t corr = __float_as_uint(P.lo) * 0x11111111u;
#pragma unroll
    for (int ch = cg; ch < cg + SP; ++ch) {
      const int i = (ch << 9) | (lane << 3);
      const int64_t q = gbase + (i >> LOGG);
      uint32_t w = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) w += quant_bits(v[ch * 8 + j], P) << (4 * j);
      w -= corr;
      if (q < n_groups) {
        const int64_t row = q / G;
        const int64_t col = ((q - row * G) << LOGG) + (i & ((1 << LOGG) - 1));
        *reinterpret_cast<uint32_t*>(codes + row * ldc + (col >> 1)) = w;
        if constexpr (DBG) {
          float* yp = ydbg + row * ldy + col;
          *reinterpret_cast<float4*>(yp) =
              make_float4(v[ch * 8 + 0], v[ch * 8 + 1], v[ch * 8 + 2], v[ch * 8 + 3]);
          *reinterpret_cast<float4*>(yp + 4) =
              make_float4(v[ch * 8 + 4], v[ch * 8 + 5], v[ch * 8 + 6], v[ch * 8 + 7]);
        }
        const bool writer = (LOGG >= 9) ? (lane == 0 && ch == cg)
                                        : ((lane & ((1 << (LOGG >= 9 ? 0 : LOGG - 3)) - 1)) == 0);
        if (writer) {
          scale[q] = P.s16;
          zero[q] = P.z;
        }
      }
    }
  }
}

template <int LOGE, int LOGG>
hipError_t launch_t(const uint16_t* x, int64_t n_groups, int G, int64_t ldx,
                    bool had, uint8_t* codes, int64_t ldc, uint16_t* scale,
                    int16_t* zero, float* ydbg, int64_t ldy, hipStream_t stream) {
  constexpr int T = 64 << LOGE;
  constexpr int GPT = T >> LOGG;
  const int64_t nblk = (n_groups + GPT - 1) / GPT;
  const dim3 grid((unsigned)nblk), block(64);
  const float cnorm = (float)(1.0 / __builtin_sqrt((double)(1 << LOGG)));
  if (had) {
    if (ydbg)
      hipLaunchKernelGGL((rotate_quantize_kernel<LOGE, LOGG, true, true>), grid, block, 0, stream,
                         x, n_groups, G, ldx, codes, ldc, scale, zero, ydbg, ldy, cnorm);
    else
      hipLaunchKernelGGL((rotate_quantize_kernel<LOGE, LOGG, true, false>), grid, block, 0, stream,
                         x, n_groups, G, ldx, codes, ldc, scale, zero, ydbg, ldy, cnorm);
  } else {
    if (ydbg)
      hipLaunchKernelGGL((rotate_quantize_kernel<LOGE, LOGG, false, true>), grid, block, 0, stream,
                         x, n_groups, G, ldx, codes, ldc, scale, zero, ydbg, ldy, 1.0f);
    else
      hipLaunchKernelGGL((rotate_quantize_kernel<LOGE, LOGG, false, false>), grid, block, 0, stream,
                         x, n_groups, G, ldx, codes, ldc, scale, zero, ydbg, ldy, 1.0f);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rotate_quantize(const uint16_t* x, int64_t n_groups, int G,
                                  int64_t ldx, int log2g, bool hadamard,
                                  uint8_t* codes, int64_t ldc_bytes,
                                  uint16_t* scale, int16_t* zero, float* y_debug,
                                  int64_t ldy, hipStream_t stream) {
#define OFFQ_RQ_CASE(L, LE)                                                          \
  case L:                                                                            \
    return launch_t<LE, L>(x, n_groups, G, ldx, hadamard, codes, ldc_bytes, scale, \
                           zero, y_debug, ldy, stream);
  switch (log2g) {
    OFFQ_RQ_CASE(4, 6)
    OFFQ_RQ_CASE(5, 6)
    OFFQ_RQ_CASE(6, 6)
    OFFQ_RQ_CASE(7, 6)
    OFFQ_RQ_CASE(8, 6)
    OFFQ_RQ_CASE(9, 6)
    OFFQ_RQ_CASE(10, 6)
    OFFQ_RQ_CASE(11, 6)
    OFFQ_RQ_CASE(12, 6)
    OFFQ_RQ_CASE(13, 7)
    default:
      return hipErrorInvalidValue;
  }
#undef OFFQ_RQ_CASE
}

}  // namespace offq
