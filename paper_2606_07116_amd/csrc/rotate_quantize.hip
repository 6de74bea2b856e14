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

// Butterflies over the index bits held in registers in layout A, except bit 0
// (that stage is done while the bf16 input is converted).
template <int LOGE, int LOGG>
__device__ __forceinline__ void stages_A(float* v) {
  constexpr int E = 1 << LOGE;
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

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Where group q lives: row q / G and first channel (q % G) * g.  G == 1 is
// the common case (one group per row, and every KV row); otherwise q / G is
// evaluated as (q * m) >> sh with m = ceil(2^sh / G), sh = 31 + ceil(log2 G),
// exact for every q < 2^31.
template <bool G1>
__device__ __forceinline__ void group_loc(uint32_t q, int G, uint32_t m, int sh, int log2g,
                                          uint32_t& row, uint32_t& col0) {
  if constexpr (G1) {
    row = q;
    col0 = 0;
  } else {
    row = (uint32_t)(((uint64_t)q * m) >> sh);
    col0 = (q - row * (uint32_t)G) << log2g;
  }
}

template <int LOGE, int LOGG, bool HAD, bool DBG, bool G1>
__global__ __launch_bounds__(64) void rotate_quantize_kernel(
    const uint16_t* __restrict__ x, int64_t n_groups, int G, uint32_t dm, int dsh, int64_t ldx,
    uint8_t* __restrict__ codes, int64_t ldc, uint16_t* __restrict__ scale,
    int16_t* __restrict__ zero, float* __restrict__ ydbg, int64_t ldy, float cnorm) {
  constexpr int E = 1 << LOGE;
  constexpr int T = 64 * E;
  constexpr int NCH = E / 8;
  constexpr int GPT = T >> LOGG;  // groups per tile (>= 1)
  static_assert(GPT >= 1, "tile smaller than a group");
  // With an even log2(g) the normalisation 1/sqrt(g) is a power of two: the
  // butterflies' output is kept unscaled and the factor is folded into the
  // quantizer's reciprocal scale, which gives bit-identical codes.
  constexpr bool FOLD = HAD && (LOGG % 2 == 0);
  __shared__ __attribute__((aligned(16))) float lds[T];

  const int lane = threadIdx.x;
  const int64_t gbase = (int64_t)blockIdx.x * GPT;
  const bool full = gbase + GPT <= n_groups;

  // per chunk: row and first channel of the 8 elements this lane holds
  uint32_t crow[NCH], ccol[NCH];
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    const int i = (ch << 9) | (lane << 3);
    int64_t q = gbase + (i >> LOGG);
    if (q >= n_groups) q = n_groups - 1;  // clamp: only read, never stored
    uint32_t row, col0;
    group_loc<G1>((uint32_t)q, G, dm, dsh, LOGG, row, col0);
    crow[ch] = row;
    ccol[ch] = col0 + (i & ((1 << LOGG) - 1));
  }

  float v[E];

  // ---- load (layout A): chunk ch of lane = 8 consecutive bf16 -------------
  // With the rotation, butterfly stage 0 (pairs 2j, 2j+1 = the two halves of
  // one 32-bit word) is fused with the bf16 -> fp32 conversion: one dot2 each
  // for the sum and the difference.
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    uint4 d = *reinterpret_cast<const uint4*>(x + (int64_t)crow[ch] * ldx + ccol[ch]);
    const uint32_t w[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if constexpr (HAD) {
        const bf16x2_t b = __builtin_bit_cast(bf16x2_t, w[j]);
        const bf16x2_t pp = {(__bf16)1.0f, (__bf16)1.0f};
        const bf16x2_t pm = {(__bf16)1.0f, (__bf16)-1.0f};
        v[ch * 8 + 2 * j] = __builtin_amdgcn_fdot2_f32_bf16(b, pp, 0.0f, false);
        v[ch * 8 + 2 * j + 1] = __builtin_amdgcn_fdot2_f32_bf16(b, pm, 0.0f, false);
      } else {
        v[ch * 8 + 2 * j] = bf16_lo(w[j]);
        v[ch * 8 + 2 * j + 1] = bf16_hi(w[j]);
      }
    }
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
      const float c = FOLD ? 1.0f : cnorm;
      v[ch * 8 + 0] = a.x * c;
      v[ch * 8 + 1] = a.y * c;
      v[ch * 8 + 2] = a.z * c;
      v[ch * 8 + 3] = a.w * c;
      v[ch * 8 + 4] = b.x * c;
      v[ch * 8 + 5] = b.y * c;
      v[ch * 8 + 6] = b.z * c;
      v[ch * 8 + 7] = b.w * c;
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
    // group max / min of the quantized values y (= v * cnorm, exact when folded)
    QParams P = FOLD ? quant_params(cmx[cg] * cnorm, cmn[cg] * cnorm)
                     : quant_params(cmx[cg], cmn[cg]);
    if constexpr (FOLD) P.r *= cnorm;  // exact: cnorm is a power of two
    const uint32_t corr = __float_as_uint(P.lo) * 0x11111111u;
#pragma unroll
    for (int ch = cg; ch < cg + SP; ++ch) {
      const int i = (ch << 9) | (lane << 3);
      const int64_t q = gbase + (i >> LOGG);
      uint32_t w = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) w += quant_bits(v[ch * 8 + j], P) << (4 * j);
      w -= corr;
      if (full || q < n_groups) {
        *reinterpret_cast<uint32_t*>(codes + (int64_t)crow[ch] * ldc + (ccol[ch] >> 1)) = w;
        if constexpr (DBG) {
          const float c = FOLD ? cnorm : 1.0f;
          float* yp = ydbg + (int64_t)crow[ch] * ldy + ccol[ch];
          *reinterpret_cast<float4*>(yp) = make_float4(v[ch * 8 + 0] * c, v[ch * 8 + 1] * c,
                                                       v[ch * 8 + 2] * c, v[ch * 8 + 3] * c);
          *reinterpret_cast<float4*>(yp + 4) = make_float4(v[ch * 8 + 4] * c, v[ch * 8 + 5] * c,
                                                           v[ch * 8 + 6] * c, v[ch * 8 + 7] * c);
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
hipError_t launch_t(const uint16_t* x, int64_t n_groups, int G, int64_t ldx, bool had,
                    uint8_t* codes, int64_t ldc, uint16_t* scale, int16_t* zero, float* ydbg,
                    int64_t ldy, hipStream_t stream) {
  constexpr int T = 64 << LOGE;
  constexpr int GPT = T >> LOGG;
  const int64_t nblk = (n_groups + GPT - 1) / GPT;
  const dim3 grid((unsigned)nblk), block(64);
  const float cnorm = (float)(1.0 / __builtin_sqrt((double)(1 << LOGG)));
  // magic multiplier for q / G (q < 2^31)
  int lg = 0;
  while ((1 << lg) < G) ++lg;
  const int dsh = 31 + lg;
  const uint32_t dm = (uint32_t)(((uint64_t(1) << dsh) + (uint64_t)G - 1) / (uint64_t)G);
#define OFFQ_RQ(HD, DB, G1)                                                                     \
  hipLaunchKernelGGL((rotate_quantize_kernel<LOGE, LOGG, HD, DB, G1>), grid, block, 0, stream, \
                     x, n_groups, G, dm, dsh, ldx, codes, ldc, scale, zero, ydbg, ldy,         \
                     HD ? cnorm : 1.0f)
#define OFFQ_RQ_G(HD, DB) \
  if (G == 1) OFFQ_RQ(HD, DB, true); else OFFQ_RQ(HD, DB, false);
  if (had) {
    if (ydbg) { OFFQ_RQ_G(true, true) } else { OFFQ_RQ_G(true, false) }
  } else {
    if (ydbg) { OFFQ_RQ_G(false, true) } else { OFFQ_RQ_G(false, false) }
  }
#undef OFFQ_RQ_G
#undef OFFQ_RQ
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
