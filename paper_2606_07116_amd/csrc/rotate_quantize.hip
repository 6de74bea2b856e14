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
// elements of the group sequence, i.e. T / g whole groups, with E registers
// per lane: 16 for g <= 128, 32 for g = 256 and 512, 64 for g = 1024 .. 4096,
// 128 for g = 8192.  A workgroup takes one tile, except with 4096-element
// tiles, whose LDS buffer leaves two waves per SIMD: there the grid holds the
// resident workgroups and each walks its tiles with the next one's loads in
// flight.  Tile element i sits in
//   layout A: lane i[8:3], register i[2:0] | i[high:9] << 3
//             (16-byte chunks: coalesced bf16 loads, packed code stores)
//   layout B: lane i[2:0] | i[S+2:S] << 3, register i[S-1:3] (| i[12] << 6
//             when E = 128), with S = 3 + min(log2 E, 6)
// The Walsh-Hadamard butterflies for the index bits held in registers run in
// registers: bits {0, 1, 2, 9, ...} in layout A, then bits {3, ..., S-1} in
// layout B, which completes every group (for g = 512, bit 8 is lane bit 3 of
// layout B: one DPP exchange between lanes l and l ^ 8).  Group statistics, parameters and
// codes are computed in layout B for g >= 128 (a lane then holds 16 or more
// elements of a single group), in layout A for smaller groups.  The codes
// return to layout A through LDS and are packed 8 per dword.  The layouts are
// exchanged through a padded LDS buffer; one wave per workgroup.
#include <type_traits>

#include "common.h"
#include "internal.h"

namespace offq {
namespace {

// Tiles of 2^LOGE registers per lane that one workgroup walks in a loop (the
// next tile's loads in flight) rather than one per workgroup: those whose LDS
// buffer leaves few waves resident.
#ifndef RQ_LOOP_MIN_LOGE
#define RQ_LOOP_MIN_LOGE 6
#endif
#define RQ_LOOPS(LOGE) ((LOGE) >= RQ_LOOP_MIN_LOGE)

template <int LOGG>
struct Geom {
  static constexpr int LOGE = LOGG <= 7 ? 4 : LOGG <= 9 ? 5 : LOGG <= 12 ? 6 : 7;
  static constexpr int E = 1 << LOGE;
  static constexpr int T = 64 * E;
  static constexpr int NCH = E / 8;      // 16-byte chunks per lane in layout A
  static constexpr int GPT = T >> LOGG;  // groups per tile
  static constexpr int SH = (LOGE < 6 ? LOGE : 6) + 3;
  // LDS word of tile element i: 4 words of padding after every 32 elements and
  // 8 after every 2^SH.  A layout-B 4-byte access then puts the 64 lanes in 64
  // distinct banks (32 distinct per half-wave), each 8-lane phase of a
  // layout-A 16-byte access covers 32 distinct banks, and every address is a
  // per-lane base plus a compile-time offset.
  static constexpr int word(int i) { return i + 4 * (i >> 5) + 8 * (i >> SH); }
  static constexpr int WORDS = word(T - 1) + 1;
  // layout A: element (lane, chunk ch, j) is i = 512 ch + 8 lane + j
  static constexpr int elem_a(int lane, int ch, int j) { return 512 * ch + 8 * lane + j; }
  static constexpr int a_base(int lane) {
    return 8 * lane + 4 * (lane >> 2) + 8 * (lane >> (SH - 3));
  }
  static constexpr int a_off(int ch) { return 576 * ch + 8 * ((512 * ch) >> SH); }
  // layout B: element (lane, register r)
  static constexpr int elem_b(int lane, int r) {
    return (lane & 7) + 8 * (r & 63) + (1 << SH) * (lane >> 3) + 4096 * (r >> 6);
  }
  static constexpr int b_base(int lane) {
    return (lane & 7) + ((1 << SH) + (1 << (SH - 3)) + 8) * (lane >> 3);
  }
  static constexpr int b_off(int r) {
    return 8 * (r & 63) + 4 * ((r & 63) >> 2) + word(4096) * (r >> 6);
  }
};

// The affine address maps agree with word(element) for every lane, chunk and
// register of every tile shape.
template <int LOGG>
constexpr bool maps_ok() {
  using Gm = Geom<LOGG>;
  for (int lane = 0; lane < 64; ++lane) {
    for (int ch = 0; ch < Gm::NCH; ++ch)
      for (int j = 0; j < 8; j += 4)
        if (Gm::word(Gm::elem_a(lane, ch, j)) != Gm::a_base(lane) + Gm::a_off(ch) + j)
          return false;
    for (int r = 0; r < Gm::E; ++r)
      if (Gm::word(Gm::elem_b(lane, r)) != Gm::b_base(lane) + Gm::b_off(r)) return false;
  }
  return true;
}
static_assert(maps_ok<7>() && maps_ok<8>() && maps_ok<9>() && maps_ok<13>(), "LDS maps");

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

// A butterfly stage with the normalisation c folded in:
// (a + b) c and (a - b) c evaluated as fma(a, c, +-(b c)).
template <int E, int RB>
__device__ __forceinline__ void butterfly_scaled(float* v, float c) {
#pragma unroll
  for (int r = 0; r < E; ++r) {
    if (!(r & (1 << RB))) {
      const float a = v[r], bc = v[r | (1 << RB)] * c;
      v[r] = __builtin_fmaf(a, c, bc);
      v[r | (1 << RB)] = __builtin_fmaf(a, c, -bc);
    }
  }
}

// Butterflies over the index bits held in registers in layout A, except bit 0
// (that stage is done while the bf16 input is converted): register bits 1, 2
// and 3.. (index bits 9..).
template <int LOGE, int LOGG>
__device__ __forceinline__ void stages_A(float* v) {
  constexpr int E = 1 << LOGE;
  if constexpr (LOGG > 1) butterfly<E, 1>(v);
  if constexpr (LOGG > 2) butterfly<E, 2>(v);
  if constexpr (LOGG > 9) butterfly<E, 3>(v);   // index bit 9
  if constexpr (LOGG > 10) butterfly<E, 4>(v);  // index bit 10
  if constexpr (LOGG > 11) butterfly<E, 5>(v);  // index bit 11
  if constexpr (LOGG > 12) butterfly<E, 6>(v);  // index bit 12
}

// Butterflies over index bits 3 .. min(log2 g, 9) - 1, held in registers
// 0, 1, .. of layout B.  They complete the transform, so the last one applies
// the factor c when SCALED.
template <int LOGE, int LOGG, bool SCALED, int K>
__device__ __forceinline__ void stage_B(float* v, float c) {
  constexpr int E = 1 << LOGE;
  constexpr int LAST = (LOGG < 9 ? LOGG : 9) - 4;
  if constexpr (K < LAST || (K == LAST && !SCALED)) butterfly<E, K>(v);
  if constexpr (K == LAST && SCALED) butterfly_scaled<E, K>(v, c);
}
template <int LOGE, int LOGG, bool SCALED>
__device__ __forceinline__ void stages_B(float* v, float c) {
  stage_B<LOGE, LOGG, SCALED, 0>(v, c);
  stage_B<LOGE, LOGG, SCALED, 1>(v, c);
  stage_B<LOGE, LOGG, SCALED, 2>(v, c);
  stage_B<LOGE, LOGG, SCALED, 3>(v, c);
  stage_B<LOGE, LOGG, SCALED, 4>(v, c);
  stage_B<LOGE, LOGG, SCALED, 5>(v, c);
}

// a.lo * b.lo + a.hi * b.hi for two packed bf16 pairs, fp32 result.  Through
// the builtin, not inline asm: a VALU that reads a dot result within a few
// cycles needs wait states that only the compiler's hazard tracking inserts.
typedef __bf16 rq_bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(rq_bf16x2, a),
                                         __builtin_bit_cast(rq_bf16x2, b), 0.0f, false);
}

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(float,
                            __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xf, 0xf, true));
}

// max / min over the lanes that differ in lane bits 0 .. NB-1 (all get it)
template <int NB>
__device__ __forceinline__ void lane_reduce(float& mx, float& mn) {
  if constexpr (NB > 0) {
    mx = fmaxf(mx, dpp<0xb1>(mx));  // quad_perm [1,0,3,2]
    mn = fminf(mn, dpp<0xb1>(mn));
  }
  if constexpr (NB > 1) {
    mx = fmaxf(mx, dpp<0x4e>(mx));  // quad_perm [2,3,0,1]
    mn = fminf(mn, dpp<0x4e>(mn));
  }
  if constexpr (NB > 2) {
    mx = fmaxf(mx, dpp<0x141>(mx));  // row_half_mirror
    mn = fminf(mn, dpp<0x141>(mn));
  }
  if constexpr (NB > 3) {
    mx = fmaxf(mx, dpp<0x140>(mx));  // row_mirror
    mn = fminf(mn, dpp<0x140>(mn));
  }
  if constexpr (NB > 4) {
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mn = fminf(mn, __shfl_xor(mn, 16));
  }
  if constexpr (NB > 5) {
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    mn = fminf(mn, __shfl_xor(mn, 32));
  }
}

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

template <int LOGG, bool HAD, bool DBG, bool G1>
__global__ __launch_bounds__(64) void rotate_quantize_kernel(
    const uint16_t* __restrict__ x, int64_t n_groups, int G, uint32_t dm, int dsh, int64_t ldx,
    uint8_t* __restrict__ codes, int64_t ldc, uint16_t* __restrict__ scale,
    int16_t* __restrict__ zero, float* __restrict__ ydbg, int64_t ldy, float cnorm) {
  using Gm = Geom<LOGG>;
  constexpr int LOGE = Gm::LOGE, E = Gm::E, NCH = Gm::NCH, GPT = Gm::GPT;
  static_assert(GPT >= 1, "tile smaller than a group");
  // With an even log2(g) the normalisation 1/sqrt(g) is a power of two: the
  // butterflies' output is kept unscaled and the factor is folded into the
  // quantizer's reciprocal scale, which gives bit-identical codes.
  constexpr bool FOLD = HAD && (LOGG % 2 == 0);
  constexpr bool STATS_B = LOGG >= 7;
  // g = 512 on 2048-element tiles: index bit 8 is lane bit 3 of layout B
  constexpr bool LANE8 = LOGG == 9 && LOGE == 5;
  static_assert(!LANE8 || !FOLD, "g = 512 carries the normalisation in its last stage");
  __shared__ __attribute__((aligned(16))) float lds[Gm::WORDS];
  __shared__ uint32_t s_corr[STATS_B ? GPT : 1];  // bits(lo) * 0x11111111 per group

  // (the id builtins directly: this file's NaN/IEEE flags keep the device
  // library's id functions from being inlined)
  const int lane = (int)__builtin_amdgcn_workitem_id_x();
  float* const la = lds + Gm::a_base(lane);
  float* const lb = lds + Gm::b_base(lane);
  // GPT is a power of two: tiles by shift (no 64-bit division)
  constexpr int LOG_GPT = LOGE + 6 - LOGG;
  static_assert((1 << LOG_GPT) == GPT, "groups per tile");
  const int64_t n_tiles = (n_groups + GPT - 1) >> LOG_GPT;

  // Per chunk: element offset into x and byte offset into the codes of the 8
  // elements this lane holds in layout A.  For g >= 512 the chunk's group is
  // the same for every lane (scalar arithmetic).  Groups past the end are
  // clamped to the last one: read, never stored.
  // With one group per row and g < 512 the tile is GPT whole rows: a chunk's
  // elements are addressed from a wave-uniform base (the chunk's first row in
  // a full tile, the tile's first row otherwise) plus a 32-bit lane offset,
  // which in a full tile is the same for every chunk (the launcher checks
  // that GPT rows fit in 32-bit offsets).
  constexpr bool ROWS = LOGG < 9 && G1;
  struct Addr {
    int64_t xoff[NCH], coff[NCH];
    const uint16_t* xb[NCH];
    uint8_t* cb[NCH];
    uint32_t xo[NCH], co[NCH];
  };
  // (a 64-bit comparison is vector work on gfx950; readfirstlane keeps the
  // flag, and the addressing chosen by it, in scalar registers)
  auto is_full = [&](int64_t gbase) -> bool {
    return __builtin_amdgcn_readfirstlane((int)(gbase + GPT <= n_groups)) != 0;
  };
  auto locate = [&](int64_t gbase, bool full, Addr& A) __attribute__((always_inline)) {
    if constexpr (ROWS) {
      const uint16_t* const xt = x + gbase * ldx;
      uint8_t* const ct = codes + gbase * ldc;
      // row gbase + (ch << (9 - log2 g)) + (lane >> (log2 g - 3)), clamped
      const int lr = lane >> (LOGG - 3);
      const int c = 8 * (lane & ((1 << (LOGG - 3)) - 1));
      if (full) {
        // (24-bit multiplies: lr < 64 and the launcher keeps strides below 2^24)
        const uint32_t xl = (uint32_t)lr * ((uint32_t)ldx & 0xffffffu) + c;
        const uint32_t cl = (uint32_t)lr * ((uint32_t)ldc & 0xffffffu) + (c >> 1);
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch) {
          const int r0 = ch << (9 - LOGG);
          A.xb[ch] = xt + (int64_t)r0 * ldx;
          A.cb[ch] = ct + (int64_t)r0 * ldc;
          A.xo[ch] = xl;
          A.co[ch] = cl;
        }
      } else {
        const int last = (int)(n_groups - 1 - gbase);  // < GPT - 1 here
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch) {
          const int r = min((ch << (9 - LOGG)) + lr, last);
          A.xb[ch] = xt;
          A.cb[ch] = ct;
          A.xo[ch] = (uint32_t)(r * (int)ldx + c);
          A.co[ch] = (uint32_t)(r * (int)ldc + (c >> 1));
        }
      }
    } else {
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        int64_t q;
        int c;  // channel of the chunk's first element inside its group
        if constexpr (LOGG >= 9) {
          q = gbase + (ch >> (LOGG - 9));
          c = ((ch & ((1 << (LOGG - 9)) - 1)) << 9) + 8 * lane;
        } else {
          q = gbase + (ch << (9 - LOGG)) + (lane >> (LOGG - 3));
          c = 8 * (lane & ((1 << (LOGG - 3)) - 1));
        }
        if (q >= n_groups) q = n_groups - 1;
        uint32_t row, col0;
        group_loc<G1>((uint32_t)q, G, dm, dsh, LOGG, row, col0);
        A.xoff[ch] = (int64_t)row * ldx + col0 + c;
        A.coff[ch] = (int64_t)row * ldc + ((col0 + c) >> 1);
      }
    }
  };
  auto xptr = [&](const Addr& A, int ch) -> const uint16_t* {
    if constexpr (ROWS) return A.xb[ch] + A.xo[ch];
    else return x + A.xoff[ch];
  };
  auto cptr = [&](const Addr& A, int ch) -> uint8_t* {
    if constexpr (ROWS) return A.cb[ch] + A.co[ch];
    else return codes + A.coff[ch];
  };

  // Each workgroup walks the tiles blockIdx.x, + gridDim.x, ...; a tile's
  // 16-byte chunks (layout A: chunk ch of a lane = 8 consecutive bf16) are
  // requested while the previous tile is rotated and quantized, so that a
  // resident wave always has a load in flight (a 4096-element tile's LDS
  // leaves two waves per SIMD).
  uint4 raw[NCH];
  auto request = [&](int64_t gbase) __attribute__((always_inline)) {
    Addr A;
    locate(gbase, is_full(gbase), A);
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) raw[ch] = *reinterpret_cast<const uint4*>(xptr(A, ch));
  };
  float v[E];
  // ---- widen (layout A) ------------------------------------------------------
  // With the rotation, butterfly stage 0 (pairs 2j, 2j+1 = the two halves of
  // one 32-bit word) is fused with the bf16 -> fp32 conversion: one dot2 each
  // for the sum and the difference.
  auto widen = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      const uint4 d = raw[ch];
      const uint32_t w[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if constexpr (HAD) {
          v[ch * 8 + 2 * j] = dot2_bf16(w[j], 0x3f803f80u);      // (1, 1)
          v[ch * 8 + 2 * j + 1] = dot2_bf16(w[j], 0xbf803f80u);  // (1, -1)
        } else {
          v[ch * 8 + 2 * j] = bf16_lo(w[j]);
          v[ch * 8 + 2 * j + 1] = bf16_hi(w[j]);
        }
      }
    }
  };
  // The rest of a tile (its chunks widened in v), in one copy for full tiles,
  // whose stores are all unconditional (so that the wait for the next tile's
  // chunks, issued before them, counts them exactly instead of draining
  // them), and one for the partial last tile.
  auto rest = [&](int64_t gbase, auto FULLC) __attribute__((always_inline)) {
    constexpr bool full = decltype(FULLC)::value;
    Addr A;
    locate(gbase, full, A);
    // groups of the tile that exist (uniform)
    const int nleft = full ? GPT : (int)(n_groups - gbase);
    auto stored = [&](int ch) -> bool { return full || (((ch << 9) | (lane << 3)) >> LOGG) < nleft; };

    if constexpr (HAD) stages_A<LOGE, LOGG>(v);

    // ---- A -> B ---------------------------------------------------------------
  #pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      *reinterpret_cast<float4*>(la + Gm::a_off(ch)) =
          make_float4(v[ch * 8 + 0], v[ch * 8 + 1], v[ch * 8 + 2], v[ch * 8 + 3]);
      *reinterpret_cast<float4*>(la + Gm::a_off(ch) + 4) =
          make_float4(v[ch * 8 + 4], v[ch * 8 + 5], v[ch * 8 + 6], v[ch * 8 + 7]);
    }
    __syncthreads();
  #pragma unroll
    for (int r = 0; r < E; ++r) v[r] = lb[Gm::b_off(r)];
    if constexpr (HAD) {
      if constexpr (LANE8) {
        stages_B<LOGE, 8, false>(v, 1.0f);  // index bits 3..7
        // bit 8 (g = 512 on 2048-element tiles): lanes l and l ^ 8, the lower
        // one keeps a + b, the upper one a - b; the last stage carries
        // 1 / sqrt(g): a c + b c, a c - b c
        const float sc = (lane & 8) ? -cnorm : cnorm;
#pragma unroll
        for (int r = 0; r < E; ++r) v[r] = __builtin_fmaf(v[r], sc, dpp<0x128>(v[r]) * cnorm);  // row_ror:8
      } else {
        stages_B<LOGE, LOGG, !FOLD>(v, cnorm);
      }
    }
    // v now holds y in layout B (y / cnorm when folded)

    if constexpr (DBG) {
      // y to global through LDS, in layout A (16-byte stores)
      const float c = FOLD ? cnorm : 1.0f;
      __syncthreads();
  #pragma unroll
      for (int r = 0; r < E; ++r) lb[Gm::b_off(r)] = v[r] * c;
      __syncthreads();
  #pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        if (stored(ch)) {
          const int64_t xe = xptr(A, ch) - x;
          const int64_t row = xe / ldx;
          float* yp = ydbg + row * ldy + (xe - row * ldx);
          *reinterpret_cast<float4*>(yp) = *reinterpret_cast<const float4*>(la + Gm::a_off(ch));
          *reinterpret_cast<float4*>(yp + 4) =
              *reinterpret_cast<const float4*>(la + Gm::a_off(ch) + 4);
        }
      }
    }

    uint32_t corr[NCH];  // per chunk: bits(lo) * 0x11111111 of its group
    if constexpr (STATS_B) {
      // ---- statistics, parameters and codes in layout B ----------------------
      // All E registers of a lane belong to one group, which spans lane bits
      // 0 .. NB-1: group lane >> 3 of the tile when g <= 256, lane >> 4 for
      // g = 512 (2048-element tiles), lane >> (log2 g - 6) when g >= 1024.
      constexpr int NB = LANE8 ? 4 : LOGG <= 9 ? 3 : LOGG - 6;
      float mx = v[0], mn = v[0];
  #pragma unroll
      for (int r = 1; r < E; ++r) {
        mx = fmaxf(mx, v[r]);
        mn = fminf(mn, v[r]);
      }
      lane_reduce<NB < 6 ? NB : 6>(mx, mn);
      QParams P = FOLD ? quant_params(mx * cnorm, mn * cnorm) : quant_params(mx, mn);
      if constexpr (FOLD) P.r *= cnorm;  // exact: cnorm is a power of two
      const int gi = lane >> NB;
      if ((lane & ((1 << NB) - 1)) == 0) s_corr[gi] = __float_as_uint(P.lo) * 0x11111111u;
      // (full tile: every lane of the group stores the same values)
      if (full || ((lane & ((1 << NB) - 1)) == 0 && gi < nleft)) {
        scale[gbase + gi] = P.s16;
        zero[gbase + gi] = P.z;
      }
      // codes as float bits, back to layout A
      __syncthreads();
  #pragma unroll
      for (int r = 0; r < E; ++r) lb[Gm::b_off(r)] = __uint_as_float(quant_bits(v[r], P));
      __syncthreads();
  #pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        const float4 a = *reinterpret_cast<const float4*>(la + Gm::a_off(ch));
        const float4 b = *reinterpret_cast<const float4*>(la + Gm::a_off(ch) + 4);
        v[ch * 8 + 0] = a.x;
        v[ch * 8 + 1] = a.y;
        v[ch * 8 + 2] = a.z;
        v[ch * 8 + 3] = a.w;
        v[ch * 8 + 4] = b.x;
        v[ch * 8 + 5] = b.y;
        v[ch * 8 + 6] = b.z;
        v[ch * 8 + 7] = b.w;
        corr[ch] = s_corr[((ch << 9) | (lane << 3)) >> LOGG];
      }
    } else {
      // ---- back to layout A; statistics, parameters and codes there ----------
      __syncthreads();
  #pragma unroll
      for (int r = 0; r < E; ++r) lb[Gm::b_off(r)] = v[r];
      __syncthreads();
  #pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        const float4 a = *reinterpret_cast<const float4*>(la + Gm::a_off(ch));
        const float4 b = *reinterpret_cast<const float4*>(la + Gm::a_off(ch) + 4);
        v[ch * 8 + 0] = a.x;
        v[ch * 8 + 1] = a.y;
        v[ch * 8 + 2] = a.z;
        v[ch * 8 + 3] = a.w;
        v[ch * 8 + 4] = b.x;
        v[ch * 8 + 5] = b.y;
        v[ch * 8 + 6] = b.z;
        v[ch * 8 + 7] = b.w;
      }
      // a group is 2^(log2 g - 3) consecutive lanes of one chunk
  #pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        float mx = v[ch * 8], mn = v[ch * 8];
  #pragma unroll
        for (int j = 1; j < 8; ++j) {
          mx = fmaxf(mx, v[ch * 8 + j]);
          mn = fminf(mn, v[ch * 8 + j]);
        }
        lane_reduce<LOGG - 3>(mx, mn);
        QParams P = FOLD ? quant_params(mx * cnorm, mn * cnorm) : quant_params(mx, mn);
        if constexpr (FOLD) P.r *= cnorm;
        const int qt = ((ch << 9) | (lane << 3)) >> LOGG;  // group within the tile
        const int64_t q = gbase + qt;
        if (full || ((lane & ((1 << (LOGG - 3)) - 1)) == 0 && qt < nleft)) {
          scale[q] = P.s16;
          zero[q] = P.z;
        }
  #pragma unroll
        for (int j = 0; j < 8; ++j) v[ch * 8 + j] = __uint_as_float(quant_bits(v[ch * 8 + j], P));
        corr[ch] = __float_as_uint(P.lo) * 0x11111111u;
      }
    }

    // ---- pack 8 codes per dword and store (layout A) -------------------------
  #pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      uint32_t w = 0;
  #pragma unroll
      for (int j = 0; j < 8; ++j) w += __float_as_uint(v[ch * 8 + j]) << (4 * j);
      w -= corr[ch];
      if (stored(ch)) *reinterpret_cast<uint32_t*>(cptr(A, ch)) = w;
    }
  };
  const int64_t nfull = n_groups >> LOG_GPT;
  int64_t tile = __builtin_amdgcn_workgroup_id_x();
  request(tile << LOG_GPT);
  widen();
  if constexpr (RQ_LOOPS(LOGE)) {
    // Full tiles in a loop with one exit and no branch around the loads: the
    // next tile's chunks are always requested (past the last tile, the
    // current tile's again, which the cache serves), so that the loop's wait
    // for them counts exactly the loads and stores issued since.
    const int64_t step = __builtin_amdgcn_readfirstlane((int)gridDim.x);
    while (tile < nfull) {
      const int64_t next = tile + step;
      request((next < n_tiles ? next : tile) << LOG_GPT);
      rest(tile << LOG_GPT, std::true_type{});
      tile = next;
      __syncthreads();  // the next tile's exchanges reuse the LDS buffer
      widen();
    }
    if (tile < n_tiles) rest(tile << LOG_GPT, std::false_type{});
  } else {  // one tile per workgroup
    if (tile < nfull) rest(tile << LOG_GPT, std::true_type{});
    else rest(tile << LOG_GPT, std::false_type{});
  }
}

// g = 2048 NW (4096 or 8192) with one group per row, NW waves per row: wave
// w holds the row's elements [2048 w, 2048 w + 2048) in the E = 32 layouts
// of Geom<8>.  The butterflies on index bits 0-2, 9, 10 run in layout A's
// registers and on bits 3-7 in layout B's; bit 8 is lane bit 3 in layout B
// (a DPP exchange with the lane 8 away, rotating each 16-lane row by 8); bits
// 11 and up are the wave (one exchange through LDS each).  The row's max and
// min meet in LDS; every wave then quantizes its part with the row's
// parameters.  The normalisation is folded into the reciprocal scale when it
// is a power of two (g = 4096) and applied in the last exchange otherwise.
// Rows then run on NW waves each: more waves in flight for a few thousand
// rows, and a shorter chain per wave for a decode step's few rows.
template <int NW, bool HAD, bool DBG>
__global__ __launch_bounds__(64 * NW) void rotate_quantize_rows_kernel(
    const uint16_t* __restrict__ x, int64_t ldx, uint8_t* __restrict__ codes, int64_t ldc,
    uint16_t* __restrict__ scale, int16_t* __restrict__ zero, float* __restrict__ ydbg,
    int64_t ldy, float cnorm) {
  using Gm = Geom<8>;
  constexpr int E = Gm::E, NCH = Gm::NCH;
  static_assert(E == 32 && NCH == 4 && Gm::T == 2048, "2048-element tiles");
  constexpr int LOGW = NW == 2 ? 1 : 2;
  static_assert(NW == (1 << LOGW), "two or four waves");
  constexpr bool FOLD = (11 + LOGW) % 2 == 0;  // 1 / sqrt(g) a power of two
  __shared__ __attribute__((aligned(16))) float lds[NW * Gm::WORDS];
  __shared__ float s_st[NW][2];
  const int tid = (int)__builtin_amdgcn_workitem_id_x();
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t row = (int64_t)__builtin_amdgcn_workgroup_id_x();
  const uint16_t* const xr = x + row * ldx + 2048 * w;
  float* const la = lds + w * Gm::WORDS + Gm::a_base(lane);
  float* const lb = lds + w * Gm::WORDS + Gm::b_base(lane);

  float v[E];
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    const uint4 d = *reinterpret_cast<const uint4*>(xr + 512 * ch + 8 * lane);
    const uint32_t wd[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if constexpr (HAD) {
        v[ch * 8 + 2 * j] = dot2_bf16(wd[j], 0x3f803f80u);      // (1, 1)
        v[ch * 8 + 2 * j + 1] = dot2_bf16(wd[j], 0xbf803f80u);  // (1, -1)
      } else {
        v[ch * 8 + 2 * j] = bf16_lo(wd[j]);
        v[ch * 8 + 2 * j + 1] = bf16_hi(wd[j]);
      }
    }
  }
  if constexpr (HAD) stages_A<5, 11>(v);  // index bits 1, 2, 9, 10

  // ---- A -> B ---------------------------------------------------------------
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    *reinterpret_cast<float4*>(la + Gm::a_off(ch)) =
        make_float4(v[ch * 8 + 0], v[ch * 8 + 1], v[ch * 8 + 2], v[ch * 8 + 3]);
    *reinterpret_cast<float4*>(la + Gm::a_off(ch) + 4) =
        make_float4(v[ch * 8 + 4], v[ch * 8 + 5], v[ch * 8 + 6], v[ch * 8 + 7]);
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < E; ++r) v[r] = lb[Gm::b_off(r)];
  if constexpr (HAD) {
    stages_B<5, 8, false>(v, 1.0f);  // index bits 3..7
    // bit 8: lanes l and l ^ 8; the lower one keeps a + b, the upper one a - b
    const float sg = (lane & 8) ? -1.0f : 1.0f;
#pragma unroll
    for (int r = 0; r < E; ++r) v[r] = __builtin_fmaf(v[r], sg, dpp<0x128>(v[r]));  // row_ror:8
    // bits 11..: the waves w and w ^ 2^b, through LDS
#pragma unroll
    for (int b = 0; b < LOGW; ++b) {
      __syncthreads();  // every wave is done reading the regions it read last
#pragma unroll
      for (int r = 0; r < E; ++r) lb[Gm::b_off(r)] = v[r];
      __syncthreads();
      const float* const lp = lds + (w ^ (1 << b)) * Gm::WORDS + Gm::b_base(lane);
      const bool upper = (w >> b) & 1;
      if (FOLD || b < LOGW - 1) {
        const float sw = upper ? -1.0f : 1.0f;
#pragma unroll
        for (int r = 0; r < E; ++r) v[r] = __builtin_fmaf(v[r], sw, lp[Gm::b_off(r)]);
      } else {  // the last stage carries 1 / sqrt(g): a c + b c, a c - b c
        const float sc = upper ? -cnorm : cnorm;
#pragma unroll
        for (int r = 0; r < E; ++r) v[r] = __builtin_fmaf(v[r], sc, lp[Gm::b_off(r)] * cnorm);
      }
    }
  }
  // v now holds y (y / 2^-6 when folded), or x without the rotation, in layout B

  // ---- the row's max and min --------------------------------------------------
  float mx = v[0], mn = v[0];
#pragma unroll
  for (int r = 1; r < E; ++r) {
    mx = fmaxf(mx, v[r]);
    mn = fminf(mn, v[r]);
  }
  lane_reduce<6>(mx, mn);
  if (lane == 0) {
    s_st[w][0] = mx;
    s_st[w][1] = mn;
  }
  __syncthreads();  // (also: every wave is done reading the others' parts)
  mx = s_st[0][0];
  mn = s_st[0][1];
#pragma unroll
  for (int u = 1; u < NW; ++u) {
    mx = fmaxf(mx, s_st[u][0]);
    mn = fminf(mn, s_st[u][1]);
  }
  constexpr bool FOLDED = HAD && FOLD;
  QParams P = FOLDED ? quant_params(mx * cnorm, mn * cnorm) : quant_params(mx, mn);
  if constexpr (FOLDED) P.r *= cnorm;  // exact: cnorm is a power of two
  if (w == 0 && lane == 0) {
    scale[row] = P.s16;
    zero[row] = P.z;
  }

  if constexpr (DBG) {
    // y to global through LDS, in layout A (16-byte stores)
#pragma unroll
    for (int r = 0; r < E; ++r) lb[Gm::b_off(r)] = FOLDED ? v[r] * cnorm : v[r];
    __syncthreads();
    float* const yr = ydbg + row * ldy + 2048 * w;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      *reinterpret_cast<float4*>(yr + 512 * ch + 8 * lane) =
          *reinterpret_cast<const float4*>(la + Gm::a_off(ch));
      *reinterpret_cast<float4*>(yr + 512 * ch + 8 * lane + 4) =
          *reinterpret_cast<const float4*>(la + Gm::a_off(ch) + 4);
    }
    __syncthreads();
  }

  // ---- codes as float bits, back to layout A, 8 per dword --------------------
#pragma unroll
  for (int r = 0; r < E; ++r) lb[Gm::b_off(r)] = __uint_as_float(quant_bits(v[r], P));
  __syncthreads();
  const uint32_t corr = __float_as_uint(P.lo) * 0x11111111u;
  uint8_t* const cr = codes + row * ldc + 1024 * w;
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) {
    const float4 a = *reinterpret_cast<const float4*>(la + Gm::a_off(ch));
    const float4 b = *reinterpret_cast<const float4*>(la + Gm::a_off(ch) + 4);
    const float u[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    uint32_t wd = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) wd += __float_as_uint(u[j]) << (4 * j);
    *reinterpret_cast<uint32_t*>(cr + 256 * ch + 4 * lane) = wd - corr;
  }
}

// Workgroups of a kernel that are resident on the current device at once (0
// if the runtime cannot tell): compute units times workgroups per unit.
int64_t resident_workgroups(const void* kern, int threads) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, threads, 0) != hipSuccess)
    return 0;
  return (int64_t)cus * per_cu;
}

template <int LOGG>
hipError_t launch_t(const uint16_t* x, int64_t n_groups, int G, int64_t ldx, bool had,
                    uint8_t* codes, int64_t ldc, uint16_t* scale, int16_t* zero, float* ydbg,
                    int64_t ldy, hipStream_t stream) {
  constexpr int GPT = Geom<LOGG>::GPT;
  const int64_t nblk = (n_groups + GPT - 1) / GPT;
  const dim3 block(64);
  const float cnorm = (float)(1.0 / __builtin_sqrt((double)(1 << LOGG)));
  // magic multiplier for q / G (q < 2^31)
  int lg = 0;
  while ((1 << lg) < G) ++lg;
  const int dsh = 31 + lg;
  const uint32_t dm = (uint32_t)(((uint64_t(1) << dsh) + (uint64_t)G - 1) / (uint64_t)G);
  // 4096-element tiles (g >= 512): as many workgroups as stay resident, each
  // walking its tiles with the next one's loads in flight; smaller tiles
  // leave enough waves resident, one tile per workgroup
#define OFFQ_RQ(HD, DB, G1)                                                                     \
  {                                                                                            \
    auto kern = rotate_quantize_kernel<LOGG, HD, DB, G1>;                                       \
    int64_t nwg = nblk;                                                                         \
    if (RQ_LOOPS(Geom<LOGG>::LOGE)) {                                                           \
      const int64_t res = resident_workgroups((const void*)kern, 64);                           \
      if (res > 0 && res < nwg) nwg = res;                                                      \
    }                                                                                           \
    hipLaunchKernelGGL(kern, dim3((unsigned)nwg), block, 0, stream, x, n_groups, G, dm, dsh,    \
                       ldx, codes, ldc, scale, zero, ydbg, ldy, HD ? cnorm : 1.0f);              \
  }
  // one group per row: the fast addressing when GPT rows fit in 32-bit
  // offsets and the strides in 24 bits
  const bool g1 = G == 1 && (LOGG >= 9 || (GPT * ldx < (int64_t(1) << 31) &&
                                           GPT * ldc < (int64_t(1) << 31) &&
                                           ldx < (int64_t(1) << 24) && ldc < (int64_t(1) << 24)));
  if constexpr (LOGG == 12 || LOGG == 13) {
    // one group per row: a row on 2 (g = 4096) or 4 (g = 8192) waves
    if (G == 1) {
      constexpr int NW = 1 << (LOGG - 11);
#define OFFQ_RQW(HD, DB)                                                                \
  hipLaunchKernelGGL((rotate_quantize_rows_kernel<NW, HD, DB>), dim3((unsigned)n_groups), \
                     dim3(64 * NW), 0, stream, x, ldx, codes, ldc, scale, zero, ydbg, ldy, cnorm)
      if (had) {
        if (ydbg) OFFQ_RQW(true, true); else OFFQ_RQW(true, false);
      } else {
        if (ydbg) OFFQ_RQW(false, true); else OFFQ_RQW(false, false);
      }
#undef OFFQ_RQW
      return hipGetLastError();
    }
  }
#define OFFQ_RQ_G(HD, DB) \
  if (g1) OFFQ_RQ(HD, DB, true) else OFFQ_RQ(HD, DB, false)
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
#define OFFQ_RQ_CASE(L)                                                                        \
  case L:                                                                                      \
    return launch_t<L>(x, n_groups, G, ldx, hadamard, codes, ldc_bytes, scale, zero, y_debug, \
                       ldy, stream);
  switch (log2g) {
    OFFQ_RQ_CASE(4)
    OFFQ_RQ_CASE(5)
    OFFQ_RQ_CASE(6)
    OFFQ_RQ_CASE(7)
    OFFQ_RQ_CASE(8)
    OFFQ_RQ_CASE(9)
    OFFQ_RQ_CASE(10)
    OFFQ_RQ_CASE(11)
    OFFQ_RQ_CASE(12)
    OFFQ_RQ_CASE(13)
    default:
      return hipErrorInvalidValue;
  }
#undef OFFQ_RQ_CASE
}

}  // namespace offq
