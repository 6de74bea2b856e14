// W4A4 GEMM on MFMA (gfx950, v_mfma_i32_32x32x32_i8), for one or several
// quantization groups per row: g = K (full-width online Hadamard: attention
// projection, MLP up/gate) and g < K (block-diagonal rotation, e.g. the MLP
// down projection with 28 groups of 512 channels).
//
//   acc_b[m,n] = sum_{k in group b} q_a[m,k] q_w[n,k]                 (int32)
//   Y[m,n]     = sw[n] * sum_b s[m,b] * (acc_b[m,n] - z[m,b] * colsum[b,n])
//
// (the dequantised product of Eq. 1 with one scale/zero-point per row and
// group; the z * colsum terms carry the absorbed offsets).
//
// Organisation
// * 8 waves per workgroup, two per SIMD.  FM = 2: waves 4 x 2, each 64 tokens
//   x 64 channels (2 x 2 MFMA tiles of 32 x 32), workgroup tile 256 x 128,
//   any number of groups up to GMAX.  FM = 4: waves 2 x 4, each 128 x 64,
//   workgroup tile 256 x 256, one group per row.
// * Operand unpacking (4-bit nibbles to int8 MFMA operands) is VALU work that
//   does not overlap the MFMAs, so each packed byte is unpacked as few times
//   as possible: the operand that four waves share (the weights for FM = 2,
//   the activations for FM = 4) is unpacked once, when its stage is written
//   to LDS, into two int8 planes; the other operand stays packed in LDS and
//   is unpacked in registers by each of the two waves that read it.
// * Stages of 128 k go global memory -> registers (two or four stages ahead)
//   -> an LDS ring of three or four slots; one LDS-only barrier per stage.
//   16-byte chunks are XOR-swizzled by row to spread the LDS banks.  For
//   FM = 2 the packed parts of all slots form one LDS region and the
//   unpacked parts another, each addressed from one register per lane
//   pattern with immediate offsets.
// * Activation codes (0..15) feed the signed i8 MFMA unchanged; weight nibbles
//   are widened to 16 q (high nibble masked, low nibble shifted), so every
//   accumulator holds 16 acc exactly.  Both operands split each 16-byte chunk
//   (32 k) into its low and high nibbles: the same k-permutation on both
//   sides.  The MFMA takes the weight fragment as its row operand and
//   accumulates the transposed tile.
// * At the end of each group (g / 128 stages) the accumulators are folded
//   into fp32 running sums F, F += (s / 16) acc, and the next group's first
//   MFMA starts from zero.  The zero-point terms -sum_b s z colsum_b form a
//   rank-G product added after the last group with fp32 MFMAs (k = group).
//   Row scales, zero-points, column sums and weight scales of the tile sit in
//   LDS from the prologue.  With one group the fold runs in the epilogue, so
//   F takes no registers during the main loop.
// * Epilogue: Y = sw * F -> bf16 through LDS for 16-byte coalesced stores.
// * Tile order is XCD-aware (see tile_of): each XCD walks a block of tile
//   rows, keeping its A and W panels in its own L2.
#include <type_traits>

#include "common.h"
#include "gemm_common.h"
#include "internal.h"

namespace offq {
namespace {

using namespace gemm;

template <int FM, bool ONEG, bool STREAM = false>
struct GCfg {
  static constexpr int THREADS = 512;              // 8 waves, 2 per SIMD
  static constexpr int WAVES_M = FM == 2 ? 4 : 2;
  static constexpr int WROWS = 32 * FM;            // token rows per wave
  static constexpr int BM = WAVES_M * WROWS;       // 256
  static constexpr int BN = (8 / WAVES_M) * 64;    // 128 or 256
  static constexpr bool X_IS_W = FM == 2;          // operand unpacked into LDS
  static constexpr int P_ROWS = X_IS_W ? BM : BN;  // packed operand rows
  static constexpr int X_ROWS = X_IS_W ? BN : BM;  // unpacked operand rows
  static constexpr int P_SLOTS = P_ROWS * 4;       // 16-byte slots: 4 packed chunks per row
  static constexpr int X_SLOTS = X_ROWS * 8;       // 8 int8 chunks per row (4 x lo/hi)
  static constexpr int STAGE_SLOTS = P_SLOTS + X_SLOTS;
  static constexpr int P_LD = P_ROWS * 4 / THREADS;  // packed chunks loaded per thread
  static constexpr int X_LD = X_ROWS * 4 / THREADS;
  static constexpr int KSTAGE = 128;               // k per stage
  // groups whose parameters fit in LDS; LDS ring depth (with four slots the
  // slot of every stage in a 4-stage unrolled loop is a compile-time constant)
  // (STREAM: any number of groups, their parameters staged with the stages
  // through a ring of GR entries)
  static constexpr int GMAX = (FM == 2 && !ONEG && !STREAM) ? 28 : 1;
  static constexpr int NBUF = (FM == 2 && (ONEG || STREAM)) ? 4 : 3;
  static constexpr int GR = STREAM ? 4 : 1;
  // stages held in registers between their global load and their LDS store:
  // the loads are issued NRB stages before the store (one with streamed
  // group parameters, which leaves the registers for reading fragments two
  // k-steps ahead)
  static constexpr int NRB = (FM == 2 && ONEG) ? 4 : STREAM ? 1 : 2;
};

// packed rows: 4 chunks, swizzle c ^ (row/4 mod 4); int8 rows: 8 chunks,
// swizzle c ^ (row/2 mod 8).  (Chosen by measurement: these gave the fewest
// LDS bank-conflict cycles of the XOR swizzles tried.)
__device__ __forceinline__ int pslot(int row, int c) { return row * 4 + (c ^ ((row >> 2) & 3)); }
__device__ __forceinline__ int xslot(int row, int c) { return row * 8 + (c ^ ((row >> 1) & 7)); }

typedef float v16f __attribute__((ext_vector_type(16)));
typedef unsigned int gemm_u32x4 __attribute__((ext_vector_type(4)));

// MODE: stages per group: 1, 2, 4, or a multiple of 8 (MODE 8).  ONEG: one
// group per row (g = K).  STREAM: several groups, any number of them: each
// group's parameters travel with its stages (row scales and zero-points of
// the tile's rows, column sums of its columns) through a small LDS ring, and
// its zero-point term is applied right after its fold, in pairs of groups.
template <bool DBG, int MODE, int FM, bool ONEG, bool STREAM>
__global__ __launch_bounds__(512) void w4a4_gemm_grouped_kernel(
    const uint8_t* __restrict__ A, const uint16_t* __restrict__ a_scale,
    const int16_t* __restrict__ a_zero, const uint8_t* __restrict__ W,
    const uint16_t* __restrict__ w_scale, const int32_t* __restrict__ w_colsum, int M, int N,
    int K, int log2g, uint16_t* __restrict__ Y, int64_t ldy, int32_t* __restrict__ acc_dbg) {
  using C = GCfg<FM, ONEG, STREAM>;
  constexpr bool XW = C::X_IS_W;
  __shared__ uint4 ring[C::NBUF * C::STAGE_SLOTS];
  // per group b: s / 16 and z of the tile's rows, colsum of its columns
  __shared__ float sRS[C::GMAX][C::BM];
  __shared__ short sZ[C::GMAX][C::BM];
  __shared__ float sCS[C::GMAX][C::BN];
  // STREAM: per group b (entry b mod GR): s / 16 and -s z of the rows,
  // colsum of the columns
  __shared__ float gRS[C::GR][C::BM];
  __shared__ float gSZ[C::GR][C::BM];
  __shared__ float gCS[C::GR][C::BN];
  __shared__ __attribute__((aligned(16))) float sSW[C::BN];  // weight scales

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int h = lane >> 5, fr = lane & 31;
  const int wm = wave % C::WAVES_M, wn = wave / C::WAVES_M;

  const int tiles_m = (M + C::BM - 1) / C::BM;
  const int tiles_n = (N + C::BN - 1) / C::BN;
  int ti, tj;
  tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n, ti, tj);
  const int tm = ti * C::BM, tn = tj * C::BN;
  const int64_t ldk = K >> 1;
  const int nst = K / C::KSTAGE;
  const int G = K >> log2g;
  const int spg = 1 << (log2g - 7);  // stages per group

  // LDS addressing.  FM = 2: the packed parts of all ring slots form one
  // region and the unpacked parts another (each at most 64 KB), and every
  // lane pattern (row, swizzled chunk) has one element index, region start
  // included, computed once and hidden from the optimiser: slot and fragment
  // offsets then stay within the 16-bit immediate of ds_read / ds_write,
  // and the loop holds one address register per pattern.  (Folded into
  // per-slot addresses, slots beyond 64 KB each took a register of their
  // own.)  FM = 4: slot s holds its packed then its unpacked part.
  constexpr bool SPLIT = FM == 2;
  constexpr int PBASE = 0, XBASE = SPLIT ? C::NBUF * C::P_SLOTS : C::P_SLOTS;
  constexpr int PSTEP = SPLIT ? C::P_SLOTS : C::STAGE_SLOTS;  // slot stride, packed part
  constexpr int XSTEP = SPLIT ? C::X_SLOTS : C::STAGE_SLOTS;  // slot stride, unpacked part
  static_assert(!SPLIT || (C::NBUF * C::P_SLOTS * 16 <= 65536 && C::NBUF * C::X_SLOTS * 16 <= 65536),
                "each region within one 16-bit LDS offset");
  auto opaque = [](int v) __attribute__((always_inline)) {
    asm volatile("" : "+v"(v));
    return v;
  };
  // ---- global -> registers -> LDS staging -----------------------------------
  // Chunk s = tid + 512 i of an operand's stage is row s / 4, packed chunk
  // s % 4 (16 bytes = 32 k); rows past M (N) read as zero.  Activation rows
  // are row-major (stride K / 2); the weights are in the blocked layout, where
  // a stage of a row is 64 bytes of a 1 KB block of 16 rows.
  const uint8_t* pbase = XW ? A + (int64_t)tm * ldk : W + (int64_t)tn * ldk;
  const uint8_t* xbase = XW ? W + (int64_t)tn * ldk : A + (int64_t)tm * ldk;
  // (weights: bands of 16 rows of the blocked layout, K a multiple of 128, so a
  // band is 16 ldk bytes; the padding rows of the last band hold zero codes)
  const int wrows = (N - tn + 15) & ~15;
  const int prows = XW ? M - tm : wrows, xrows = XW ? wrows : M - tm;
  const __amdgpu_buffer_rsrc_t prsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)pbase, 0, (int)((int64_t)prows * ldk), 0x00020000);
  const __amdgpu_buffer_rsrc_t xrsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)xbase, 0, (int)((int64_t)xrows * ldk), 0x00020000);
  // the same buffers with no valid bytes: loads past the last stage read zeros
  const __amdgpu_buffer_rsrc_t prsrc0 = __builtin_amdgcn_make_buffer_rsrc((void*)pbase, 0, 0, 0x00020000);
  const __amdgpu_buffer_rsrc_t xrsrc0 = __builtin_amdgcn_make_buffer_rsrc((void*)xbase, 0, 0, 0x00020000);
  const int crow = tid >> 2, cch = tid & 3;
  const int voff_a = crow * (int)ldk + cch * 16;
  const int voff_w = (crow >> 4) * 16 * (int)ldk + (crow & 15) * 64 + cch * 16;
  const int pvoff = XW ? voff_a : voff_w, xvoff = XW ? voff_w : voff_a;
  const int vstep = (C::THREADS / 4) * (int)ldk;  // 128 rows (8 weight bands)
  constexpr int NLD = C::P_LD + C::X_LD;
  v4i rgb[C::NRB][NLD];   // stages in flight
  v4i ra[NLD], rb[NLD];    // stages 0 and 1 in the prologue
  uint32_t gqb[C::NRB][2] = {}, gqa0[2] = {}, gqa1[2] = {};  // STREAM: their group parameters
  auto gload = [&](int st, v4i (&rg)[NLD]) __attribute__((always_inline)) {
    const bool ok = st < nst;
    const __amdgpu_buffer_rsrc_t pr = ok ? prsrc : prsrc0, xr = ok ? xrsrc : xrsrc0;
    // a stage is 64 bytes of an activation row, one 1 KB block of a weight band
    const int soff = ok ? st * (C::KSTAGE / 2) : 0;
    const int psoff = XW ? soff : 16 * soff, xsoff = XW ? 16 * soff : soff;
#pragma unroll
    for (int i = 0; i < C::P_LD; ++i)
      rg[i] = __builtin_amdgcn_raw_buffer_load_b128(pr, pvoff + i * vstep, psoff, 0);
#pragma unroll
    for (int i = 0; i < C::X_LD; ++i)
      rg[C::P_LD + i] = __builtin_amdgcn_raw_buffer_load_b128(xr, xvoff + i * vstep, xsoff, 0);
  };
  // element index of this thread's chunk in slot 0 (row crow + 128 i adds
  // 512 i packed / 1024 i unpacked slots: the swizzles repeat every 128 rows)
  const int ps_idx = SPLIT ? opaque(PBASE + pslot(crow, cch)) : 0;
  const int xs_idx0 = SPLIT ? opaque(XBASE + xslot(crow, 2 * cch)) : 0;
  const int xs_idx1 = SPLIT ? opaque(XBASE + xslot(crow, 2 * cch + 1)) : 0;
  auto lstore_p = [&](int slot, const v4i (&rg)[NLD]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < C::P_LD; ++i) {
      if constexpr (SPLIT)
        ring[ps_idx + slot * PSTEP + 512 * i] = __builtin_bit_cast(uint4, rg[i]);
      else
        ring[slot * PSTEP + pslot(crow + 128 * i, cch)] = __builtin_bit_cast(uint4, rg[i]);
    }
  };
  auto lstore_x = [&](int slot, const v4i (&rg)[NLD]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < C::X_LD; ++i) {
      const uint4 d = __builtin_bit_cast(uint4, rg[C::P_LD + i]);
      v4i lo, hi;
      if constexpr (XW) {
        lo = wgt_lo16(d);
        hi = wgt_hi16(d);
      } else {
        lo = act_lo(d);
        hi = act_hi(d);
      }
      if constexpr (SPLIT) {
        ring[xs_idx0 + slot * XSTEP + 1024 * i] = __builtin_bit_cast(uint4, lo);
        ring[xs_idx1 + slot * XSTEP + 1024 * i] = __builtin_bit_cast(uint4, hi);
      } else {
        uint4* X = ring + slot * XSTEP + XBASE;
        X[xslot(crow + 128 * i, 2 * cch)] = __builtin_bit_cast(uint4, lo);
        X[xslot(crow + 128 * i, 2 * cch + 1)] = __builtin_bit_cast(uint4, hi);
      }
    }
  };
  auto lstore = [&](int slot, const v4i (&rg)[NLD]) __attribute__((always_inline)) {
    lstore_p(slot, rg);
    lstore_x(slot, rg);
  };

  // STREAM: the parameters of stage st's group, loaded with the stage's data
  // (thread t < BM: scale and zero-point of row tm + t; BM <= t < BM + BN:
  // colsum of column tn + t - BM) and stored with it.  Rows past M and
  // columns past N read as zero.
  const int lgs = log2g - 7;  // log2(stages per group)
  const __amdgpu_buffer_rsrc_t srsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a_scale + (int64_t)tm * G), 0, STREAM ? (int)((int64_t)min(C::BM, M - tm) * G * 2) : 0,
      0x00020000);
  const __amdgpu_buffer_rsrc_t zrsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a_zero + (int64_t)tm * G), 0, STREAM ? (int)((int64_t)min(C::BM, M - tm) * G * 2) : 0,
      0x00020000);
  const __amdgpu_buffer_rsrc_t crsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(w_colsum + tn), 0, STREAM ? (int)(((int64_t)G * N - tn) * 4) : 0, 0x00020000);
  // Waves 0-3 carry the row parameters, waves 4-5 the column sums (tests on
  // the wave index: scalar branches).  A column past N reads its neighbour's
  // sum in the same buffer (or 0 past its end); it only reaches outputs past
  // N, which are never stored.
  static_assert(C::BM % 64 == 0 && C::BN % 64 == 0, "whole waves per parameter kind");
  const int gt_c = tid - C::BM;  // column of a colsum thread
  const bool g_row = wave < C::BM / 64, g_col = !g_row && wave < (C::BM + C::BN) / 64;
  auto gload_g = [&](int st, uint32_t (&gq)[2]) __attribute__((always_inline)) {
    if constexpr (STREAM) {
      const int b = min(st, nst - 1) >> lgs;
      if (g_row) {
        gq[0] = __builtin_amdgcn_raw_buffer_load_b16(srsrc, (tid * G + b) * 2, 0, 0);
        gq[1] = __builtin_amdgcn_raw_buffer_load_b16(zrsrc, (tid * G + b) * 2, 0, 0);
      } else if (g_col) {
        gq[0] = __builtin_amdgcn_raw_buffer_load_b32(crsrc, (b * N + gt_c) * 4, 0, 0);
      }
    }
  };
  auto lstore_g = [&](int st, const uint32_t (&gq)[2]) __attribute__((always_inline)) {
    if constexpr (STREAM) {
      const int e = (min(st, nst - 1) >> lgs) & (C::GR - 1);
      if (g_row) {
        const float sc = fp16_bits_to_f32((uint16_t)gq[0]);
        gRS[e][tid] = sc * 0.0625f;
        gSZ[e][tid] = -(sc * (float)(int16_t)gq[1]);
      } else if (g_col) {
        gCS[e][gt_c] = (float)(int32_t)gq[0];
      }
    }
  };

  // ---- fragments ---------------------------------------------------------------
  // Per 64 k (chunk column c = 2h + jj of the stage) a wave reads its packed
  // fragments (one 16-byte chunk each) and, per plane pl, its unpacked
  // fragments; lane row fr, fragment f is 32 rows further (which keeps both
  // swizzles).
  constexpr int NPF = XW ? FM : 2;  // packed fragments per wave
  constexpr int NXF = XW ? 2 : FM;  // unpacked fragments per wave
  const int prow0 = (XW ? wm * C::WROWS : wn * 64) + fr;
  const int xrow0 = (XW ? wn * 64 : wm * C::WROWS) + fr;
  // element indices of the lane's fragments in slot 0, per chunk column
  int pr_idx[2] = {}, xr_idx[4] = {};
  if constexpr (SPLIT) {
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) pr_idx[jj] = opaque(PBASE + pslot(prow0, 2 * h + jj));
#pragma unroll
    for (int q = 0; q < 4; ++q) xr_idx[q] = opaque(XBASE + xslot(xrow0, 4 * h + q));
  }
  auto pread = [&](int slot, int jj, uint4 (&pp)[NPF]) __attribute__((always_inline)) {
#pragma unroll
    for (int f = 0; f < NPF; ++f) {
      if constexpr (SPLIT) pp[f] = ring[pr_idx[jj] + slot * PSTEP + f * 32 * 4];
      else pp[f] = ring[slot * PSTEP + pslot(prow0, 2 * h + jj) + f * 32 * 4];
    }
  };
  auto xread = [&](int slot, int jj, int pl, uint4 (&px)[NXF]) __attribute__((always_inline)) {
#pragma unroll
    for (int f = 0; f < NXF; ++f) {
      if constexpr (SPLIT) px[f] = ring[xr_idx[2 * jj + pl] + slot * XSTEP + f * 32 * 8];
      else px[f] = ring[slot * XSTEP + XBASE + xslot(xrow0, 4 * h + 2 * jj + pl) + f * 32 * 8];
    }
  };

  // With one group per row (the only case of FM = 4) F is first written by
  // the single fold after the loop, so it takes no registers during it.
  constexpr bool SINGLE = ONEG;
  v16i acc[FM][2];
  v16f F[FM][2];
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      acc[a][b] = v16i{};
      if constexpr (!SINGLE) F[a][b] = v16f{};
    }

  // Lane column fr of fragment fm is token row wm*WROWS + fm*32 + fr; register
  // i of fragment (fm, fn) is output channel wn*64 + fn*32 + 8*(i/4) + 4*h + i%4.
  // F += (s / 16) * acc for fragment row fm, rs[fm] = s / 16 of the group.
  float rs[FM] = {};
  auto read_rs = [&](int b) __attribute__((always_inline)) {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int r = wm * C::WROWS + fm * 32 + fr;
      rs[fm] = STREAM ? gRS[b & (C::GR - 1)][r] : sRS[b][r];
    }
  };
  // STREAM: zero-point terms of groups b0 and b0 + 1 (b0 even; a group past
  // the last adds nothing), F += sum (-s z)[m] colsum[n], with the fp32 MFMA
  // over k = group: lane half h supplies group b0 + h.
  auto zp_pair = [&](int b0) __attribute__((always_inline)) {
    const int e = b0 + h;
    const bool ok = e < G;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const float szv = ok ? gSZ[e & (C::GR - 1)][wm * C::WROWS + fm * 32 + fr] : 0.0f;
#pragma unroll
      for (int fn = 0; fn < 2; ++fn) {
        const float csv = ok ? gCS[e & (C::GR - 1)][wn * 64 + fn * 32 + fr] : 0.0f;
        F[fm][fn] = __builtin_amdgcn_mfma_f32_32x32x2f32(csv, szv, F[fm][fn], 0, 0, 0);
      }
    }
  };
  auto fold_row = [&](int fm) __attribute__((always_inline)) {
#pragma unroll
    for (int fn = 0; fn < 2; ++fn)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        F[fm][fn][i] = SINGLE ? rs[fm] * (float)acc[fm][fn][i]
                              : __builtin_fmaf(rs[fm], (float)acc[fm][fn][i], F[fm][fn][i]);
  };
  // several groups: the fold of group b (and, STREAM, the zero-point terms
  // of the pair of groups that b completes)
  auto fold_group = [&](int b) __attribute__((always_inline)) {
    read_rs(b);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) fold_row(fm);
    if constexpr (STREAM) {
      if ((b & 1) || b == G - 1) zp_pair(b & ~1);
    }
  };

  // one k-step of 32: plane pl of the packed fragments pp against the
  // unpacked plane px; FRESH: start the accumulators from zero.
  auto mma1 = [&](const uint4 (&pp)[NPF], const uint4 (&px)[NXF], auto PL, auto FC)
      __attribute__((always_inline)) {
    constexpr bool HI = decltype(PL)::value;
    constexpr bool FRESH = decltype(FC)::value;
    if constexpr (XW) {  // activations packed, weights unpacked
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
        const v4i ua = HI ? act_hi(pp[fm]) : act_lo(pp[fm]);
#pragma unroll
        for (int fn = 0; fn < 2; ++fn)
          acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(
              __builtin_bit_cast(v4i, px[fn]), ua, FRESH ? v16i{} : acc[fm][fn], 0, 0, 0);
      }
    } else {  // weights packed, activations unpacked
#pragma unroll
      for (int fn = 0; fn < 2; ++fn) {
        const v4i ub = HI ? wgt_hi16(pp[fn]) : wgt_lo16(pp[fn]);
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
          acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(
              ub, __builtin_bit_cast(v4i, px[fm]), FRESH ? v16i{} : acc[fm][fn], 0, 0, 0);
      }
    }
    if constexpr (FM == 4) {
      // keep the 128 accumulators in accumulation registers (an empty asm
      // with AGPR operands), leaving the vector registers to the pipeline
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < 2; ++fn) asm volatile("" : "+a"(acc[fm][fn]));
    }
  };
  auto dump = [&](int b) __attribute__((always_inline)) {  // debug: raw accumulators of group b
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int row = tm + wm * C::WROWS + fm * 32 + fr;
      if (row >= M) continue;
#pragma unroll
      for (int fn = 0; fn < 2; ++fn)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c0 = tn + wn * 64 + fn * 32 + q * 8 + h * 4;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (c0 + e < N)
              acc_dbg[((int64_t)b * M + row) * N + c0 + e] = acc[fm][fn][q * 4 + e] >> 4;
        }
    }
  };

  // ---- prologue: the group parameters and weight scales of the tile, then
  // the first four stages are requested together; the parameters go to LDS,
  // stages 0 and 1 into the ring, 2 and 3 stay in registers ----------------
  {
    // Row parameters: a contiguous block of 256 G entries of the [M, G]
    // arrays, read coalesced (entry e = tid + 512 p is row e / G, group
    // e % G); column sums: group b, column c = colsum[b * N + tn + c].  They
    // are requested first, so that writing them waits for nothing else.
    const float inv_g = STREAM ? 0.0f : 1.0f / (float)G;
    const int64_t base = (int64_t)tm * G;
    const int nrow_e = min(C::BM, M - tm) * G;  // valid entries of the block
    constexpr int PE = (C::GMAX * C::BM + C::THREADS - 1) / C::THREADS;
    constexpr int PC = (C::GMAX * C::BN + C::THREADS - 1) / C::THREADS;
    uint16_t sv[PE];
    int16_t zv[PE];
#pragma unroll
    for (int p = 0; p < PE; ++p) {
      const int e = tid + C::THREADS * p;
      const bool ok = !STREAM && e < C::BM * G && e < nrow_e;
      sv[p] = ok ? a_scale[base + e] : (uint16_t)0;
      zv[p] = ok ? a_zero[base + e] : (int16_t)0;
    }
    float cv[PC];
#pragma unroll
    for (int p = 0; p < PC; ++p) {
      const int b = (C::THREADS / C::BN) * p + tid / C::BN, c = tid % C::BN;
      cv[p] = (!STREAM && b < G && b < C::GMAX && tn + c < N)
                  ? (float)w_colsum[(int64_t)b * N + tn + c]
                  : 0.0f;
    }
    const float swv = (tid < C::BN && tn + tid < N) ? fp16_bits_to_f32(w_scale[tn + tid]) : 0.0f;
    gload(0, ra);
    gload_g(0, gqa0);
    gload(1, rb);
    gload_g(1, gqa1);
    // stage s > 1 waits in buffer s mod NRB
#pragma unroll
    for (int s2 = 2; s2 < 2 + C::NRB; ++s2) {
      gload(s2, rgb[s2 % C::NRB]);
      gload_g(s2, gqb[s2 % C::NRB]);
    }
#pragma unroll
    for (int p = 0; p < PE; ++p) {
      const int e = tid + C::THREADS * p;
      if (!STREAM && e < C::BM * G) {
        // exact: e < 2^13, and (e + 1/2) / G stays 1/(2G) away from integers
        const int r = (int)(((float)e + 0.5f) * inv_g);
        const int b = e - r * G;
        sRS[b][r] = fp16_bits_to_f32(sv[p]) * 0.0625f;
        sZ[b][r] = zv[p];
      }
    }
#pragma unroll
    for (int p = 0; p < PC; ++p) {
      const int b = (C::THREADS / C::BN) * p + tid / C::BN;
      if (!STREAM && b < G && b < C::GMAX) sCS[b][tid % C::BN] = cv[p];
    }
    if (tid < C::BN) sSW[tid] = swv;
  }
  lstore(0, ra);
  lstore_g(0, gqa0);
  lstore(1, rb);
  lstore_g(1, gqa1);
  lds_barrier();
  // FM = 2 reads each k-step's unpacked fragments two k-steps ahead (xa, xb,
  // x2, x3 hold k-steps 0..3 of a stage).
  constexpr bool PF2 = FM == 2;
  uint4 pa[NPF], pb[NPF], xa[NXF], xb[NXF], x2[NXF], x3[NXF];
  pread(0, 0, pa);
  xread(0, 0, 0, xa);
  if constexpr (PF2) xread(0, 0, 1, xb);

  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;

  // One stage st; J = st mod 4 (which fixes the register buffer of stage
  // st + 2, (st + 2) mod NRB).
  // FRESH marks the first stage of a group, LAST its last one (which folds).
  // Each k-step's fragments are read during the previous k-step's MFMAs; on
  // entry pa / xa hold the stage's first ones.  The body has no branches, so
  // that the compiler can interleave the LDS traffic, the unpacking and the
  // global loads with the MFMAs: past the last stage the stores fill a slot
  // that is never read again and the loads read zeros.
  // PH: st mod 3 when the caller knows it (three-slot ring), else -1.
  auto body = [&](auto JC, auto FC, auto LC, int st, auto PHC) __attribute__((always_inline)) {
    constexpr int J = decltype(JC)::value;
    constexpr int PH = decltype(PHC)::value;
    v4i(&rg)[NLD] = rgb[(J + 2) % C::NRB];
    uint32_t(&gq)[2] = gqb[(J + 2) % C::NRB];
    // ring slot of stage st + d (J = st mod 4): a compile-time constant with
    // four slots, or with three when the phase is known
    auto slot_of = [&](int d) __attribute__((always_inline)) {
      return C::NBUF == 4 ? ((J + d) & 3) : PH >= 0 ? (PH + d) % 3 : (st + d) % 3;
    };
    const int slot = slot_of(0);
    // Four k-steps.  Stage st + 2 goes into the slot read during stage
    // st - 2 (or st - 1 with three slots), its packed part during k-step 1
    // and its unpacked part during k-step 2, each after that k-step's
    // fragment reads (so that the reads do not queue behind the writes of
    // all waves); then its register buffer takes stage st + 2 + NRB.  The
    // scheduling barriers keep this order.
    using LO = std::false_type;
    using HI = std::true_type;
    if constexpr (STREAM) {  // the group parameters of stage st + 2 in, stage st + 2 + NRB out
      lstore_g(st + 2, gq);
      gload_g(st + 2 + C::NRB, gq);
    }
    if constexpr (PF2) {  // on entry pa, xa (k-step 0) and xb (k-step 1) are loaded
      pread(slot, 1, pb);
      xread(slot, 1, 0, x2);
      __builtin_amdgcn_sched_barrier(0);
      mma1(pa, xa, LO{}, FC);
      xread(slot, 1, 1, x3);
      lstore_p(slot_of(2), rg);
      __builtin_amdgcn_sched_barrier(0);
      mma1(pa, xb, HI{}, LO{});
      pread(slot_of(1), 0, pa);  // past the last stage: stale, unused
      xread(slot_of(1), 0, 0, xa);
      lstore_x(slot_of(2), rg);
      __builtin_amdgcn_sched_barrier(0);
      mma1(pb, x2, LO{}, LO{});
      xread(slot_of(1), 0, 1, xb);
      gload(st + 2 + C::NRB, rg);
      __builtin_amdgcn_sched_barrier(0);
      mma1(pb, x3, HI{}, LO{});
    } else {  // FM = 4 (one group); on entry pa, xa (k-step 0) are loaded
      xread(slot, 0, 1, xb);
      __builtin_amdgcn_sched_barrier(0);
      mma1(pa, xa, LO{}, FC);
      pread(slot, 1, pb);
      xread(slot, 1, 0, xa);
      lstore_p(slot_of(2), rg);
      __builtin_amdgcn_sched_barrier(0);
      mma1(pa, xb, HI{}, LO{});
      xread(slot, 1, 1, xb);
      lstore_x(slot_of(2), rg);
      __builtin_amdgcn_sched_barrier(0);
      mma1(pb, xa, LO{}, LO{});
      pread(slot_of(1), 0, pa);  // past the last stage: stale, unused
      xread(slot_of(1), 0, 0, xa);
      gload(st + 2 + C::NRB, rg);
      __builtin_amdgcn_sched_barrier(0);
      mma1(pb, xb, HI{}, LO{});
    }
    if constexpr (decltype(LC)::value) {  // the group's last stage
      const int b = st >> (log2g - 7);
      if constexpr (DBG) {
        dump(b);
      } else if constexpr (!SINGLE) {
        fold_group(b);
      }
    }
    lds_barrier();
  };
  // four stages from st (a multiple of 4); FIRST / LASTG: they start / end a group
  // (PHC: st mod 3, or -1 when not known at compile time)
  using PN = std::integral_constant<int, -1>;
  auto four = [&](int st, auto FIRST, auto LASTG, auto PHC) __attribute__((always_inline)) {
    using Fl = std::false_type;
    constexpr int P = decltype(PHC)::value;
    using P1 = std::integral_constant<int, P < 0 ? -1 : (P + 1) % 3>;
    using P2 = std::integral_constant<int, P < 0 ? -1 : (P + 2) % 3>;
    body(I0{}, FIRST, Fl{}, st, PHC);
    body(I1{}, Fl{}, Fl{}, st + 1, P1{});
    body(I2{}, Fl{}, Fl{}, st + 2, P2{});
    body(I3{}, Fl{}, LASTG, st + 3, PHC);
  };

  using T = std::true_type;
  using Fl = std::false_type;
  int st = 0;
  if constexpr (MODE == 1) {  // every stage is a group
    for (; st + 4 <= nst; st += 4) {
      body(I0{}, T{}, T{}, st, PN{});
      body(I1{}, T{}, T{}, st + 1, PN{});
      body(I2{}, T{}, T{}, st + 2, PN{});
      body(I3{}, T{}, T{}, st + 3, PN{});
    }
    if (st < nst) body(I0{}, T{}, T{}, st, PN{});
    if (st + 1 < nst) body(I1{}, T{}, T{}, st + 1, PN{});
    if (st + 2 < nst) body(I2{}, T{}, T{}, st + 2, PN{});
  } else if constexpr (MODE == 2) {  // groups of two stages
    for (; st + 4 <= nst; st += 4) {
      body(I0{}, T{}, Fl{}, st, PN{});
      body(I1{}, Fl{}, T{}, st + 1, PN{});
      body(I2{}, T{}, Fl{}, st + 2, PN{});
      body(I3{}, Fl{}, T{}, st + 3, PN{});
    }
    if (st < nst) {
      body(I0{}, T{}, Fl{}, st, PN{});
      body(I1{}, Fl{}, T{}, st + 1, PN{});
    }
  } else if constexpr (MODE == 4) {  // groups of four stages
    if constexpr (C::NBUF == 3) {
      // twelve stages per iteration, so that every stage's ring slot is known
      using Q0 = std::integral_constant<int, 0>;
      using Q1 = std::integral_constant<int, 1>;
      using Q2 = std::integral_constant<int, 2>;
      for (; st + 12 <= nst; st += 12) {
        four(st, T{}, T{}, Q0{});
        four(st + 4, T{}, T{}, Q1{});
        four(st + 8, T{}, T{}, Q2{});
      }
      if (st < nst) four(st, T{}, T{}, Q0{});
      if (st + 4 < nst) four(st + 4, T{}, T{}, Q1{});
    } else {
      for (; st < nst; st += 4) four(st, T{}, T{}, PN{});
    }
  } else {  // groups of 8k stages: first four, middle fours, last four
    for (; st < nst; st += 4) {
      four(st, T{}, Fl{}, PN{});
      for (st += 4; (st & (spg - 1)) != spg - 4; st += 4) four(st, Fl{}, Fl{}, PN{});
      four(st, Fl{}, T{}, PN{});
    }
  }
  if constexpr (SINGLE && !DBG) read_rs(0);
  if constexpr (DBG) return;

  // ---- finish one fragment row at a time ----------------------------------
  // zero-point correction F += sum_b (-s z)[m, b] * colsum[b, n] (fp32 MFMAs
  // with k = group: lane half h supplies group 2 kk + h), then Y = sw * F as
  // bf16 into a private LDS area per wave: rows of 16 8-byte units, unit u of
  // row r stored at u ^ (r & 15).  (With one group the fold happens here.)
  uint32_t* ot = reinterpret_cast<uint32_t*>(ring) + wave * (C::WROWS * 32);
  const bool vec = (tm + C::BM <= M) && (tn + C::BN <= N) && (ldy % 8 == 0) &&
                   ((reinterpret_cast<uintptr_t>(Y) & 15) == 0);
  float sw[2][4][4];
#pragma unroll
  for (int fn = 0; fn < 2; ++fn)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 v = *reinterpret_cast<const float4*>(&sSW[wn * 64 + fn * 32 + q * 8 + h * 4]);
      sw[fn][q][0] = v.x;
      sw[fn][q][1] = v.y;
      sw[fn][q][2] = v.z;
      sw[fn][q][3] = v.w;
    }
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    if constexpr (SINGLE) fold_row(fm);
    const int r = wm * C::WROWS + fm * 32 + fr;
    for (int kk = 0; kk < (STREAM ? 0 : (G + 1) / 2); ++kk) {  // (STREAM: applied per pair)
      const int b = 2 * kk + h;
      const bool ok = b < G;
      const float szv = ok ? -16.0f * sRS[b][r] * (float)sZ[b][r] : 0.0f;
#pragma unroll
      for (int fn = 0; fn < 2; ++fn) {
        const float csv = ok ? sCS[b][wn * 64 + fn * 32 + fr] : 0.0f;
        F[fm][fn] = __builtin_amdgcn_mfma_f32_32x32x2f32(csv, szv, F[fm][fn], 0, 0, 0);
      }
    }
    const int lr = fm * 32 + fr;  // row within the wave's tile
#pragma unroll
    for (int fn = 0; fn < 2; ++fn)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int u = fn * 8 + q * 2 + h;
        const v16f& f = F[fm][fn];
        *reinterpret_cast<uint2*>(ot + lr * 32 + ((u ^ (lr & 15)) * 2)) =
            make_uint2(bf16x2_rne(sw[fn][q][0] * f[q * 4 + 0], sw[fn][q][1] * f[q * 4 + 1]),
                       bf16x2_rne(sw[fn][q][2] * f[q * 4 + 2], sw[fn][q][3] * f[q * 4 + 3]));
      }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
  // lane l of pass p: row 8p + l/8, 16-byte piece l%8 (units 2k, 2k+1)
#pragma unroll 4
  for (int p = 0; p < C::WROWS / 8; ++p) {
    const int r = 8 * p + (lane >> 3);
    const int k = lane & 7;
    const int pu = (2 * k) ^ (r & 15);
    uint4 d = *reinterpret_cast<const uint4*>(ot + r * 32 + (pu & ~1) * 2);
    if (pu & 1) d = make_uint4(d.z, d.w, d.x, d.y);
    const int row = tm + wm * C::WROWS + r;
    const int col = tn + wn * 64 + 8 * k;
    if (vec) {
      // write-once output: a non-temporal store (measured 1-4 % faster than
      // a cached one across the prefill shapes)
      const gemm_u32x4 dv = {d.x, d.y, d.z, d.w};
      __builtin_nontemporal_store(dv, reinterpret_cast<gemm_u32x4*>(Y + (int64_t)row * ldy + col));
    } else if (row < M) {
      const uint32_t w4[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (col + e < N) Y[(int64_t)row * ldy + col + e] = (uint16_t)(w4[e >> 1] >> (16 * (e & 1)));
    }
  }
}

}  // namespace

bool gemm_grouped_supported(int64_t M, int64_t N, int64_t K, int log2g) {
  // stages of 128 k never straddle a group; buffer offsets (codes, and the
  // streamed group parameters) are 32-bit
  const int64_t G = K >> log2g;
  return log2g >= 7 && K % 128 == 0 && M * (K / 2) < (int64_t(1) << 31) &&
         N * (K / 2) < (int64_t(1) << 31) && G * N * 4 < (int64_t(1) << 31) &&
         256 * G * 2 < (int64_t(1) << 31);
}

template <int FM, bool ONEG, bool STREAM = false>
hipError_t launch_g(const uint8_t* a_codes, const uint16_t* a_scale, const int16_t* a_zero,
                    const uint8_t* w_codes, const uint16_t* w_scale, const int32_t* w_colsum,
                    int64_t M, int64_t N, int64_t K, int log2g, uint16_t* y, int64_t ldy,
                    int32_t* acc_debug, hipStream_t stream) {
  using C = GCfg<FM, ONEG, STREAM>;
  const int64_t tiles = ((M + C::BM - 1) / C::BM) * ((N + C::BN - 1) / C::BN);
  const dim3 grid((unsigned)tiles), block(C::THREADS);
#define OFFQ_GG(D, MD)                                                                        \
  hipLaunchKernelGGL((w4a4_gemm_grouped_kernel<D, MD, FM, ONEG, STREAM>), grid, block, 0, stream, a_codes,  \
                     a_scale, a_zero, w_codes, w_scale, w_colsum, (int)M, (int)N, (int)K, log2g, \
                     y, ldy, acc_debug)
#define OFFQ_GG_M(D)                                                                 \
  if (log2g == 7) OFFQ_GG(D, 1); else if (log2g == 8) OFFQ_GG(D, 2);                \
  else if (log2g == 9) OFFQ_GG(D, 4); else OFFQ_GG(D, 8);
  // A debug request runs an accumulator-only pass, then the regular kernel.
  if (acc_debug) { OFFQ_GG_M(true) }
  OFFQ_GG_M(false)
#undef OFFQ_GG_M
#undef OFFQ_GG
  return hipGetLastError();
}

hipError_t launch_w4a4_gemm_grouped(const uint8_t* a_codes, const uint16_t* a_scale,
                                    const int16_t* a_zero, const uint8_t* w_codes,
                                    const uint16_t* w_scale, const int32_t* w_colsum, int64_t M,
                                    int64_t N, int64_t K, int log2g, uint16_t* y, int64_t ldy,
                                    int32_t* acc_debug, hipStream_t stream) {
  // one group per row and enough 256 x 256 tiles to fill the chip: the wider
  // wave tiles
  const bool wide = (K >> log2g) == 1 && ((M + 255) / 256) * ((N + 255) / 256) >= 384;
  if (wide)
    return launch_g<4, true>(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K, log2g,
                             y, ldy, acc_debug, stream);
  if ((K >> log2g) == 1)
    return launch_g<2, true>(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K, log2g,
                             y, ldy, acc_debug, stream);
  // several groups: the parameters of up to 28 groups sit in LDS for the whole
  // tile; more groups stream theirs with the stages
  if ((K >> log2g) > GCfg<2, false>::GMAX)
    return launch_g<2, false, true>(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K,
                                    log2g, y, ldy, acc_debug, stream);
  return launch_g<2, false>(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K, log2g,
                            y, ldy, acc_debug, stream);
}

}  // namespace offq
