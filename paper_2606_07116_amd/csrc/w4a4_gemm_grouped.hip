// W4A4 GEMM for several quantization groups per row (g < K): the case of a
// block-diagonal online rotation, e.g. the MLP down projection with 28 groups
// of 512 channels.  gfx950, v_mfma_i32_32x32x32_i8.
//
//   acc_b[m,n] = sum_{k in group b} q_a[m,k] q_w[n,k]                 (int32)
//   Y[m,n]     = sw[n] * sum_b s[m,b] * (acc_b[m,n] - z[m,b] * colsum[b,n])
//
// (the dequantised product of Eq. 1 with one scale/zero-point per row and
// group; the z * colsum terms carry the absorbed offsets).
//
// Organisation
// * 8 waves per workgroup (two per SIMD) in a 4 x 2 arrangement, each owning
//   64 tokens x 64 output channels (2 x 2 MFMA tiles of 32 x 32): 64 int32
//   accumulators for the current group and 64 fp32 running sums F; workgroup
//   tile 256 x 128.  While one wave of a SIMD folds, the other multiplies.
// * Stages of 128 k go from global memory straight into a 4-deep LDS ring
//   (buffer loads with the LDS destination, 3 stages ahead; rows past the end
//   read as zero), so no registers hold staged data.  One barrier per stage,
//   preceded by a wait for the stage two ahead only.  The stage loop is
//   unrolled by the ring depth, which makes the ring offsets of every LDS
//   access compile-time constants.
// * Fragment reads, unpacking and the transposed MFMA are those of the
//   one-group kernel.
// * At the end of each group (g / 128 stages) the accumulators are folded
//   into the running sums, F += (s / 16) * acc in fp32 (s / 16 undoes the 16x
//   widening of the weight codes), and the first MFMA of the next group starts
//   from a zero accumulator.  The row scales, zero-points and column sums of
//   the tile's groups are loaded into LDS once, in the prologue.
// * After the last group the zero-point terms are added with one fp32 MFMA
//   per pair of groups: F += sum_b (-s z)[m, b] * colsum[b, n].
// * Epilogue: Y = sw * F -> bf16 through LDS for 16-byte coalesced stores.
#include <type_traits>

#include "common.h"
#include "gemm_common.h"
#include "internal.h"

namespace offq {
namespace {

using namespace gemm;

// FM: 32-row MFMA tiles per wave along the tokens.  FM = 2: 8 waves of
// 64 x 64 in a 4 x 2 arrangement (workgroup tile 256 x 128), any number of
// groups up to GMAX; FM = 4: 8 waves of 128 x 64 in a 2 x 4 arrangement
// (256 x 256), one group per row only (no registers for running sums).
template <int FM>
struct GCfg {
  static constexpr int THREADS = 512;              // 8 waves, 2 per SIMD
  static constexpr int WAVES_M = FM == 2 ? 4 : 2;
  static constexpr int WROWS = 32 * FM;            // token rows per wave
  static constexpr int BM = WAVES_M * WROWS;       // 256
  static constexpr int BN = (8 / WAVES_M) * 64;    // 128 or 256
  static constexpr int NC = 4;                     // 16-byte chunks per row and stage
  static constexpr int A_SLOTS = BM * NC;
  static constexpr int B_SLOTS = BN * NC;
  static constexpr int STAGE_SLOTS = A_SLOTS + B_SLOTS;
  static constexpr int A_LD = A_SLOTS / THREADS;   // loads per thread and stage
  static constexpr int B_LD = B_SLOTS / THREADS;
  static constexpr int KSTAGE = 128;               // k per stage
  static constexpr int NBUF = 4;                   // LDS ring depth
  static constexpr int GMAX = FM == 2 ? 28 : 1;    // groups whose parameters fit in LDS
};

// s_waitcnt with only the vector-memory counter bounded (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// 16 bytes per lane from a buffer straight into LDS: lane l writes bytes
// [lds + 16 l, lds + 16 l + 16) (lds is the wave-uniform LDS byte address).
// Issued as inline assembly, so the compiler neither tracks these writes nor
// inserts waits for them: the ring's own vmcnt waits and barriers order them.
__device__ __forceinline__ void buffer_to_lds16(__amdgpu_buffer_rsrc_t rsrc, uint32_t lds,
                                                int voff, int soff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :: "s"(lds), "v"(voff), "s"(rsrc), "s"(soff) : "memory", "m0");
}

// Workgroup barrier for the ring: waits for the wave's own LDS operations,
// synchronises, and is a compiler-level memory barrier.  The buffer-to-LDS
// loads a stage needs are waited for with wait_vmcnt before it.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

typedef float v16f __attribute__((ext_vector_type(16)));

// MODE: stages per group: 1, 2, 4, or a multiple of 8 (MODE 8).
template <bool DBG, int MODE, int FM>
__global__ __launch_bounds__(512) void w4a4_gemm_grouped_kernel(
    const uint8_t* __restrict__ A, const uint16_t* __restrict__ a_scale,
    const int16_t* __restrict__ a_zero, const uint8_t* __restrict__ W,
    const uint16_t* __restrict__ w_scale, const int32_t* __restrict__ w_colsum, int M, int N,
    int K, int log2g, uint16_t* __restrict__ Y, int64_t ldy, int32_t* __restrict__ acc_dbg) {
  using C = GCfg<FM>;
  __shared__ uint4 ring[C::NBUF * C::STAGE_SLOTS];
  // per group b: s / 16 and z of the tile's rows, colsum of its columns
  __shared__ float sRS[C::GMAX][C::BM];
  __shared__ short sZ[C::GMAX][C::BM];
  __shared__ float sCS[C::GMAX][C::BN];

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

  constexpr int RSTEP = C::THREADS / C::NC;
  const int row0 = tid / C::NC;
  const int chunk = swz<C::NC>(row0, tid % C::NC);
  const __amdgpu_buffer_rsrc_t arsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(A + (int64_t)tm * ldk), 0, (int)((int64_t)(M - tm) * ldk), 0x00020000);
  const __amdgpu_buffer_rsrc_t brsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(W + (int64_t)tn * ldk), 0, (int)((int64_t)(N - tn) * ldk), 0x00020000);
  const int voff = row0 * (int)ldk + chunk * 16;
  const int vstep = RSTEP * (int)ldk;
  const uint32_t ring_lds = lds_addr(ring) + wave * 64 * 16;

  // stage st into ring buffer J: this thread's slots tid + 512 i, written by
  // each wave as 64 consecutive 16-byte slots per load
  auto dma = [&](int J, int st) __attribute__((always_inline)) {
    const uint32_t base = ring_lds + J * (C::STAGE_SLOTS * 16);
    const int soff = st * (C::KSTAGE / 2);
#pragma unroll
    for (int i = 0; i < C::A_LD; ++i)
      buffer_to_lds16(arsrc, base + i * C::THREADS * 16, voff + i * vstep, soff);
#pragma unroll
    for (int i = 0; i < C::B_LD; ++i)
      buffer_to_lds16(brsrc, base + (C::A_SLOTS + i * C::THREADS) * 16, voff + i * vstep, soff);
  };
  // this lane's fragment slots for chunk column 2h + jj; fragments f are 32
  // rows apart, which keeps the swizzle
  const uint4* a_frag0 = ring + (wm * C::WROWS + fr) * C::NC + swz<C::NC>(fr, 2 * h);
  const uint4* a_frag1 = ring + (wm * C::WROWS + fr) * C::NC + swz<C::NC>(fr, 2 * h + 1);
  const uint4* b_frag0 = ring + C::A_SLOTS + (wn * 64 + fr) * C::NC + swz<C::NC>(fr, 2 * h);
  const uint4* b_frag1 = ring + C::A_SLOTS + (wn * 64 + fr) * C::NC + swz<C::NC>(fr, 2 * h + 1);
  auto fread = [&](auto JC, int jj, uint4* pa, uint4* pb) __attribute__((always_inline)) {
    constexpr int J = decltype(JC)::value;
    const uint4* As = (jj ? a_frag1 : a_frag0) + J * C::STAGE_SLOTS;
    const uint4* Bs = (jj ? b_frag1 : b_frag0) + J * C::STAGE_SLOTS;
#pragma unroll
    for (int f = 0; f < FM; ++f) pa[f] = As[f * 32 * C::NC];
#pragma unroll
    for (int f = 0; f < 2; ++f) pb[f] = Bs[f * 32 * C::NC];
  };

  // With one group per row (the only case of FM = 4) F is first written by
  // the single fold after the loop, so it takes no registers during it.
  constexpr bool SINGLE = C::GMAX == 1;
  v16i acc[FM][2];
  v16f F[FM][2];
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      acc[a][b] = v16i{};
      if constexpr (!SINGLE) F[a][b] = v16f{};
    }

  // Lane column fr of fragment fm is token row wm*64 + fm*32 + fr; register
  // i of fragment (fm, fn) is output channel wn*64 + fn*32 + 8*(i/4) + 4*h + i%4.
  // F += (s / 16) * acc for fragment row fm (s / 16 undoes the 16x widening
  // of the weight codes), with rs[fm] = s / 16 of the finished group.
  float rs[FM] = {};
  auto read_rs = [&](int b) __attribute__((always_inline)) {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) rs[fm] = sRS[b][wm * C::WROWS + fm * 32 + fr];
  };
  auto fold_row = [&](int fm) __attribute__((always_inline)) {
#pragma unroll
    for (int fn = 0; fn < 2; ++fn)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        F[fm][fn][i] = SINGLE ? rs[fm] * (float)acc[fm][fn][i]
                              : __builtin_fmaf(rs[fm], (float)acc[fm][fn][i], F[fm][fn][i]);
  };
  // two k-steps (low and high nibbles of one 16-byte chunk per fragment);
  // FRESH: the low-nibble MFMAs start the accumulators from zero.  Operands
  // are unpacked just before use to keep the live registers down.
  auto mma2 = [&](const uint4* pa, const uint4* pb, auto FC) __attribute__((always_inline)) {
    constexpr bool FRESH = decltype(FC)::value;
    const v4i ub0 = wgt_lo16(pb[0]), ub1 = wgt_lo16(pb[1]);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const v4i ua = act_lo(pa[fm]);
      acc[fm][0] = __builtin_amdgcn_mfma_i32_32x32x32_i8(ub0, ua, FRESH ? v16i{} : acc[fm][0], 0, 0, 0);
      acc[fm][1] = __builtin_amdgcn_mfma_i32_32x32x32_i8(ub1, ua, FRESH ? v16i{} : acc[fm][1], 0, 0, 0);
    }
    const v4i nb0 = wgt_hi16(pb[0]), nb1 = wgt_hi16(pb[1]);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const v4i na = act_hi(pa[fm]);
      acc[fm][0] = __builtin_amdgcn_mfma_i32_32x32x32_i8(nb0, na, acc[fm][0], 0, 0, 0);
      acc[fm][1] = __builtin_amdgcn_mfma_i32_32x32x32_i8(nb1, na, acc[fm][1], 0, 0, 0);
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

  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;

  // prologue: stages 0, 1, 2 in flight to the ring; the group parameters of
  // the tile into LDS meanwhile
  dma(0, 0);
  if (nst > 1) dma(1, 1);
  if (nst > 2) dma(2, 2);
  {
    // Row parameters of the tile: a contiguous block of 256 * G entries of the
    // [M, G] arrays, read coalesced (entry e = tid + 512 p is row e / G, group
    // e % G); column sums: group b, column c = colsum[b * N + tn + c].  All
    // loads are issued before the first LDS write.
    const float inv_g = 1.0f / (float)G;
    const int64_t base = (int64_t)tm * G;
    const int nrow_e = min(C::BM, M - tm) * G;  // valid entries of the block
    constexpr int PE = (C::GMAX * C::BM + C::THREADS - 1) / C::THREADS;  // row entries per thread
    constexpr int PC = (C::GMAX * C::BN + C::THREADS - 1) / C::THREADS;  // column entries per thread
    uint16_t sv[PE];
    int16_t zv[PE];
#pragma unroll
    for (int p = 0; p < PE; ++p) {
      const int e = tid + C::THREADS * p;
      const bool ok = e < C::BM * G && e < nrow_e;
      sv[p] = ok ? a_scale[base + e] : (uint16_t)0;
      zv[p] = ok ? a_zero[base + e] : (int16_t)0;
    }
    float cv[PC];
#pragma unroll
    for (int p = 0; p < PC; ++p) {
      const int b = (C::THREADS / C::BN) * p + tid / C::BN, c = tid % C::BN;
      cv[p] = (b < G && b < C::GMAX && tn + c < N) ? (float)w_colsum[(int64_t)b * N + tn + c] : 0.0f;
    }
#pragma unroll
    for (int p = 0; p < PE; ++p) {
      const int e = tid + C::THREADS * p;
      if (e < C::BM * G) {
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
      if (b < G && b < C::GMAX) sCS[b][tid % C::BN] = cv[p];
    }
  }
  // stages 0 and 1 landed (stage 2 may still be in flight)
  if (nst > 2) wait_vmcnt<C::A_LD + C::B_LD>();
  else wait_vmcnt<0>();
  ring_barrier();
  uint4 pc_a[4], pc_b[2];
  fread(I0{}, 0, pc_a, pc_b);

  // One stage st on ring buffer J = st % 4; FRESH marks the first stage of a
  // group, whose last stage folds the accumulators.
  auto body = [&](auto JC, auto FC, int st) __attribute__((always_inline)) {
    constexpr int J = decltype(JC)::value;
    using NEXT = std::integral_constant<int, (J + 1) % 4>;
    const bool ahead = st + 3 < nst;
    if (ahead) dma((J + 3) % 4, st + 3);
    uint4 p1_a[4], p1_b[2];
    fread(JC, 1, p1_a, p1_b);
    mma2(pc_a, pc_b, FC);
    fread(NEXT{}, 0, pc_a, pc_b);  // past the last stage: stale, unused
    mma2(p1_a, p1_b, std::false_type{});
    if ((st & (spg - 1)) == spg - 1) {  // the group's last stage
      const int b = st >> (log2g - 7);
      if constexpr (DBG) {
        dump(b);
      } else {
        read_rs(b);
        if constexpr (!SINGLE) {
#pragma unroll
          for (int fm = 0; fm < FM; ++fm) fold_row(fm);
        }
      }
    }
    // stage st + 2 has landed; stage st + 3 may still be in flight
    if (ahead) wait_vmcnt<C::A_LD + C::B_LD>();
    else wait_vmcnt<0>();
    ring_barrier();
  };

  using T = std::true_type;
  using Fl = std::false_type;
  int st = 0;
  if constexpr (MODE == 1) {  // every stage starts a group
    for (; st + 4 <= nst; st += 4) {
      body(I0{}, T{}, st);
      body(I1{}, T{}, st + 1);
      body(I2{}, T{}, st + 2);
      body(I3{}, T{}, st + 3);
    }
    if (st < nst) body(I0{}, T{}, st);
    if (st + 1 < nst) body(I1{}, T{}, st + 1);
    if (st + 2 < nst) body(I2{}, T{}, st + 2);
  } else if constexpr (MODE == 2) {  // groups of two stages
    for (; st + 4 <= nst; st += 4) {
      body(I0{}, T{}, st);
      body(I1{}, Fl{}, st + 1);
      body(I2{}, T{}, st + 2);
      body(I3{}, Fl{}, st + 3);
    }
    if (st < nst) {
      body(I0{}, T{}, st);
      body(I1{}, Fl{}, st + 1);
    }
  } else if constexpr (MODE == 4) {  // groups of four stages
    for (; st < nst; st += 4) {
      body(I0{}, T{}, st);
      body(I1{}, Fl{}, st + 1);
      body(I2{}, Fl{}, st + 2);
      body(I3{}, Fl{}, st + 3);
    }
  } else {  // groups of 8k stages
    for (; st < nst; st += 8) {
      if ((st & (spg - 1)) == 0) body(I0{}, T{}, st);
      else body(I0{}, Fl{}, st);
      body(I1{}, Fl{}, st + 1);
      body(I2{}, Fl{}, st + 2);
      body(I3{}, Fl{}, st + 3);
      body(I0{}, Fl{}, st + 4);
      body(I1{}, Fl{}, st + 5);
      body(I2{}, Fl{}, st + 6);
      body(I3{}, Fl{}, st + 7);
    }
  }
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
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = tn + wn * 64 + fn * 32 + q * 8 + h * 4 + e;
        sw[fn][q][e] = c < N ? fp16_bits_to_f32(w_scale[c]) : 0.0f;
      }
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    if constexpr (SINGLE) fold_row(fm);
    const int r = wm * C::WROWS + fm * 32 + fr;
    for (int kk = 0; kk < (G + 1) / 2; ++kk) {
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
      *reinterpret_cast<uint4*>(Y + (int64_t)row * ldy + col) = d;
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
  // stages of 128 k never straddle a group; the group parameters of a tile
  // fit in LDS; buffer offsets are 32-bit
  return log2g >= 7 && K % 128 == 0 && (K >> log2g) <= GCfg<2>::GMAX &&
         M * (K / 2) < (int64_t(1) << 31) && N * (K / 2) < (int64_t(1) << 31);
}

template <int FM>
hipError_t launch_g(const uint8_t* a_codes, const uint16_t* a_scale, const int16_t* a_zero,
                    const uint8_t* w_codes, const uint16_t* w_scale, const int32_t* w_colsum,
                    int64_t M, int64_t N, int64_t K, int log2g, uint16_t* y, int64_t ldy,
                    int32_t* acc_debug, hipStream_t stream) {
  using C = GCfg<FM>;
  const int64_t tiles = ((M + C::BM - 1) / C::BM) * ((N + C::BN - 1) / C::BN);
  const dim3 grid((unsigned)tiles), block(C::THREADS);
#define OFFQ_GG(D, MD)                                                                        \
  hipLaunchKernelGGL((w4a4_gemm_grouped_kernel<D, MD, FM>), grid, block, 0, stream, a_codes,  \
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
    return launch_g<4>(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K, log2g, y,
                       ldy, acc_debug, stream);
  return launch_g<2>(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K, log2g, y,
                     ldy, acc_debug, stream);
}

}  // namespace offq
