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
// * 4 waves per workgroup in a 2 x 2 arrangement, each owning 128 tokens x 64
//   output channels (4 x 2 MFMA tiles of 32 x 32): 128 int32 accumulators for
//   the current group and 128 fp32 running sums; workgroup tile 256 x 128.
// * Operand staging, fragment reads, unpacking and the transposed MFMA are
//   those of the one-group kernel: stages of 128 k through a 3-deep LDS ring,
//   one LDS-only barrier per stage.
// * At the end of each group (g / 128 stages) every accumulator is folded into
//   its running sum, F += (s / 16) * acc + (-s z) * colsum, in fp32, and the
//   first MFMA of the next group starts from a zero accumulator.  The row
//   parameters (s / 16, -s z) and the column sums of a group are staged in LDS
//   one group ahead (double buffered).
// * Epilogue: Y = sw * F -> bf16 through LDS for 16-byte coalesced stores.
#include <type_traits>

#include "common.h"
#include "gemm_common.h"
#include "internal.h"

namespace offq {
namespace {

using namespace gemm;

struct GCfg {
  static constexpr int BM = 256;
  static constexpr int BN = 128;
  static constexpr int NC = 4;                     // 16-byte chunks per row and stage
  static constexpr int A_SLOTS = BM * NC;
  static constexpr int B_SLOTS = BN * NC;
  static constexpr int STAGE_SLOTS = A_SLOTS + B_SLOTS;
  static constexpr int A_LD = A_SLOTS / 256;       // loads per thread and stage
  static constexpr int B_LD = B_SLOTS / 256;
  static constexpr int KSTAGE = 128;               // k per stage
  static constexpr int NBUF = 3;                   // LDS ring depth
};

template <bool DBG>
__global__ __launch_bounds__(256) void w4a4_gemm_grouped_kernel(
    const uint8_t* __restrict__ A, const uint16_t* __restrict__ a_scale,
    const int16_t* __restrict__ a_zero, const uint8_t* __restrict__ W,
    const uint16_t* __restrict__ w_scale, const int32_t* __restrict__ w_colsum, int M, int N,
    int K, int log2g, uint16_t* __restrict__ Y, int64_t ldy, int32_t* __restrict__ acc_dbg) {
  using C = GCfg;
  __shared__ uint4 lds[C::NBUF * C::STAGE_SLOTS];
  __shared__ __attribute__((aligned(16))) float2 sRP[2][C::BM];  // (s / 16, -s z) per row
  __shared__ __attribute__((aligned(16))) float sCS[2][C::BN];   // colsum per column

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 5, fr = lane & 31;
  const int wm = wave & 1, wn = wave >> 1;

  const int tiles_m = (M + C::BM - 1) / C::BM;
  const int tiles_n = (N + C::BN - 1) / C::BN;
  int ti, tj;
  tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n, ti, tj);
  const int tm = ti * C::BM, tn = tj * C::BN;
  const int64_t ldk = K >> 1;
  const int nst = K / C::KSTAGE;
  const int G = K >> log2g;
  const int spg = 1 << (log2g - 7);  // stages per group

  // ---- per-group parameters, staged one group ahead ----------------------
  float p_s = 0.0f, p_z = 0.0f, p_c = 0.0f;
  auto param_load = [&](int b) {
    const int row = tm + tid;
    if (row < M) {
      p_s = fp16_bits_to_f32(a_scale[(int64_t)row * G + b]);
      p_z = (float)a_zero[(int64_t)row * G + b];
    } else {
      p_s = 0.0f;
      p_z = 0.0f;
    }
    if (tid < C::BN) {
      const int col = tn + tid;
      p_c = col < N ? (float)w_colsum[(int64_t)b * N + col] : 0.0f;
    }
  };
  auto param_store = [&](int b) {
    // s / 16 undoes the 16x widening of the weight codes (exact)
    sRP[b & 1][tid] = make_float2(p_s * 0.0625f, -(p_s * p_z));
    if (tid < C::BN) sCS[b & 1][tid] = p_c;
  };

  constexpr int RSTEP = 256 / C::NC;
  const int row0 = tid / C::NC;
  const int chunk = swz<C::NC>(row0, tid % C::NC);
  const __amdgpu_buffer_rsrc_t arsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(A + (int64_t)tm * ldk), 0, (int)((int64_t)(M - tm) * ldk), 0x00020000);
  const __amdgpu_buffer_rsrc_t brsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(W + (int64_t)tn * ldk), 0, (int)((int64_t)(N - tn) * ldk), 0x00020000);
  const int voff = row0 * (int)ldk + chunk * 16;
  const int vstep = RSTEP * (int)ldk;

  v4i ra[C::A_LD], rb[C::B_LD];
  auto gload = [&](int st) {
    const int soff = st * (C::KSTAGE / 2);
#pragma unroll
    for (int i = 0; i < C::A_LD; ++i)
      ra[i] = __builtin_amdgcn_raw_buffer_load_b128(arsrc, voff + i * vstep, soff, 0);
#pragma unroll
    for (int i = 0; i < C::B_LD; ++i)
      rb[i] = __builtin_amdgcn_raw_buffer_load_b128(brsrc, voff + i * vstep, soff, 0);
  };
  auto lstore = [&](int buf) {
    v4i* base = reinterpret_cast<v4i*>(lds + buf * C::STAGE_SLOTS);
#pragma unroll
    for (int i = 0; i < C::A_LD; ++i) base[tid + 256 * i] = ra[i];
#pragma unroll
    for (int i = 0; i < C::B_LD; ++i) base[C::A_SLOTS + tid + 256 * i] = rb[i];
  };
  auto fread = [&](int buf, int jj, uint4* pa, uint4* pb) {
    const uint4* As = lds + buf * C::STAGE_SLOTS;
    const uint4* Bs = As + C::A_SLOTS;
    const int c = 2 * h + jj;
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      const int r = wm * 128 + f * 32 + fr;
      pa[f] = As[r * C::NC + swz<C::NC>(r, c)];
    }
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      const int r = wn * 64 + f * 32 + fr;
      pb[f] = Bs[r * C::NC + swz<C::NC>(r, c)];
    }
  };

  v16i acc[4][2];
  float F[4][2][16];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      acc[a][b] = v16i{};
#pragma unroll
      for (int i = 0; i < 16; ++i) F[a][b][i] = 0.0f;
    }

  // two k-steps (low and high nibbles of one 16-byte chunk per fragment);
  // FRESH: the low-nibble MFMAs start the accumulators from zero
  auto mma2 = [&](const uint4* pa, const uint4* pb, auto FC) {
    constexpr bool FRESH = decltype(FC)::value;
    v4i ua[4], ub[2];
#pragma unroll
    for (int f = 0; f < 4; ++f) ua[f] = act_lo(pa[f]);
#pragma unroll
    for (int f = 0; f < 2; ++f) ub[f] = wgt_lo16(pb[f]);
    v4i na[4], nb[2];
#pragma unroll
    for (int f = 0; f < 4; ++f) na[f] = act_hi(pa[f]);
#pragma unroll
    for (int f = 0; f < 2; ++f) nb[f] = wgt_hi16(pb[f]);
#pragma unroll
    for (int fm = 0; fm < 4; ++fm)
#pragma unroll
      for (int fn = 0; fn < 2; ++fn)
        acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(ub[fn], ua[fm],
                                                            FRESH ? v16i{} : acc[fm][fn], 0, 0, 0);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
    }
#pragma unroll
    for (int fm = 0; fm < 4; ++fm)
#pragma unroll
      for (int fn = 0; fn < 2; ++fn)
        acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(nb[fn], na[fm], acc[fm][fn], 0, 0, 0);
  };

  // Lane column fr of fragment fm is token row wm*128 + fm*32 + fr; register
  // i of fragment (fn) is output channel wn*64 + fn*32 + 8*(i/4) + 4*h + i%4.
  auto fold = [&](int b) {
    float2 rp[4];
#pragma unroll
    for (int fm = 0; fm < 4; ++fm) rp[fm] = sRP[b & 1][wm * 128 + fm * 32 + fr];
#pragma unroll
    for (int fn = 0; fn < 2; ++fn)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 c4 =
            *reinterpret_cast<const float4*>(&sCS[b & 1][wn * 64 + fn * 32 + q * 8 + h * 4]);
        const float cs[4] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
        for (int fm = 0; fm < 4; ++fm)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float& f = F[fm][fn][q * 4 + e];
            f = __builtin_fmaf(rp[fm].x, (float)acc[fm][fn][q * 4 + e], f);
            f = __builtin_fmaf(rp[fm].y, cs[e], f);
          }
      }
  };
  auto dump = [&](int b) {  // debug: the raw accumulators of group b
#pragma unroll
    for (int fm = 0; fm < 4; ++fm) {
      const int row = tm + wm * 128 + fm * 32 + fr;
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

  // prologue: parameters of group 0, stages 0 and 1 into the ring, stage 2
  // into registers
  param_load(0);
  param_store(0);
  gload(0);
  lstore(0);
  if (nst > 1) {
    gload(1);
    lstore(1);
  }
  if (nst > 2) gload(2);
  lds_barrier();
  uint4 pc_a[4], pc_b[2];
  fread(0, 0, pc_a, pc_b);

  for (int st = 0; st < nst; ++st) {
    const int buf = st % C::NBUF;
    const int b = st >> (log2g - 7);
    const bool first = (st & (spg - 1)) == 0;
    const bool last = (st & (spg - 1)) == spg - 1;
    if (st + 2 < nst) lstore((st + 2) % C::NBUF);
    // the next group's parameters: loaded before the stage prefetch so that
    // writing them to LDS does not wait for it
    const bool stage_next = first && b + 1 < G;
    if (stage_next) param_load(b + 1);
    if (st + 3 < nst) gload(st + 3);
    uint4 p1_a[4], p1_b[2];
    fread(buf, 1, p1_a, p1_b);
    if (first) mma2(pc_a, pc_b, std::true_type{});
    else mma2(pc_a, pc_b, std::false_type{});
    if (st + 1 < nst) fread((st + 1) % C::NBUF, 0, pc_a, pc_b);
    mma2(p1_a, p1_b, std::false_type{});
    if (stage_next) param_store(b + 1);
    if (last) {
      if constexpr (DBG) dump(b);
      else fold(b);
    }
    lds_barrier();
  }
  if constexpr (DBG) return;

  // ---- epilogue: Y = sw * F -> bf16 ---------------------------------------
  // Each wave writes its 128 x 64 bf16 tile to a private 16 KB LDS area (rows
  // of 16 8-byte units, unit u of row r stored at u ^ (r & 15)), then reads
  // 16-byte pieces back row by row: each store instruction covers 8 rows of
  // 128 contiguous bytes.
  uint32_t* ot = reinterpret_cast<uint32_t*>(lds) + wave * (128 * 32);
  const bool vec = (tm + C::BM <= M) && (tn + C::BN <= N) && (ldy % 8 == 0) &&
                   ((reinterpret_cast<uintptr_t>(Y) & 15) == 0);
#pragma unroll
  for (int fn = 0; fn < 2; ++fn)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int lc = tn + wn * 64 + fn * 32 + q * 8 + h * 4;
      float sw[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) sw[e] = lc + e < N ? fp16_bits_to_f32(w_scale[lc + e]) : 0.0f;
      const int u = fn * 8 + q * 2 + h;
#pragma unroll
      for (int fm = 0; fm < 4; ++fm) {
        const int r = fm * 32 + fr;
        const float* f = &F[fm][fn][q * 4];
        *reinterpret_cast<uint2*>(ot + r * 32 + ((u ^ (r & 15)) * 2)) =
            make_uint2(bf16x2_rne(sw[0] * f[0], sw[1] * f[1]), bf16x2_rne(sw[2] * f[2], sw[3] * f[3]));
      }
    }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
  // lane l of pass p: row 8p + l/8, 16-byte piece l%8 (units 2k, 2k+1)
#pragma unroll 4
  for (int p = 0; p < 16; ++p) {
    const int r = 8 * p + (lane >> 3);
    const int k = lane & 7;
    const int pu = (2 * k) ^ (r & 15);
    uint4 d = *reinterpret_cast<const uint4*>(ot + r * 32 + (pu & ~1) * 2);
    if (pu & 1) d = make_uint4(d.z, d.w, d.x, d.y);
    const int row = tm + wm * 128 + r;
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
  // stages of 128 k never straddle a group; buffer offsets are 32-bit
  return log2g >= 7 && K % 128 == 0 && M * (K / 2) < (int64_t(1) << 31) &&
         N * (K / 2) < (int64_t(1) << 31);
}

hipError_t launch_w4a4_gemm_grouped(const uint8_t* a_codes, const uint16_t* a_scale,
                                    const int16_t* a_zero, const uint8_t* w_codes,
                                    const uint16_t* w_scale, const int32_t* w_colsum, int64_t M,
                                    int64_t N, int64_t K, int log2g, uint16_t* y, int64_t ldy,
                                    int32_t* acc_debug, hipStream_t stream) {
  using C = GCfg;
  const int64_t tiles = ((M + C::BM - 1) / C::BM) * ((N + C::BN - 1) / C::BN);
  const dim3 grid((unsigned)tiles), block(256);
#define OFFQ_GG(D)                                                                            \
  hipLaunchKernelGGL((w4a4_gemm_grouped_kernel<D>), grid, block, 0, stream, a_codes, a_scale, \
                     a_zero, w_codes, w_scale, w_colsum, (int)M, (int)N, (int)K, log2g, y, ldy, \
                     acc_debug)
  // A debug request runs an accumulator-only pass, then the regular kernel.
  if (acc_debug) OFFQ_GG(true);
  OFFQ_GG(false);
#undef OFFQ_GG
  return hipGetLastError();
}

}  // namespace offq
