// W4A4 GEMM for one quantization group per row (g = K): the case of every
// full-width online Hadamard (attention projection, MLP up/gate, KV-chain
// projection).  gfx950, v_mfma_i32_32x32x32_i8.
//
//   acc[m,n] = sum_k q_a[m,k] q_w[n,k]                                (int32)
//   Y[m,n]   = sw[n] * s[m] * (acc[m,n] - z[m] * colsum[n])          -> bf16
//
// (the dequantised product of Eq. 1 with one scale/zero-point per row; the
// z * colsum term is the absorbed offset's correction).
//
// Organisation
// * 4 waves per workgroup, each owning a 128 x 128 output tile (4 x 4 MFMA
//   tiles of 32 x 32, 256 int32 accumulators, kept in AGPRs).
// * SPLITK = 1: waves arranged 2 x 2 -> 256 x 256 workgroup tile.
//   SPLITK = 2: two 128-row sub-tiles x two k-slots -> 256 x 128 workgroup
//   tile; the two k-slots are summed through LDS at the end.  Used when the
//   256 x 256 tiling leaves compute units idle.
// * Per stage every wave consumes 128 k (64 packed bytes per row); the stage
//   (A: 256 rows, B: 256 or 128 rows, 64 * SPLITK bytes each) is staged
//   through registers into a double-buffered LDS ring.  Rows are stored as
//   16-byte chunks whose order is XOR-swizzled with the row so that the
//   fragment reads (one row per lane, 8 lanes per LDS cycle) hit 8 different
//   bank groups.
// * The MFMA takes the weight fragment as its row operand and the activation
//   fragment as its column operand, i.e. it accumulates the transposed tile, so
//   that each lane ends with four consecutive output columns of one row.
// * Operands: activation codes (0..15) feed the signed i8 MFMA unchanged;
//   weight nibbles are widened to 16 * q (high nibble by a mask, low nibble by
//   a shift and a mask).  Each lane's 16-byte chunk gives two MFMA operands
//   (low nibbles, high nibbles): the same k-permutation on both operands.
//   The accumulator holds 16 * acc exactly.
// * Tile order: consecutive workgroups are dispatched to different XCDs, so
//   the linear id is first regrouped per XCD and then walked in groups of 4
//   tile rows, keeping each XCD's A and B panels within its own L2.
#include "common.h"
#include "internal.h"

namespace offq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

template <int SPLITK>
struct Cfg {
  static constexpr int BM = 256;
  static constexpr int BN = SPLITK == 1 ? 256 : 128;
  static constexpr int NC = 4 * SPLITK;            // 16-byte chunks per row and stage
  static constexpr int ROWB = 16 * NC;             // bytes per row and stage
  static constexpr int A_SLOTS = BM * NC;          // 16-byte slots of the A stage
  static constexpr int B_SLOTS = BN * NC;
  static constexpr int STAGE_SLOTS = A_SLOTS + B_SLOTS;
  static constexpr int A_LD = A_SLOTS / 256;       // loads per thread and stage
  static constexpr int B_LD = B_SLOTS / 256;
  static constexpr int KSTAGE = 128 * SPLITK;      // k per stage
};

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

__device__ __forceinline__ int acc_row(int i, int h) { return ((i >> 2) << 3) + (h << 2) + (i & 3); }

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

template <int SPLITK, bool DBG, bool WIDE>
__global__ __launch_bounds__(256) void w4a4_gemm_1g_kernel(
    const uint8_t* __restrict__ A, const uint16_t* __restrict__ a_scale,
    const int16_t* __restrict__ a_zero, const uint8_t* __restrict__ W,
    const uint16_t* __restrict__ w_scale, const int32_t* __restrict__ w_colsum, int M, int N,
    int K, uint16_t* __restrict__ Y, int64_t ldy, int32_t* __restrict__ acc_dbg) {
  using C = Cfg<SPLITK>;
  __shared__ uint4 lds[2 * C::STAGE_SLOTS];
  __shared__ __attribute__((aligned(16))) float sS[C::BM];
  __shared__ __attribute__((aligned(16))) int sZ[C::BM];
  __shared__ __attribute__((aligned(16))) float sSW[C::BN];
  __shared__ __attribute__((aligned(16))) int sCS[C::BN];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 5, fr = lane & 31;
  const int wm = wave & 1;
  const int wn = SPLITK == 1 ? (wave >> 1) : 0;
  const int ks = SPLITK == 1 ? 0 : (wave >> 1);

  const int tiles_m = (M + C::BM - 1) / C::BM;
  const int tiles_n = (N + C::BN - 1) / C::BN;
  int ti, tj;
  tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n, ti, tj);
  const int tm = ti * C::BM, tn = tj * C::BN;
  const int64_t ldk = K >> 1;
  const int nst = K / C::KSTAGE;

  // row scales / zero-points and column scales / weight sums of the tile
  {
    const int row = tm + tid;
    sS[tid] = row < M ? fp16_bits_to_f32(a_scale[row]) : 0.0f;
    sZ[tid] = row < M ? (int)a_zero[row] : 0;
    if (tid < C::BN) {
      const int col = tn + tid;
      sSW[tid] = col < N ? fp16_bits_to_f32(w_scale[col]) : 0.0f;
      sCS[tid] = col < N ? w_colsum[col] : 0;
    }
  }

  // This thread's 16-byte slots of a stage are slot = tid + 256 i, i.e. rows
  // tid / NC + i * (256 / NC) with the same (swizzled) chunk for every i.
  // Loads go through buffer descriptors whose size ends at row M (resp. N):
  // rows past the end read as zero.
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

  v16i acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = v16i{};

  gload(0);
  lstore(0);
  __syncthreads();

  for (int st = 0; st < nst; ++st) {
    const int buf = st & 1;
    if (st + 1 < nst) gload(st + 1);
    const uint4* As = lds + buf * C::STAGE_SLOTS;
    const uint4* Bs = As + C::A_SLOTS;
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int c = ks * 4 + 2 * h + jj;
      uint4 pa[4], pb[4];
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        const int ra_ = wm * 128 + f * 32 + fr;
        const int rb_ = wn * 128 + f * 32 + fr;
        pa[f] = As[ra_ * C::NC + swz<C::NC>(ra_, c)];
        pb[f] = Bs[rb_ * C::NC + swz<C::NC>(rb_, c)];
      }
#pragma unroll
      for (int sel = 0; sel < 2; ++sel) {
        v4i a[4], b[4];
#pragma unroll
        for (int f = 0; f < 4; ++f) {
          a[f] = sel ? act_hi(pa[f]) : act_lo(pa[f]);
          b[f] = sel ? wgt_hi16(pb[f]) : wgt_lo16(pb[f]);
        }
#pragma unroll
        for (int fm = 0; fm < 4; ++fm)
#pragma unroll
          for (int fn = 0; fn < 4; ++fn)
            acc[fm][fn] =
                __builtin_amdgcn_mfma_i32_32x32x32_i8(b[fn], a[fm], acc[fm][fn], 0, 0, 0);
      }
    }
    if (st + 1 < nst) lstore(buf ^ 1);
    __syncthreads();
  }

  if constexpr (SPLITK == 2) {
    // sum the two k-slots: waves of slot 1 hand their accumulators to slot 0,
    // 16 bytes per lane and access, in two rounds of two fragment rows
    v4i* red = reinterpret_cast<v4i*>(lds);
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      if (ks == 1) {
#pragma unroll
        for (int f2 = 0; f2 < 2; ++f2)
#pragma unroll
          for (int fn = 0; fn < 4; ++fn)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const v16i& t = acc[half * 2 + f2][fn];
              red[((((wm * 2 + f2) * 4 + fn) * 4 + q) * 64) + lane] =
                  v4i{t[4 * q], t[4 * q + 1], t[4 * q + 2], t[4 * q + 3]};
            }
      }
      __syncthreads();
      if (ks == 0) {
#pragma unroll
        for (int f2 = 0; f2 < 2; ++f2)
#pragma unroll
          for (int fn = 0; fn < 4; ++fn)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const v4i o = red[((((wm * 2 + f2) * 4 + fn) * 4 + q) * 64) + lane];
              acc[half * 2 + f2][fn][4 * q + 0] += o[0];
              acc[half * 2 + f2][fn][4 * q + 1] += o[1];
              acc[half * 2 + f2][fn][4 * q + 2] += o[2];
              acc[half * 2 + f2][fn][4 * q + 3] += o[3];
            }
      }
      __syncthreads();
    }
    if (ks == 1) return;
  }

  // epilogue: Y = sw * s * ((acc >> 4) - z * colsum) -> bf16.  The MFMA
  // computes the transposed tile (weights as the row operand), so lane column
  // fr is output row m and register i of fragment (fm, fn) is output column
  // fn*32 + 8*(i/4) + 4*h + i%4: four consecutive columns per 4 registers,
  // stored as one 8-byte write.
  if constexpr (DBG) {
    // accumulator-only launch: store acc (int32), four consecutive columns per
    // 4 registers; the output Y comes from a second, regular launch
#pragma unroll
    for (int fm = 0; fm < 4; ++fm) {
      const int row = tm + wm * 128 + fm * 32 + fr;
      if (row >= M) continue;
#pragma unroll
      for (int fn = 0; fn < 4; ++fn)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c0 = tn + wn * 128 + fn * 32 + q * 8 + h * 4;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (c0 + e < N) acc_dbg[(int64_t)row * N + c0 + e] = acc[fm][fn][q * 4 + e] >> 4;
        }
    }
    return;
  }
  const bool full = (tm + C::BM <= M) && (tn + C::BN <= N);
  const bool vec = full && (ldy % 4 == 0) && ((reinterpret_cast<uintptr_t>(Y) & 7) == 0);
  if (vec) {
    // interior tile: no bounds checks, 8-byte stores
#pragma unroll
    for (int fm = 0; fm < 4; ++fm) {
      const int lr = wm * 128 + fm * 32 + fr;
      const float rs = sS[lr];
      const int rz = sZ[lr];
      uint16_t* yrow = Y + (int64_t)(tm + lr) * ldy + tn + wn * 128 + h * 4;
#pragma unroll
      for (int fn = 0; fn < 4; ++fn) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int lc = wn * 128 + fn * 32 + q * 8 + h * 4;
          const int4 c4 = *reinterpret_cast<const int4*>(&sCS[lc]);
          const float4 s4 = *reinterpret_cast<const float4*>(&sSW[lc]);
          const int cs[4] = {c4.x, c4.y, c4.z, c4.w};
          const float sw[4] = {s4.x, s4.y, s4.z, s4.w};
          uint32_t v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int a = acc[fm][fn][q * 4 + e] >> 4;
            float d;
            if constexpr (!WIDE) d = (float)(a - rz * cs[e]);
            else d = (float)((long long)a - (long long)rz * (long long)cs[e]);
            v[e] = f32_to_bf16_rne(sw[e] * (rs * d));
          }
          *reinterpret_cast<uint2*>(yrow + fn * 32 + q * 8) =
              make_uint2(v[0] | (v[1] << 16), v[2] | (v[3] << 16));
        }
      }
    }
    return;
  }
  // edge tiles: checked scalar stores
#pragma unroll
  for (int fm = 0; fm < 4; ++fm) {
    const int lr = wm * 128 + fm * 32 + fr;
    const int row = tm + lr;
    if (row >= M) continue;
    const float rs = sS[lr];
    const int rz = sZ[lr];
#pragma unroll
    for (int fn = 0; fn < 4; ++fn) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int col = tn + wn * 128 + fn * 32 + acc_row(i, h);
        if (col < N) {
          const int a = acc[fm][fn][i] >> 4;
          const int cs = sCS[col - tn];
          const float sw = sSW[col - tn];
          float d;
          if constexpr (!WIDE) d = (float)(a - rz * cs);
          else d = (float)((long long)a - (long long)rz * (long long)cs);
          Y[(int64_t)row * ldy + col] = f32_to_bf16_rne(sw * (rs * d));
        }
      }
    }
  }
}

template <int SPLITK>
hipError_t launch_s(const uint8_t* a_codes, const uint16_t* a_scale, const int16_t* a_zero,
                    const uint8_t* w_codes, const uint16_t* w_scale, const int32_t* w_colsum,
                    int64_t M, int64_t N, int64_t K, uint16_t* y, int64_t ldy,
                    int32_t* acc_debug, hipStream_t stream) {
  using C = Cfg<SPLITK>;
  const int64_t tiles = ((M + C::BM - 1) / C::BM) * ((N + C::BN - 1) / C::BN);
  const dim3 grid((unsigned)tiles), block(256);
  // |z * colsum| < 2^31 is guaranteed for K <= 4096 (|z| <= 2^15, |colsum| <= 8 K)
  const bool wide = K > 4096;
#define OFFQ_G1(D, WD)                                                                          \
  hipLaunchKernelGGL((w4a4_gemm_1g_kernel<SPLITK, D, WD>), grid, block, 0, stream, a_codes,    \
                     a_scale, a_zero, w_codes, w_scale, w_colsum, (int)M, (int)N, (int)K, y, ldy, \
                     acc_debug)
  // A debug request runs an accumulator-only pass, then the regular kernel,
  // so that Y is always produced by the same code path.
  if (acc_debug) OFFQ_G1(true, false);
  if (wide) OFFQ_G1(false, true); else OFFQ_G1(false, false);
#undef OFFQ_G1
  return hipGetLastError();
}

}  // namespace

bool gemm_1g_supported(int64_t M, int64_t N, int64_t K) {
  // buffer offsets are 32-bit
  return K % 256 == 0 && M * (K / 2) < (int64_t(1) << 31) && N * (K / 2) < (int64_t(1) << 31);
}

hipError_t launch_w4a4_gemm_1g(const uint8_t* a_codes, const uint16_t* a_scale,
                               const int16_t* a_zero, const uint8_t* w_codes,
                               const uint16_t* w_scale, const int32_t* w_colsum, int64_t M,
                               int64_t N, int64_t K, uint16_t* y, int64_t ldy,
                               int32_t* acc_debug, hipStream_t stream) {
  // Prefer the 256 x 256 tiling unless it leaves much of the chip idle.
  const int64_t tiles1 = ((M + 255) / 256) * ((N + 255) / 256);
  if (tiles1 >= 384)
    return launch_s<1>(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K, y, ldy,
                       acc_debug, stream);
  return launch_s<2>(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K, y, ldy,
                     acc_debug, stream);
}

}  // namespace offq
