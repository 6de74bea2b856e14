// W4A4 decode GEMV (M <= 16 tokens), gfx950, v_mfma_i32_16x16x64_i8.
//
//   acc_b[m,n] = sum_{k in group b} q_a[m,k] q_w[n,k]                 (int32)
//   Y[m,n]     = sw[n] * sum_b s[m,b] * (acc_b[m,n] - z[m,b] * colsum[b,n])
//
// (the dequantised product of Eq. 1; the z * colsum terms carry the absorbed
// offsets).  The int4 weights are streamed once from HBM; the few token rows
// are padded to the MFMA's 16 columns, which costs MFMA slots that are idle
// anyway in a memory-bound kernel.
//
// Organisation
// * A workgroup of P waves owns T row tiles of 16 output channels; the P
//   waves split K and their fp32 partial sums are added through LDS at the
//   end.
// * Per step of 128 k every lane loads 16 packed bytes of one weight row per
//   tile (lane l: row l % 16, k-block l / 16: the wave reads one 1 KB block
//   of the blocked weight layout, contiguous in memory) and the
//   same 16 bytes of its token row l % 16 (rows >= M read as zero through the
//   buffer descriptor), and runs two MFMAs per tile (low and high nibbles, the
//   same k-permutation on both operands).  Weight nibbles are widened to 16 q.
//   Steps go in batches of 4; the next batch's loads are issued before the
//   current batch is multiplied.  One activation load serves T weight loads:
//   the activation rows are re-read by every row tile, so with T = 1 they
//   would double the load traffic of M = 16.
// * Accumulators are folded per group: F += (s / 16) * acc - s z colsum (the
//   zero-point term added by the wave that holds the group's first k), with
//   the group parameters of the workgroup preloaded into LDS.
#include "common.h"
#include "gemm_common.h"
#include "internal.h"

namespace offq {
namespace {

using namespace gemm;

typedef unsigned int p_u32x2 __attribute__((ext_vector_type(2)));

constexpr int KSTEP = 128;  // k per step (64 packed bytes per row)
constexpr int GMAX = 256;   // groups whose parameters fit in LDS

// T: 16-channel row tiles per wave (one activation load serves T weight
// loads); P: waves per workgroup, each taking 1/P of K; BATCH: steps of 128 k
// per batch of loads (registers).
template <int T, int P, int BATCH>
struct GvCfg {
  static constexpr int THREADS = 64 * P;
};

template <int T, int P, int BATCH, bool DBG>
__global__ __launch_bounds__(64 * P) void w4a4_gemv_kernel(
    const uint8_t* __restrict__ A, const uint16_t* __restrict__ a_scale,
    const int16_t* __restrict__ a_zero, const uint8_t* __restrict__ W,
    const uint16_t* __restrict__ w_scale, const int32_t* __restrict__ w_colsum, int M, int N,
    int K, int log2g, uint16_t* __restrict__ Y, int64_t ldy, int32_t* __restrict__ acc_dbg) {
  constexpr int NT = GvCfg<T, P, BATCH>::THREADS;
  __shared__ float red[P][64][T * 4];
  // per group: s / 16 and -s z of the 16 token rows, colsum of the tile's channels
  extern __shared__ float gpar[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, kb = lane >> 4;
  const int n0 = (int)blockIdx.x * (16 * T);
  const int ldk = K >> 1;
  const int G = K >> log2g;
  const int kq = K / P;                  // k per wave
  const int k0 = wave * kq;
  const int nb = kq / (KSTEP * BATCH);   // batches per wave
  float* const sS = gpar;                // [G][16]
  float* const sSZ = gpar + G * 16;      // [G][16]
  float* const sCS = gpar + G * 32;      // [G][16 T]
  float* const sSW = gpar + G * (32 + 16 * T);  // [16 T] weight scales of the tile


  // rows past N (weights) and past M (tokens) read as zero
  // (weights: the tile's bands of the blocked layout, K a multiple of 128, so a
  // band is 16 ldk bytes; the padding rows of the last band hold zero codes)
  const __amdgpu_buffer_rsrc_t wrsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(W + (int64_t)n0 * ldk), 0, (int)((int64_t)((min(16 * T, N - n0) + 15) & ~15) * ldk),
      0x00020000);
  const __amdgpu_buffer_rsrc_t arsrc =
      __builtin_amdgcn_make_buffer_rsrc((void*)A, 0, M * ldk, 0x00020000);
  const int a_off = r16 * ldk + (k0 >> 1) + 16 * kb;
  int w_off[T];
#pragma unroll
  for (int t = 0; t < T; ++t) w_off[t] = (t * (K >> 7) + (k0 >> 7)) * 1024 + r16 * 64 + 16 * kb;

  v4i acc[T];
  float F[T][4];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    acc[t] = v4i{};
#pragma unroll
    for (int i = 0; i < 4; ++i) F[t][i] = 0.0f;
  }

  // Register i of tile t is output channel n0 + 16 t + 4 kb + i, token row
  // r16 (the lane's column).  The zero-point term of a group is added by the
  // wave that holds the group's first k.
  auto fold = [&](int b) __attribute__((always_inline)) {
    if constexpr (DBG) {
#pragma unroll
      for (int t = 0; t < T; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int n = n0 + 16 * t + 4 * kb + i;
          if (r16 < M && n < N)
            atomicAdd(&acc_dbg[((int64_t)b * M + r16) * N + n], acc[t][i] >> 4);
        }
    } else {
      const float s = sS[b * 16 + r16];
      const float sz = (b << log2g) >= k0 ? sSZ[b * 16 + r16] : 0.0f;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const float4 c4 = *reinterpret_cast<const float4*>(&sCS[b * 16 * T + 16 * t + 4 * kb]);
        const float cs[4] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          F[t][i] = __builtin_fmaf(s, (float)acc[t][i], F[t][i]);
          F[t][i] = __builtin_fmaf(sz, cs[i], F[t][i]);
        }
      }
    }
#pragma unroll
    for (int t = 0; t < T; ++t) acc[t] = v4i{};
  };

  uint4 wa0[BATCH][T], aa0[BATCH], wa1[BATCH][T], aa1[BATCH];
  auto load = [&](int bt, uint4 (&wa)[BATCH][T], uint4 (&aa)[BATCH]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < BATCH; ++u) {
      const int so = (bt * BATCH + u) * (KSTEP / 2);
      aa[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(arsrc, a_off, so, 0));
#pragma unroll
      for (int t = 0; t < T; ++t)
        wa[u][t] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(wrsrc, w_off[t], 16 * so, 0));
    }
  };
  const int gmask = (1 << (log2g - 7)) - 1;  // steps per group - 1
  auto compute = [&](int bt, const uint4 (&wa)[BATCH][T], const uint4 (&aa)[BATCH]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < BATCH; ++u) {
      const v4i alo = act_lo(aa[u]), ahi = act_hi(aa[u]);
#pragma unroll
      for (int t = 0; t < T; ++t) {
        acc[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wgt_lo16(wa[u][t]), alo, acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wgt_hi16(wa[u][t]), ahi, acc[t], 0, 0, 0);
      }
      // the step ends a group, or the wave's part of it
      const int sabs = (k0 >> 7) + bt * BATCH + u;
      if ((sabs & gmask) == gmask || bt * BATCH + u == nb * BATCH - 1) fold(sabs >> (log2g - 7));
    }
  };

  // Group parameters of the workgroup into LDS: the first PRE entries per
  // thread are requested before the first two batches and written after
  // them (so that the weight stream starts at once and the writes wait for
  // the parameters only); the rest, if any, after.
  constexpr int PRE = 4;
  auto par_s = [&](int i, float& s, float& sz) __attribute__((always_inline)) {
    const int b = i >> 4, m = i & 15;
    const bool ok = m < M;
    s = ok ? fp16_bits_to_f32(a_scale[(int64_t)m * G + b]) : 0.0f;
    sz = ok ? -(s * (float)a_zero[(int64_t)m * G + b]) : 0.0f;
    s *= 0.0625f;  // undoes the 16x widening of the weight codes
  };
  auto par_c = [&](int i) __attribute__((always_inline)) {
    const int b = i / (16 * T), c = i % (16 * T);
    return n0 + c < N ? (float)w_colsum[(int64_t)b * N + n0 + c] : 0.0f;
  };
  float ps[PRE], pz[PRE], pc[PRE];
#pragma unroll
  for (int p = 0; p < PRE; ++p) {
    const int i = tid + p * NT;
    if (i < G * 16) par_s(i, ps[p], pz[p]);
    if (i < G * 16 * T) pc[p] = par_c(i);
  }
  load(0, wa0, aa0);
  if (nb > 1) load(1, wa1, aa1);
#pragma unroll
  for (int p = 0; p < PRE; ++p) {
    const int i = tid + p * NT;
    if (i < G * 16) {
      sS[i] = ps[p];
      sSZ[i] = pz[p];
    }
    if (i < G * 16 * T) sCS[i] = pc[p];
  }
  for (int i = tid + PRE * NT; i < G * 16; i += NT) par_s(i, sS[i], sSZ[i]);
  for (int i = tid + PRE * NT; i < G * 16 * T; i += NT) sCS[i] = par_c(i);
  // the tile's weight scales, for the end (a load there would add one memory
  // latency after the last step)
  for (int i = tid; i < 16 * T; i += NT) sSW[i] = n0 + i < N ? fp16_bits_to_f32(w_scale[n0 + i]) : 0.0f;
  __syncthreads();
  int bt = 0;
  for (; bt + 2 <= nb; bt += 2) {
    compute(bt, wa0, aa0);
    if (bt + 2 < nb) load(bt + 2, wa0, aa0);
    compute(bt + 1, wa1, aa1);
    if (bt + 3 < nb) load(bt + 3, wa1, aa1);
  }
  if (bt < nb) compute(bt, wa0, aa0);
  if constexpr (DBG) return;

  // ---- sum the P parts of K and store ---------------------------------------
  // Wave w finishes row tiles w, w + P, ...: four consecutive channels per
  // lane and tile, one 8-byte store where the row allows it.
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][lane][t * 4 + i] = F[t][i];
  __syncthreads();
  const bool vec = (ldy & 3) == 0 && (reinterpret_cast<uintptr_t>(Y) & 7) == 0;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    if (t % P != wave || r16 >= M) continue;
    const int c = 16 * t + 4 * kb;
    const int n = n0 + c;
    float f[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[i] = 0.0f;
#pragma unroll
      for (int w = 0; w < P; ++w) f[i] += red[w][lane][t * 4 + i];
      f[i] *= sSW[c + i];
    }
    uint16_t* const yp = Y + (int64_t)r16 * ldy + n;
    if (vec && n + 3 < N) {
      const p_u32x2 v = {bf16x2_rne(f[0], f[1]), bf16x2_rne(f[2], f[3])};
      *reinterpret_cast<p_u32x2*>(yp) = v;
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (n + i < N) yp[i] = f32_to_bf16_rne(f[i]);
    }
  }
}

}  // namespace

// Launch shape (T row tiles per wave, K in P parts, BATCH steps per load
// batch), as measured at M = 16 (g = 128 ... 8192) on the blocked weight
// layout: wide layers (>= 16384 channels) take two row tiles per wave and K
// in eighths, batches of two steps (8192 -> 28672: 27.0 -> 25.1 us at
// M = 16, 27.0 -> 22.8 at M = 1, against four tiles and K in quarters, the
// best shape of the row-major layout; the same at 4096 -> 28672), or four
// tiles and K in quarters when K is not a multiple of 2048; narrower ones
// need more waves in flight:
// K in eighths with two tiles per wave from 6144 channels, one below, where K
// splits into eighths of whole batches (from K = 16384 with two tiles: K in
// sixteenths, batches of two steps: 26.7-27.8 against 29.9-31.4 us at
// 28672 -> 8192); a K that is a multiple of 2048 but not of 4096 (14336,
// 6144, 2048) one tile per wave, K in sixteenths and batches of one step
// (4096 <- 14336 at g = 128: 15.0 -> 11.0 us against quarters in batches of
// four; 7.9 against 12.3 us at M = 1).  A K that is not a whole number of
// such batches (short rows, e.g. K = 256) takes one tile per wave, batches
// of one step and K in as many parts (4, 2, 1) as it divides into.
static void gemv_shape(int64_t N, int64_t K, int& T, int& P, int& B) {
  if (N >= 16384) {
    if (K % 2048 == 0) T = 2, P = 8, B = 2;
    else T = 4, P = 4, B = 2;
  } else if (K % 4096 == 0) {
    T = N >= 6144 ? 2 : 1, P = T == 2 && K >= 16384 ? 16 : 8;
    B = P == 16 ? 2 : 4;
  } else if (K % 2048 == 0) {
    T = 1, P = 16, B = 1;
  } else {
    T = 4, P = 4, B = 2;
  }
  if (K % ((int64_t)P * KSTEP * B) != 0) {
    T = 1, B = 1;
    P = K % (4 * KSTEP) == 0 ? 4 : K % (2 * KSTEP) == 0 ? 2 : 1;
  }
}

bool gemv_mfma_supported(int64_t M, int64_t N, int64_t K, int log2g) {
  // each wave's part of K is a whole number of batches (a part may end inside
  // a group: the group's zero-point term is added once, by the wave holding
  // its first k); no step straddles a group; the group parameters fit in LDS;
  // 32-bit buffer offsets
  int T, P, B;
  gemv_shape(N, K, T, P, B);
  const int64_t batch = (int64_t)P * KSTEP * B;
  // group parameters (dynamic) + the partial sums of the P waves (static)
  const int64_t lds = ((K >> log2g) * (32 + 16 * T) + 16 * T) * 4 + (int64_t)P * 64 * 4 * T * 4;
  return M <= 16 && log2g >= 7 && K % batch == 0 && (K >> log2g) <= GMAX &&
         lds <= 160 * 1024 &&
         32 * (K / 2) < (int64_t(1) << 31) && M * (K / 2) < (int64_t(1) << 31);
}

template <int T, int P, int BATCH>
hipError_t launch_gv(const uint8_t* a_codes, const uint16_t* a_scale, const int16_t* a_zero,
                     const uint8_t* w_codes, const uint16_t* w_scale, const int32_t* w_colsum,
                     int64_t M, int64_t N, int64_t K, int log2g, uint16_t* y, int64_t ldy,
                     int32_t* acc_debug, hipStream_t stream) {
  const int rows = 16 * T;
  const dim3 grid((unsigned)((N + rows - 1) / rows)), block(64 * P);
  const size_t lds = ((size_t)(K >> log2g) * (32 + rows) + rows) * sizeof(float);
  // A debug request runs an accumulator-only pass (partial sums added
  // atomically into the zeroed buffer), then the regular kernel.
  if (acc_debug) {
    hipError_t e = hipMemsetAsync(acc_debug, 0, (size_t)(K >> log2g) * M * N * sizeof(int32_t),
                                  stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((w4a4_gemv_kernel<T, P, BATCH, true>), grid, block, lds, stream, a_codes,
                       a_scale, a_zero, w_codes, w_scale, w_colsum, (int)M, (int)N, (int)K, log2g,
                       y, ldy, acc_debug);
  }
  hipLaunchKernelGGL((w4a4_gemv_kernel<T, P, BATCH, false>), grid, block, lds, stream, a_codes, a_scale,
                     a_zero, w_codes, w_scale, w_colsum, (int)M, (int)N, (int)K, log2g, y, ldy,
                     acc_debug);
  return hipGetLastError();
}

hipError_t launch_w4a4_gemv_mfma(const uint8_t* a_codes, const uint16_t* a_scale,
                                 const int16_t* a_zero, const uint8_t* w_codes,
                                 const uint16_t* w_scale, const int32_t* w_colsum, int64_t M,
                                 int64_t N, int64_t K, int log2g, uint16_t* y, int64_t ldy,
                                 int32_t* acc_debug, hipStream_t stream) {
  int T, P, B;
  gemv_shape(N, K, T, P, B);
#define OFFQ_GV(T, P, B)                                                                         \
  return launch_gv<T, P, B>(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K, log2g, \
                            y, ldy, acc_debug, stream)
  if (B == 1) {
    if (P == 16) OFFQ_GV(1, 16, 1);
    if (P == 4) OFFQ_GV(1, 4, 1);
    if (P == 2) OFFQ_GV(1, 2, 1);
    OFFQ_GV(1, 1, 1);
  }
  if (T == 4) OFFQ_GV(4, 4, 2);
  if (T == 2 && P == 16) OFFQ_GV(2, 16, 2);
  if (T == 2 && B == 2) OFFQ_GV(2, 8, 2);
  if (T == 2) OFFQ_GV(2, 8, 4);
  if (P == 8) OFFQ_GV(1, 8, 4);
  OFFQ_GV(1, 4, 4);
#undef OFFQ_GV
}

}  // namespace offq
