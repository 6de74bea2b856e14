// int4 x int4 GEMM with int32 accumulation and the OffQ dequantising epilogue
// (gfx950, v_mfma_i32_32x32x32_i8).
//
//   acc_b[m,n] = sum_{k in group b} q_a[m,k] q_w[n,k]
//   Y[m,n]     = sw[n] * sum_b s[m,b] * (acc_b[m,n] - z[m,b] * colsum[b,n])
//
// which is the product of the dequantised operands x_hat = s (q_a - z) and
// w_hat = sw q_w of Eq. 1 (sec. 3): the zero-point term, which carries the
// absorbed offset, becomes a correction through per-column weight sums.
//
// Operand handling: activation codes are unsigned 0..15 and go to the signed
// i8 MFMA unchanged; weight codes are signed 4-bit and are widened as 16*q
// (mask of the high nibble / shift of the low nibble into the high nibble),
// so every MFMA accumulates 16 * acc exactly and one arithmetic shift restores
// acc.  Both operands split each 16-byte k-slice into its low and its high
// nibbles (the same k-permutation on both sides, so dot products are
// unchanged).
#include "common.h"
#include "internal.h"

namespace offq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 128;  // tile rows (tokens)
constexpr int BN = 128;  // tile columns (output channels)
// k-step per iteration: 64 int4 = 32 bytes per row, held in LDS as two
// 16-byte halves per row, the halves of rows with bit 2 set swapped to spread
// the fragment reads over all LDS banks.
__device__ __forceinline__ int slot(int row, int half) {
  return row * 2 + (half ^ ((row >> 2) & 1));
}

__device__ __forceinline__ void unpack_act(const uint4 d, v4i& lo, v4i& hi) {
  lo = v4i{(int)(d.x & 0x0f0f0f0fu), (int)(d.y & 0x0f0f0f0fu),
           (int)(d.z & 0x0f0f0f0fu), (int)(d.w & 0x0f0f0f0fu)};
  hi = v4i{(int)((d.x >> 4) & 0x0f0f0f0fu), (int)((d.y >> 4) & 0x0f0f0f0fu),
           (int)((d.z >> 4) & 0x0f0f0f0fu), (int)((d.w >> 4) & 0x0f0f0f0fu)};
}

__device__ __forceinline__ void unpack_wgt16(const uint4 d, v4i& lo, v4i& hi) {
  lo = v4i{(int)((d.x << 4) & 0xf0f0f0f0u), (int)((d.y << 4) & 0xf0f0f0f0u),
           (int)((d.z << 4) & 0xf0f0f0f0u), (int)((d.w << 4) & 0xf0f0f0f0u)};
  hi = v4i{(int)(d.x & 0xf0f0f0f0u), (int)(d.y & 0xf0f0f0f0u),
           (int)(d.z & 0xf0f0f0f0u), (int)(d.w & 0xf0f0f0f0u)};
}

// Row of accumulator register i of a 32x32 MFMA tile held by a lane in the
// upper (h = 1) or lower (h = 0) half of the wave; the column is lane % 32.
__device__ __forceinline__ int acc_row(int i, int h) {
  return ((i >> 2) << 3) + (h << 2) + (i & 3);
}

template <bool DBG, bool WIDE>
__global__ __launch_bounds__(256) void w4a4_gemm_kernel(
    const uint8_t* __restrict__ A, const uint16_t* __restrict__ a_scale,
    const int16_t* __restrict__ a_zero, const uint8_t* __restrict__ W,
    const uint16_t* __restrict__ w_scale, const int32_t* __restrict__ w_colsum,
    int M, int N, int K, int log2g, uint16_t* __restrict__ Y, int64_t ldy,
    int32_t* __restrict__ acc_dbg) {
  __shared__ uint4 As[2][BM * 2];
  __shared__ uint4 Bs[2][BN * 2];
  __shared__ __attribute__((aligned(16))) float sS[BM];
  __shared__ __attribute__((aligned(16))) int sZ[BM];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int tiles_n = (N + BN - 1) / BN;
  const int tm = (int)(blockIdx.x / tiles_n) * BM;
  const int tn = (int)(blockIdx.x % tiles_n) * BN;
  const int64_t ldk = K >> 1;  // bytes per code row
  const int G = K >> log2g;
  const int ipg = 1 << (log2g - 6);  // k-iterations per group
  const int nk = K >> 6;

  // global -> LDS assignment: thread t moves 16 bytes of row t/2 of each tile
  const int lrow = tid >> 1, lhalf = tid & 1;
  const bool a_ok = tm + lrow < M;
  const bool b_ok = tn + lrow < N;
  const uint8_t* a_src = A + (int64_t)(a_ok ? tm + lrow : 0) * ldk + lhalf * 16;
  // weights in the blocked layout: k-step kit of row r is bytes 32 kit + 16 lhalf
  const int64_t KB = wblk_kblocks(K);
  const int64_t b_row = b_ok ? tn + lrow : 0;
  auto b_src = [&](int kit) { return W + wblk_off(b_row, 32 * kit + 16 * lhalf, KB); };
  const int st = slot(lrow, lhalf);

  const int fr = lane & 31, fh = lane >> 5;

  v16i acc[2][2];
  float yac[2][2][16];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      acc[a][b] = v16i{};
#pragma unroll
      for (int i = 0; i < 16; ++i) yac[a][b][i] = 0.0f;
    }

  const uint4 z4 = make_uint4(0u, 0u, 0u, 0u);
  uint4 ra = a_ok ? *reinterpret_cast<const uint4*>(a_src) : z4;
  uint4 rb = b_ok ? *reinterpret_cast<const uint4*>(b_src(0)) : z4;
  As[0][st] = ra;
  Bs[0][st] = rb;
  __syncthreads();

  for (int kit = 0; kit < nk; ++kit) {
    const int buf = kit & 1;
    if (kit + 1 < nk) {
      ra = a_ok ? *reinterpret_cast<const uint4*>(a_src + (int64_t)(kit + 1) * 32) : z4;
      rb = b_ok ? *reinterpret_cast<const uint4*>(b_src(kit + 1)) : z4;
    }
    v4i alo[2], ahi[2], blo[2], bhi[2];
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      const int r = wm * 64 + f * 32 + fr;
      unpack_act(As[buf][slot(r, fh)], alo[f], ahi[f]);
      const int c = wn * 64 + f * 32 + fr;
      unpack_wgt16(Bs[buf][slot(c, fh)], blo[f], bhi[f]);
    }
#pragma unroll
    for (int fm = 0; fm < 2; ++fm)
#pragma unroll
      for (int fn = 0; fn < 2; ++fn) {
        acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(alo[fm], blo[fn], acc[fm][fn], 0, 0, 0);
        acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(ahi[fm], bhi[fn], acc[fm][fn], 0, 0, 0);
      }
    if (kit + 1 < nk) {
      As[buf ^ 1][st] = ra;
      Bs[buf ^ 1][st] = rb;
    }
    __syncthreads();

    if (((kit + 1) & (ipg - 1)) == 0) {
      // fold group b into the fp32 accumulators; row scales and zero-points
      // of the tile are staged through LDS
      const int b = kit >> (log2g - 6);
      if (tid < BM) {
        const int row = tm + tid;
        sS[tid] = row < M ? fp16_bits_to_f32(a_scale[(int64_t)row * G + b]) : 0.0f;
        sZ[tid] = row < M ? (int)a_zero[(int64_t)row * G + b] : 0;
      }
      __syncthreads();
#pragma unroll
      for (int fm = 0; fm < 2; ++fm) {
        float rs[16];
        int rz[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int r0 = wm * 64 + fm * 32 + q * 8 + fh * 4;
          const float4 s4 = *reinterpret_cast<const float4*>(&sS[r0]);
          const int4 z4i = *reinterpret_cast<const int4*>(&sZ[r0]);
          rs[q * 4 + 0] = s4.x; rs[q * 4 + 1] = s4.y; rs[q * 4 + 2] = s4.z; rs[q * 4 + 3] = s4.w;
          rz[q * 4 + 0] = z4i.x; rz[q * 4 + 1] = z4i.y; rz[q * 4 + 2] = z4i.z; rz[q * 4 + 3] = z4i.w;
        }
#pragma unroll
        for (int fn = 0; fn < 2; ++fn) {
          const int col = tn + wn * 64 + fn * 32 + fr;
          const int cs = col < N ? w_colsum[(int64_t)b * N + col] : 0;
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int a = acc[fm][fn][i] >> 4;
            float d;
            if constexpr (WIDE) {
              d = (float)((long long)a - (long long)rz[i] * (long long)cs);
            } else {
              d = (float)(a - rz[i] * cs);
            }
            yac[fm][fn][i] += rs[i] * d;
            if constexpr (DBG) {
              const int row = tm + wm * 64 + fm * 32 + acc_row(i, fh);
              if (row < M && col < N) acc_dbg[((int64_t)b * M + row) * N + col] = a;
            }
          }
          acc[fm][fn] = v16i{};
        }
      }
    }
  }

  // epilogue: per-column weight scale, bf16 round, store
#pragma unroll
  for (int fm = 0; fm < 2; ++fm)
#pragma unroll
    for (int fn = 0; fn < 2; ++fn) {
      const int col = tn + wn * 64 + fn * 32 + fr;
      if (col >= N) continue;
      const float sw = fp16_bits_to_f32(w_scale[col]);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int row = tm + wm * 64 + fm * 32 + acc_row(i, fh);
        if (row < M) Y[(int64_t)row * ldy + col] = f32_to_bf16_rne(sw * yac[fm][fn][i]);
      }
    }
}

// ---------------------------------------------------------------------------
// Decode GEMV (M <= 16) for the shapes the MFMA GEMV does not take (g = 64,
// very many groups): one wavefront per output channel n streams the weight
// row with 16-byte coalesced loads, lane l taking chunk 64 p + l (32 k) in
// pass p.  v_dot8_i32_i4 on (q_a - 8, q_w) (activation codes re-biased by
// xor 0x8 per nibble) accumulates each group in int32: a group covers
// g / 32 consecutive lanes of one pass (g <= 2048) or whole passes
// (g > 2048); when it ends, its lanes add their int32 sums (exact), and the
// group's first lane folds acc_b = sum (q_a - 8) q_w + 8 colsum_b into the
// fp32 output, F += s (acc_b - z colsum_b).  DBG also stores acc_b.
template <int MT, bool DBG>
__global__ __launch_bounds__(256) void w4a4_gemv_kernel(
    const uint8_t* __restrict__ A, const uint16_t* __restrict__ a_scale,
    const int16_t* __restrict__ a_zero, const uint8_t* __restrict__ W,
    const uint16_t* __restrict__ w_scale, const int32_t* __restrict__ w_colsum,
    int M, int N, int K, int log2g, uint16_t* __restrict__ Y, int64_t ldy,
    int32_t* __restrict__ acc_dbg) {
  const int lane = threadIdx.x & 63;
  const int n = (int)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;  // wave-uniform
  const int64_t ldk = K >> 1;
  const int G = K >> log2g;
  const int64_t KB = wblk_kblocks(K);               // weights in the blocked layout
  const int nchunks = (int)(ldk >> 4);            // 16-byte chunks (32 k) per row
  const int seg = 1 << min(log2g - 5, 6);        // lanes of one group in one pass
  const int passes = (nchunks + 63) >> 6;
  float part[MT];
  int acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    part[m] = 0.0f;
    acc[m] = 0;
  }
  const uint4 z4 = make_uint4(0u, 0u, 0u, 0u);
  for (int p = 0; p < passes; ++p) {
    const int c = (p << 6) + lane;
    const bool live = c < nchunks;  // a dead lane's zero weights add nothing
    const uint4 w = live ? *reinterpret_cast<const uint4*>(W + wblk_off(n, (int64_t)c * 16, KB)) : z4;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      if (m < M) {
        const uint4 a = live ? *reinterpret_cast<const uint4*>(A + (int64_t)m * ldk + (int64_t)c * 16) : z4;
        int d = acc[m];
        d = __builtin_amdgcn_sdot8((int)(a.x ^ 0x88888888u), (int)w.x, d, false);
        d = __builtin_amdgcn_sdot8((int)(a.y ^ 0x88888888u), (int)w.y, d, false);
        d = __builtin_amdgcn_sdot8((int)(a.z ^ 0x88888888u), (int)w.z, d, false);
        d = __builtin_amdgcn_sdot8((int)(a.w ^ 0x88888888u), (int)w.w, d, false);
        acc[m] = d;
      }
    }
    // groups end in every pass (g <= 2048), or after g / 2048 passes
    if (log2g <= 11 || ((((int64_t)p + 1) << 11) & ((int64_t(1) << log2g) - 1)) == 0) {
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        int t = acc[m];
        for (int off = 1; off < seg; off <<= 1) t += __shfl_xor(t, off);
        acc[m] = t;
      }
      if (live && (lane & (seg - 1)) == 0) {
        const int b = (int)(((int64_t)c << 5) >> log2g);
        const int cs = w_colsum[(int64_t)b * N + n];
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          if (m < M) {
            const int a_b = acc[m] + 8 * cs;  // sum_{k in b} q_a q_w
            const float s = fp16_bits_to_f32(a_scale[(int64_t)m * G + b]);
            const int z = a_zero[(int64_t)m * G + b];
            part[m] += s * (float)((long long)a_b - (long long)z * (long long)cs);
            if constexpr (DBG) acc_dbg[((int64_t)b * M + m) * N + n] = a_b;
          }
        }
      }
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[m] = 0;
    }
  }
#pragma unroll
  for (int m = 0; m < MT; ++m) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) part[m] += __shfl_xor(part[m], off);
  }
  if (lane == 0) {
    const float sw = fp16_bits_to_f32(w_scale[n]);
#pragma unroll
    for (int m = 0; m < MT; ++m)
      if (m < M) Y[(int64_t)m * ldy + n] = f32_to_bf16_rne(sw * part[m]);
  }
}

}  // namespace

hipError_t launch_w4a4_gemm(const uint8_t* a_codes, const uint16_t* a_scale,
                            const int16_t* a_zero, const uint8_t* w_codes,
                            const uint16_t* w_scale, const int32_t* w_colsum,
                            int64_t M, int64_t N, int64_t K, int log2g,
                            uint16_t* y, int64_t ldy, int32_t* acc_debug,
                            hipStream_t stream) {
  if (gemm_grouped_supported(M, N, K, log2g))
    return launch_w4a4_gemm_grouped(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N,
                                    K, log2g, y, ldy, acc_debug, stream);
  const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  const dim3 grid((unsigned)tiles), block(256);
  const bool wide = log2g >= 13;
#define OFFQ_GEMM(D, WD)                                                                 \
  hipLaunchKernelGGL((w4a4_gemm_kernel<D, WD>), grid, block, 0, stream, a_codes, a_scale, \
                     a_zero, w_codes, w_scale, w_colsum, (int)M, (int)N, (int)K, log2g, y, \
                     ldy, acc_debug)
  if (acc_debug) {
    if (wide) OFFQ_GEMM(true, true); else OFFQ_GEMM(true, false);
  } else {
    if (wide) OFFQ_GEMM(false, true); else OFFQ_GEMM(false, false);
  }
#undef OFFQ_GEMM
  return hipGetLastError();
}

hipError_t launch_w4a4_gemv(const uint8_t* a_codes, const uint16_t* a_scale,
                            const int16_t* a_zero, const uint8_t* w_codes,
                            const uint16_t* w_scale, const int32_t* w_colsum,
                            int64_t M, int64_t N, int64_t K, int log2g,
                            uint16_t* y, int64_t ldy, int32_t* acc_debug,
                            hipStream_t stream) {
  const dim3 grid((unsigned)((N + 3) / 4)), block(256);
#define OFFQ_GEMV(MT, D)                                                                  \
  hipLaunchKernelGGL((w4a4_gemv_kernel<MT, D>), grid, block, 0, stream, a_codes, a_scale, \
                     a_zero, w_codes, w_scale, w_colsum, (int)M, (int)N, (int)K, log2g, y, \
                     ldy, acc_debug)
  if (M <= 1) {
    if (acc_debug) OFFQ_GEMV(1, true); else OFFQ_GEMV(1, false);
  } else if (M <= 4) {
    if (acc_debug) OFFQ_GEMV(4, true); else OFFQ_GEMV(4, false);
  } else {
    if (acc_debug) OFFQ_GEMV(16, true); else OFFQ_GEMV(16, false);
  }
#undef OFFQ_GEMV
  return hipGetLastError();
}

}  // namespace offq
