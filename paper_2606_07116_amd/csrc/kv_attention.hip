// One decode step of attention over the 4-bit KV cache (gfx950).
//
// The cache rows are the output of the KV quantizer: per (batch b, head h,
// position j) 128 codes of 4 bits with an fp16 scale and an int16 zero-point
// (sec. 4.2: KV group = head dimension).  Keys were rotated by the per-head
// Hadamard H3 before quantization (sec. 3.3 step 2(3)), so the query meets
// them rotated the same way; values carry the offline rotation R2 (sec. 3.3
// step 2(2)), which the output projection undoes, or, if they were quantized
// with the online Hadamard as well, the output is rotated back by H3.
//
//   q_r  = bf16_rne(fl32(c * fl32(H q)))             c = fl32(1 / sqrt(128))
//   s_j  = sm_scale * sk_j * sum_d q_r[d] (ck_j[d] - zk_j)
//   p    = softmax_j(s)
//   o[d] = sum_j w_j (cv_j[d] - zv_j) / sum_j p_j,   w_j = fp16(p_j sv_j)
//   (then c * H o if asked)
//
// The work is HBM-bound (136 bytes per position and head) and unpacking the
// 4-bit codes is what costs VALU time, so the kernel is built around
// unpacking with as few instructions as possible:
// * a 4-bit code c masked in place inside a 16-bit half is the fp16
//   subnormal c 2^-24 (or 16 c 2^-24 for the high nibble of a byte); its
//   products with fp16 operands are exact in fp32, so v_dot2_f32_f16 takes
//   two codes per instruction straight from one AND of the code word, with
//   no offset and no conversion;
// * scores: the rotated query, scaled by a power of two into the fp16 range
//   (exact), is laid out as fp16 pairs (dims 8i + j, 8i + j + 4) matching
//   the nibbles j, j + 4 of code word i, divided by 16 for odd j;
// * values: a lane takes two positions at once; v_perm_b32 interleaves their
//   code bytes so that every AND yields (code of A, code of B) for one
//   dimension, dotted with the fp16 pair of their weights p sv.
//
// Grouped-query attention: query head h of batch b reads the cache of
// key/value head h / group (group = Hq / Hkv; 1 for plain multi-head).  For
// group 2 and 4 one workgroup serves the group's query heads together and
// forms both products on the matrix cores instead (below).
//
// Organisation (split over the sequence, as in flash decoding)
// * Pass 1: one workgroup of 4 waves per (b, h, chunk of 1024 positions);
//   a wave owns 256 consecutive positions, in 8 blocks of 32.  A lane
//   (quarter qd = lane & 3, row group rg = lane >> 2) takes the 16-byte
//   quarter qd of the code rows rg and rg + 16 of a block, so each load
//   instruction of a wave reads 1 KB of contiguous codes.  Partial dot
//   products meet through two DPP adds in the quad; the chunk's maximum goes
//   through LDS; the weights stay in registers for the value pass.  The
//   chunk's maximum (log2 domain), its sum of p and its unnormalised output
//   go to the workspace.
// * Pass 2: one workgroup per (b, h) merges the chunks (rescaled by
//   2^(m_i - m)), divides by the sum, optionally rotates back, stores bf16.
#include <mutex>

#include "common.h"
#include "internal.h"

namespace offq {
namespace {

constexpr int DH = 128;            // head dimension
constexpr int CH = 1024;           // positions per pass-1 workgroup
constexpr int THREADS = 256;       // 4 waves
constexpr int WAVES = THREADS / 64;
constexpr int WROWS = CH / WAVES;  // 256 positions per wave
constexpr int NIT = WROWS / 32;    // blocks of 32 positions per wave
constexpr float LOG2E = 1.4426950408889634f;
constexpr int WS_FLOATS = 2 + DH;  // per (b, h, chunk): m, l, o[128]

typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));

// acc + a.lo * b.lo + a.hi * b.hi for two packed fp16 pairs (fp32 result;
// fp16 subnormal operands are kept).  The builtin, not inline asm, so that
// the compiler's hazard tracking sees the dot instruction.
__device__ __forceinline__ float dot2_f16(uint32_t a, uint32_t b, float acc) {
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2_t, a), __builtin_bit_cast(f16x2_t, b),
                                acc, false);
}

__device__ __forceinline__ uint32_t pack_f16(float a, float b) {
  const f16x2_t h = {(_Float16)a, (_Float16)b};
  return __builtin_bit_cast(uint32_t, h);
}

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xf, 0xf, true));
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fminf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

struct ChunkSmem {
  float qf[DH];                 // rotated query, scaled into the fp16 range
  uint32_t qp[DH / 2];          // query as fp16 pairs, see the header
  float qsum, qexp;             // sum of q_r; the power-of-two exponent
  float2 kab[CH];               // per position: score (log2 domain) = a * dot + b
  float2 vsz[CH];               // per position: (sv, zv)
  float red[3][WAVES];          // per wave: max, sum p, sum w zv
  float o[WAVES][4][DH];        // per wave and DPP row: partial outputs
};

template <bool FULL>
__device__ __forceinline__ void attention_chunk(ChunkSmem& S, const uint16_t* __restrict__ q,
                                                const uint8_t* __restrict__ kc,
                                                const uint16_t* __restrict__ ks,
                                                const int16_t* __restrict__ kz,
                                                const uint8_t* __restrict__ vc,
                                                const uint16_t* __restrict__ vs,
                                                const int16_t* __restrict__ vz, int64_t row0,
                                                int64_t bh, int n, float sm2, float cnorm,
                                                float* __restrict__ rec) {
  const int tid = (int)__builtin_amdgcn_workitem_id_x();
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qd = lane & 3, rg = lane >> 2;

  // row of block it, half h (chunk-relative): wave * 256 + it * 32 + h * 16 + rg
  auto row = [&](int it, int h) {
    const int r = wave * WROWS + it * 32 + h * 16 + rg;
    return FULL ? r : min(r, n - 1);
  };

  // ---- key codes of the wave's 256 positions, issued first ---------------
  const uint8_t* kbase = kc + row0 * (DH / 2);
  // blocks of 32 positions of this wave that hold any of the chunk's n
  // positions (all of them in a full chunk); the others are skipped
  const int nact = FULL ? NIT : min(NIT, max(0, (n - wave * WROWS + 31) / 32));
  uint4 kd[NIT][2];
#pragma unroll
  for (int it = 0; it < NIT; ++it)
    if (FULL || it < nact)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        kd[it][h] =
            *reinterpret_cast<const uint4*>(kbase + (uint32_t)(row(it, h) * (DH / 2) + qd * 16));

  // ---- query: FWHT across the lanes of wave 0 (lane holds dims 2l, 2l+1) --
  if (wave == 0) {
    const float a = bf16_lo(q[bh * DH + 2 * lane]), b = bf16_lo(q[bh * DH + 2 * lane + 1]);
    float x0 = a + b, x1 = a - b;
#pragma unroll
    for (int s = 0; s < 6; ++s) {
      const float y0 = __shfl_xor(x0, 1 << s), y1 = __shfl_xor(x1, 1 << s);
      const bool up = (lane >> s) & 1;
      x0 = up ? y0 - x0 : x0 + y0;
      x1 = up ? y1 - x1 : x1 + y1;
    }
    const float r0 = bf16_lo(f32_to_bf16_rne(cnorm * x0));
    const float r1 = bf16_lo(f32_to_bf16_rne(cnorm * x1));
    const float qsum = wave_sum(r0 + r1);
    const float qmax = wave_max(fmaxf(fabsf(r0), fabsf(r1)));
    // scale so that max |q| lies in [2^14, 2^15): fp16 holds every value
    const int e = __builtin_amdgcn_frexp_expf(qmax);
    S.qf[2 * lane] = __builtin_amdgcn_ldexpf(r0, 15 - e);
    S.qf[2 * lane + 1] = __builtin_amdgcn_ldexpf(r1, 15 - e);
    if (lane == 0) {
      S.qsum = qsum;
      S.qexp = (float)e;
    }
  }
  __syncthreads();

  // ---- query pairs; per-position score and value parameters -------------
  if (tid < DH / 2) {
    // pair p = 4 i + j: dims 8 i + j and 8 i + j + 4, divided by 16 for odd j
    const int i = tid >> 2, j = tid & 3;
    const float f = (j & 1) ? 0.0625f : 1.0f;
    S.qp[tid] = pack_f16(S.qf[8 * i + j] * f, S.qf[8 * i + j + 4] * f);
  }
  {
    const float qsum = S.qsum;
    const int e = (int)S.qexp;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int r = tid * 4 + t;
      const bool valid = FULL || r < n;
      const int64_t rr = row0 + (FULL ? r : min(r, n - 1));
      const float skm = sm2 * fp16_bits_to_f32(ks[rr]);
      const float a = __builtin_amdgcn_ldexpf(skm, 9 + e);  // dot = 2^-24 sum q' c
      const float b = -skm * (float)kz[rr] * qsum;
      S.kab[r] = valid ? make_float2(a, b) : make_float2(0.0f, -__builtin_inff());
      S.vsz[r] = valid ? make_float2(fp16_bits_to_f32(vs[rr]), (float)vz[rr])
                       : make_float2(0.0f, 0.0f);
    }
  }
  __syncthreads();

  uint32_t qp[4][4];  // [word u][nibble j] of code words 4 qd + u
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int j = 0; j < 4; ++j) qp[u][j] = S.qp[16 * qd + 4 * u + j];

  const uint8_t* vbase = vc + row0 * (DH / 2);
  uint4 vd[NIT][2];

  // ---- scores (log2 domain); value codes issued after the first blocks ----
  float sc[NIT][2];
  float mloc = -__builtin_inff();
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    if (!FULL && it >= nact) {
      sc[it][0] = sc[it][1] = -__builtin_inff();
      continue;
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t w4[4] = {kd[it][h].x, kd[it][h].y, kd[it][h].z, kd[it][h].w};
      float d = 0.0f;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t w = w4[u], w8 = w >> 8;
        d = dot2_f16(qp[u][0], w & 0x000F000Fu, d);
        d = dot2_f16(qp[u][1], w & 0x00F000F0u, d);
        d = dot2_f16(qp[u][2], w8 & 0x000F000Fu, d);
        d = dot2_f16(qp[u][3], w8 & 0x00F000F0u, d);
      }
      d += dpp<0xB1>(d);  // quad_perm [1, 0, 3, 2]
      d += dpp<0x4E>(d);  // quad_perm [2, 3, 0, 1]
      const float2 ab = S.kab[wave * WROWS + it * 32 + h * 16 + rg];
      sc[it][h] = __builtin_fmaf(ab.x, d, ab.y);
      mloc = fmaxf(mloc, sc[it][h]);
    }
    if (FULL && it == 1) {
#pragma unroll
      for (int jt = 0; jt < NIT; ++jt)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          vd[jt][h] =
              *reinterpret_cast<const uint4*>(vbase + (uint32_t)(row(jt, h) * (DH / 2) + qd * 16));
    }
  }
  if (!FULL) {
#pragma unroll
    for (int jt = 0; jt < NIT; ++jt)
      if (jt < nact)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          vd[jt][h] =
              *reinterpret_cast<const uint4*>(vbase + (uint32_t)(row(jt, h) * (DH / 2) + qd * 16));
  }
  mloc = wave_max(mloc);
  if (lane == 0) S.red[0][wave] = mloc;
  __syncthreads();
  const float m = fmaxf(fmaxf(S.red[0][0], S.red[0][1]), fmaxf(S.red[0][2], S.red[0][3]));

  // ---- weights p sv as fp16 pairs (rows rg, rg + 16 of each block) --------
  uint32_t wp[NIT];
  float lsum = 0.0f, zsum = 0.0f;
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    float wf[2], zv[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float p = __builtin_amdgcn_exp2f(sc[it][h] - m);
      const float2 sz = S.vsz[wave * WROWS + it * 32 + h * 16 + rg];
      wf[h] = p * sz.x;
      zv[h] = sz.y;
      lsum += p;
    }
    wp[it] = pack_f16(wf[0], wf[1]);
    const f16x2_t wh = __builtin_bit_cast(f16x2_t, wp[it]);
    zsum = __builtin_fmaf((float)wh.x, zv[0], zsum);
    zsum = __builtin_fmaf((float)wh.y, zv[1], zsum);
  }

  // ---- values: acc[8 u + k] is dimension 32 qd + 8 u + k ------------------
  float acc[32];
#pragma unroll
  for (int k = 0; k < 32; ++k) acc[k] = 0.0f;
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    if (!FULL && it >= nact) continue;
    const uint32_t a4[4] = {vd[it][0].x, vd[it][0].y, vd[it][0].z, vd[it][0].w};
    const uint32_t b4[4] = {vd[it][1].x, vd[it][1].y, vd[it][1].z, vd[it][1].w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      // bytes (A.b0, A.b1, B.b0, B.b1) and (A.b2, A.b3, B.b2, B.b3)
      const uint32_t x0 = __builtin_amdgcn_perm(b4[u], a4[u], 0x05040100u);
      const uint32_t x1 = __builtin_amdgcn_perm(b4[u], a4[u], 0x07060302u);
      const uint32_t x08 = x0 >> 8, x18 = x1 >> 8;
      acc[8 * u + 0] = dot2_f16(wp[it], x0 & 0x000F000Fu, acc[8 * u + 0]);
      acc[8 * u + 1] = dot2_f16(wp[it], x0 & 0x00F000F0u, acc[8 * u + 1]);
      acc[8 * u + 2] = dot2_f16(wp[it], x08 & 0x000F000Fu, acc[8 * u + 2]);
      acc[8 * u + 3] = dot2_f16(wp[it], x08 & 0x00F000F0u, acc[8 * u + 3]);
      acc[8 * u + 4] = dot2_f16(wp[it], x1 & 0x000F000Fu, acc[8 * u + 4]);
      acc[8 * u + 5] = dot2_f16(wp[it], x1 & 0x00F000F0u, acc[8 * u + 5]);
      acc[8 * u + 6] = dot2_f16(wp[it], x18 & 0x000F000Fu, acc[8 * u + 6]);
      acc[8 * u + 7] = dot2_f16(wp[it], x18 & 0x00F000F0u, acc[8 * u + 7]);
    }
  }

  // ---- reductions: the 4 row groups of a DPP row, then rows and waves -----
#pragma unroll
  for (int k = 0; k < 32; ++k) {
    acc[k] += dpp<0x124>(acc[k]);  // row_ror:4
    acc[k] += dpp<0x128>(acc[k]);  // row_ror:8
  }
  if ((lane & 12) == 0) {
    float* dst = &S.o[wave][lane >> 4][32 * qd];
#pragma unroll
    for (int k = 0; k < 32; k += 4)
      *reinterpret_cast<float4*>(dst + k) = make_float4(acc[k], acc[k + 1], acc[k + 2], acc[k + 3]);
  }
  // the 4 lanes of a quad counted the same positions
  lsum = 0.25f * wave_sum(lsum);
  zsum = 0.25f * wave_sum(zsum);
  if (lane == 0) {
    S.red[1][wave] = lsum;
    S.red[2][wave] = zsum;
  }
  __syncthreads();
  if (tid < DH) {
    float o = 0.0f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w)
#pragma unroll
      for (int r = 0; r < 4; ++r) o += S.o[w][r][tid];
    // codes entered as c 2^-24 (even dims) or 16 c 2^-24 (odd dims)
    o *= (tid & 1) ? 0x1p20f : 0x1p24f;
    const float zw = S.red[2][0] + S.red[2][1] + S.red[2][2] + S.red[2][3];
    rec[2 + tid] = o - zw;
  }
  if (tid == 0) {
    rec[0] = m;
    rec[1] = S.red[1][0] + S.red[1][1] + S.red[1][2] + S.red[1][3];
  }
}

// ---------------------------------------------------------------------------
// Grouped heads together: one workgroup per (key/value head, chunk) serves
// the G query heads that share it, so each code word is loaded and unpacked
// once for all of them.  Scores: on the matrix cores, one 16x16x32 fp16
// product per 16 positions and 32 dims, the key codes as fp16 subnormals
// (the same exact products as the dot2 path above, each query scaled by its
// own power of two), the G queries as columns of the other operand (the
// remaining columns zero: the matrix cores still take far fewer cycles than
// the G dot2 chains).  Weights: per pair of adjacent positions and query,
// fp16 pairs in LDS.  Values: on the matrix cores too, the weights as the
// row operand and the value codes of 8 positions per lane (two rows'
// bytes interleaved by a permute, then masked) as the column operand.
constexpr int CHG = 512;        // positions per grouped-head workgroup
constexpr int GROWS = CHG / WAVES;
constexpr int GNK = GROWS / 16;  // groups of 16 positions per wave

// Workgroup barrier for LDS traffic only: global loads still in flight stay
// in flight (a full barrier would first wait for them).
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

typedef _Float16 h8v_t __attribute__((ext_vector_type(8)));
typedef float f4v_t __attribute__((ext_vector_type(4)));

template <int G>
struct alignas(16) GqaSmem {
  float qf[G][DH];
  uint32_t qp[G][DH / 2];
  float qsum[G], qexp[G];
  float2 kab[CHG];          // (sm2 sk, -sm2 sk zk)
  float2 vsz[CHG];          // (sv, zv)
  float sc[G][CHG];         // scores, log2 domain
  uint32_t wp[G][CHG / 2];  // fp16 weight pairs of positions (2k, 2k + 1)
  float red[3][G][WAVES];   // per wave: max, sum p, sum w zv
  float o[WAVES][G][DH];    // per wave partial outputs
};

template <int G, bool FULL>
__device__ __forceinline__ void gqa_chunk(GqaSmem<G>& S, const uint16_t* __restrict__ q,
                                          const uint8_t* __restrict__ kc,
                                          const uint16_t* __restrict__ ks,
                                          const int16_t* __restrict__ kz,
                                          const uint8_t* __restrict__ vc,
                                          const uint16_t* __restrict__ vs,
                                          const int16_t* __restrict__ vz, int64_t row0, int kvh,
                                          int n, float sm2, float cnorm, float* __restrict__ ws,
                                          int nchunk, int chunk) {
  const int tid = (int)__builtin_amdgcn_workitem_id_x();
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int pr = lane & 15, kq = lane >> 4;
  const int nact = FULL ? GNK : min(GNK, max(0, (n - wave * GROWS + 15) / 16));

  // ---- first the small loads: the query (waves < G) and the scale and
  // zero-point of two positions per thread.  Loads complete in issue order,
  // so their uses below wait for them alone while the code words requested
  // after them are still in flight.
  // (every wave loads a query, waves past G a copy, so that no branch
  // holds the load and its first use together)
  const uint16_t* qh = q + ((int64_t)kvh * G + wave % G) * DH;
  const uint32_t qlo = qh[2 * lane], qhi = qh[2 * lane + 1];
  constexpr int PPT = CHG / THREADS;  // positions per thread for the parameters
  uint16_t ksr[PPT], vsr[PPT];
  int16_t kzr[PPT], vzr[PPT];
#pragma unroll
  for (int t = 0; t < PPT; ++t) {
    const int r = tid * PPT + t;
    const int64_t rr = row0 + (FULL ? r : min(r, n - 1));
    ksr[t] = ks[rr];
    kzr[t] = kz[rr];
    vsr[t] = vs[rr];
    vzr[t] = vz[rr];
  }

  // ---- key codes: lane (position pr of a group of 16, quarter kq of its row)
  const uint8_t* kbase = kc + row0 * (DH / 2);
  uint4 kd[GNK];
#pragma unroll
  for (int gi = 0; gi < GNK; ++gi)
    if (FULL || gi < nact) {
      const int r = wave * GROWS + gi * 16 + pr;
      kd[gi] = *reinterpret_cast<const uint4*>(kbase + (uint32_t)((FULL ? r : min(r, n - 1)) *
                                                                  (DH / 2) + kq * 16));
    }

  // ---- value codes: lane (word dg = pr of the row, positions 8 kq .. 8 kq + 7
  // of each block of 32) -----------------------------------------------------
  // Requested with the key codes, so that they arrive while the scores are
  // formed.  Rows past the chunk's end read the last row (their weights are
  // zero); blocks wholly past it are skipped.
  constexpr int VB = GROWS / 32;  // blocks of 32 positions per wave
  const int nvb = FULL ? VB : min(VB, max(0, (n - wave * GROWS + 31) / 32));
  const uint32_t* vrow = reinterpret_cast<const uint32_t*>(vc + row0 * (DH / 2)) + pr;
  uint32_t vv[VB][8];
#pragma unroll
  for (int bk = 0; bk < VB; ++bk)
    if (FULL || bk < nvb)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int r = wave * GROWS + bk * 32 + 8 * kq + i;
        vv[bk][i] = vrow[(int64_t)(FULL ? r : min(r, n - 1)) * (DH / 8)];
      }

  // ---- queries: wave w rotates query w --------------------------------------
  if (wave < G) {
    const float a = bf16_lo(qlo), b = bf16_lo(qhi);
    float x0 = a + b, x1 = a - b;
#pragma unroll
    for (int s = 0; s < 6; ++s) {
      const float y0 = __shfl_xor(x0, 1 << s), y1 = __shfl_xor(x1, 1 << s);
      const bool up = (lane >> s) & 1;
      x0 = up ? y0 - x0 : x0 + y0;
      x1 = up ? y1 - x1 : x1 + y1;
    }
    const float r0 = bf16_lo(f32_to_bf16_rne(cnorm * x0));
    const float r1 = bf16_lo(f32_to_bf16_rne(cnorm * x1));
    const float qsum = wave_sum(r0 + r1);
    const float qmax = wave_max(fmaxf(fabsf(r0), fabsf(r1)));
    const int e = __builtin_amdgcn_frexp_expf(qmax);
    S.qf[wave][2 * lane] = __builtin_amdgcn_ldexpf(r0, 15 - e);
    S.qf[wave][2 * lane + 1] = __builtin_amdgcn_ldexpf(r1, 15 - e);
    if (lane == 0) {
      S.qsum[wave] = qsum;
      S.qexp[wave] = (float)e;
    }
  }
  lds_sync();
  if (tid < 64 * G) {
    const int gq = tid >> 6, p = tid & 63;
    const int i = p >> 2, j = p & 3;
    const float f = (j & 1) ? 0.0625f : 1.0f;
    S.qp[gq][p] = pack_f16(S.qf[gq][8 * i + j] * f, S.qf[gq][8 * i + j + 4] * f);
  }
#pragma unroll
  for (int t = 0; t < PPT; ++t) {
    const int r = tid * PPT + t;
    const float skm = sm2 * fp16_bits_to_f32(ksr[t]);
    S.kab[r] = make_float2(skm, -skm * (float)kzr[t]);
    S.vsz[r] = (FULL || r < n) ? make_float2(fp16_bits_to_f32(vsr[t]), (float)vzr[t])
                               : make_float2(0.0f, 0.0f);
  }
  lds_sync();

  // ---- scores on the matrix cores --------------------------------------------
  // A 16x16x32 fp16 product per group of 16 positions and word j of each
  // row quarter: A = the key codes (row = position pr, the 8 dims of word j
  // of quarter kq, unpacked by masks into fp16 subnormals c 2^-24 in the
  // order d0 d4 16d1 16d5 d2 d6 16d3 16d7), B = the queries in the same
  // order (column = query, zero past G; the odd dims pre-scaled by 1/16 in
  // qp).  Lane (pr, kq) ends with query pr's dots of positions 4 kq .. 4 kq + 3
  // of the group; every product is exact in fp32, as in the dot2 path.
  h8v_t qb[4];
  float cq = 0.0f, qs = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j) qb[j] = h8v_t{};
  if (pr < G) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      qb[j] = __builtin_bit_cast(h8v_t, *reinterpret_cast<const uint4*>(&S.qp[pr][16 * kq + 4 * j]));
    cq = __builtin_amdgcn_ldexpf(1.0f, 9 + (int)S.qexp[pr]);  // dot = 2^-24 sum q' c
    qs = S.qsum[pr];
  }
  float mloc = -__builtin_inff();
#pragma unroll
  for (int gi = 0; gi < GNK; ++gi) {
    const int rb = wave * GROWS + gi * 16 + 4 * kq;  // this lane's first position
    if (!FULL && gi >= nact) {
      if (pr < G)
        *reinterpret_cast<float4*>(&S.sc[pr][rb]) =
            make_float4(-__builtin_inff(), -__builtin_inff(), -__builtin_inff(), -__builtin_inff());
      continue;
    }
    const uint32_t w4[4] = {kd[gi].x, kd[gi].y, kd[gi].z, kd[gi].w};
    f4v_t d = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t w = w4[j], w8 = w >> 8;
      const uint4 a = make_uint4(w & 0x000F000Fu, w & 0x00F000F0u, w8 & 0x000F000Fu,
                                 w8 & 0x00F000F0u);
      d = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8v_t, a), qb[j], d, 0, 0, 0);
    }
    const float4 ab01 = *reinterpret_cast<const float4*>(&S.kab[rb]);
    const float4 ab23 = *reinterpret_cast<const float4*>(&S.kab[rb + 2]);
    const float ax[4] = {ab01.x, ab01.z, ab23.x, ab23.z}, ay[4] = {ab01.y, ab01.w, ab23.y, ab23.w};
    float sg[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      sg[r] = __builtin_fmaf(ax[r] * cq, d[r], ay[r] * qs);
      if (!FULL && rb + r >= n) sg[r] = -__builtin_inff();
      mloc = fmaxf(mloc, sg[r]);
    }
    if (pr < G) *reinterpret_cast<float4*>(&S.sc[pr][rb]) = make_float4(sg[0], sg[1], sg[2], sg[3]);
  }
  mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
  mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
  if (lane < G) S.red[0][lane][wave] = mloc;
  lds_sync();

  // ---- weights: fp16 pairs per (position pair, query) ------------------------
  float m[G];
#pragma unroll
  for (int gq = 0; gq < G; ++gq)
    m[gq] = fmaxf(fmaxf(S.red[0][gq][0], S.red[0][gq][1]), fmaxf(S.red[0][gq][2], S.red[0][gq][3]));
  float lsum[G], zsum[G];
#pragma unroll
  for (int gq = 0; gq < G; ++gq) lsum[gq] = zsum[gq] = 0.0f;
#pragma unroll
  for (int t = 0; t < CHG / 2 / THREADS; ++t) {
    const int k = tid + t * THREADS;
    const float2 sz0 = S.vsz[2 * k], sz1 = S.vsz[2 * k + 1];
#pragma unroll
    for (int gq = 0; gq < G; ++gq) {
      const float p0 = __builtin_amdgcn_exp2f(S.sc[gq][2 * k] - m[gq]);
      const float p1 = __builtin_amdgcn_exp2f(S.sc[gq][2 * k + 1] - m[gq]);
      const uint32_t w = pack_f16(p0 * sz0.x, p1 * sz1.x);
      S.wp[gq][k] = w;
      const f16x2_t wh = __builtin_bit_cast(f16x2_t, w);
      lsum[gq] += p0 + p1;
      zsum[gq] = __builtin_fmaf((float)wh.x, sz0.y, zsum[gq]);
      zsum[gq] = __builtin_fmaf((float)wh.y, sz1.y, zsum[gq]);
    }
  }
#pragma unroll
  for (int gq = 0; gq < G; ++gq) {
    const float l = wave_sum(lsum[gq]), z = wave_sum(zsum[gq]);
    if (lane == 0) {
      S.red[1][gq][wave] = l;
      S.red[2][gq][wave] = z;
    }
  }
  lds_sync();

  // ---- values on the matrix cores -------------------------------------------
  // O[q][8 dg + m] = sum over positions of W[q][pos] V[pos][8 dg + m]: one
  // 16x16x32 fp16 product per block of 32 positions and nibble m of the code
  // words.  A = the weights (row = query pr, zero past G; positions
  // 8 kq .. 8 kq + 7 of the block, the fp16 pairs of wp), B = the value codes
  // (column = word dg = pr, the same positions in pairs: the bytes of two
  // rows interleaved by a permute, nibble m masked out as fp16 subnormals,
  // 16 times the code for odd m).  Lanes 0..15 end with dims 8 dg + m of the
  // queries 0..3 (their rows of the product).
  f4v_t oacc[8];
#pragma unroll
  for (int m = 0; m < 8; ++m) oacc[m] = f4v_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int bk = 0; bk < VB; ++bk) {
    if (!FULL && bk >= nvb) continue;
    const int p0 = wave * GROWS + bk * 32 + 8 * kq;
    h8v_t aw = h8v_t{};
    if (pr < G) aw = __builtin_bit_cast(h8v_t, *reinterpret_cast<const uint4*>(&S.wp[pr][p0 / 2]));
    uint32_t xs[4][4];  // per position pair: bytes 0-1 of both rows, >> 8, bytes 2-3, >> 8
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t x0 = __builtin_amdgcn_perm(vv[bk][2 * i + 1], vv[bk][2 * i], 0x05040100u);
      const uint32_t x1 = __builtin_amdgcn_perm(vv[bk][2 * i + 1], vv[bk][2 * i], 0x07060302u);
      xs[i][0] = x0;
      xs[i][1] = x0 >> 8;
      xs[i][2] = x1;
      xs[i][3] = x1 >> 8;
    }
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const uint32_t mask = (m & 1) ? 0x00F000F0u : 0x000F000Fu;
      const uint4 bv = make_uint4(xs[0][m >> 1] & mask, xs[1][m >> 1] & mask,
                                  xs[2][m >> 1] & mask, xs[3][m >> 1] & mask);
      oacc[m] = __builtin_amdgcn_mfma_f32_16x16x32_f16(aw, __builtin_bit_cast(h8v_t, bv), oacc[m],
                                                       0, 0, 0);
    }
  }
  if (lane < 16) {
#pragma unroll
    for (int gq = 0; gq < G; ++gq) {
      float* dst = &S.o[wave][gq][8 * pr];
      *reinterpret_cast<float4*>(dst) =
          make_float4(oacc[0][gq], oacc[1][gq], oacc[2][gq], oacc[3][gq]);
      *reinterpret_cast<float4*>(dst + 4) =
          make_float4(oacc[4][gq], oacc[5][gq], oacc[6][gq], oacc[7][gq]);
    }
  }
  __syncthreads();
  for (int e = tid; e < G * DH; e += THREADS) {
    const int gq = e / DH, dd = e - gq * DH;
    float o = S.o[0][gq][dd] + S.o[1][gq][dd] + S.o[2][gq][dd] + S.o[3][gq][dd];
    o *= (dd & 1) ? 0x1p20f : 0x1p24f;  // codes entered as c 2^-24 / 16 c 2^-24
    const float zw = S.red[2][gq][0] + S.red[2][gq][1] + S.red[2][gq][2] + S.red[2][gq][3];
    float* rec = ws + (((int64_t)kvh * G + gq) * nchunk + chunk) * WS_FLOATS;
    rec[2 + dd] = o - zw;
    if (dd == 0) {
      rec[0] = fmaxf(fmaxf(S.red[0][gq][0], S.red[0][gq][1]), fmaxf(S.red[0][gq][2], S.red[0][gq][3]));
      rec[1] = S.red[1][gq][0] + S.red[1][gq][1] + S.red[1][gq][2] + S.red[1][gq][3];
    }
  }
}

template <int G>
__global__ __launch_bounds__(THREADS) __attribute__((amdgpu_waves_per_eu(4))) void kv_attention_gqa_kernel(
    const uint16_t* __restrict__ q, const uint8_t* __restrict__ kc, const uint16_t* __restrict__ ks,
    const int16_t* __restrict__ kz, const uint8_t* __restrict__ vc, const uint16_t* __restrict__ vs,
    const int16_t* __restrict__ vz, int64_t S_cap, int seq_len, int nchunk, int units, float sm2,
    float cnorm, float* __restrict__ ws) {
  __shared__ GqaSmem<G> S;
  const int unit = (int)__builtin_amdgcn_workgroup_id_x();
  if (unit >= units) return;
  // The short final chunks (seq_len not a multiple of CHG) take the lowest
  // ids, then the full chunks of every key/value head.  Workgroups start in
  // id order: the short ones finish within a few microseconds and free their
  // slots early, instead of running as a tail after the full ones (context
  // 4096 + 1 at 128 key/value heads: 128 one-position chunks, then 1024 full
  // ones, four resident per CU).
  const int nfull = seq_len / CHG;
  const int nkv = units / nchunk;
  const int nshort = units - nkv * nfull;  // nkv or 0
  int kvh, chunk;
  if (unit < nshort) {
    kvh = unit;
    chunk = nfull;
  } else {
    kvh = (unit - nshort) / nfull;
    chunk = unit - nshort - kvh * nfull;
  }
  const int j0 = chunk * CHG;
  const int n = min(CHG, seq_len - j0);
  const int64_t row0 = (int64_t)kvh * S_cap + j0;
  if (n == CHG)
    gqa_chunk<G, true>(S, q, kc, ks, kz, vc, vs, vz, row0, kvh, n, sm2, cnorm, ws, nchunk, chunk);
  else
    gqa_chunk<G, false>(S, q, kc, ks, kz, vc, vs, vz, row0, kvh, n, sm2, cnorm, ws, nchunk, chunk);
}

__global__ __launch_bounds__(THREADS) void kv_attention_chunk_kernel(
    const uint16_t* __restrict__ q, const uint8_t* __restrict__ kc, const uint16_t* __restrict__ ks,
    const int16_t* __restrict__ kz, const uint8_t* __restrict__ vc, const uint16_t* __restrict__ vs,
    const int16_t* __restrict__ vz, int64_t S_cap, int seq_len, int nchunk, int units, int group,
    float sm2, float cnorm, float* __restrict__ ws) {
  __shared__ ChunkSmem S;
  // Workgroups go to the 8 XCDs round-robin by id.  The `group` query heads
  // that read one key/value chunk get ids 8 apart, i.e. the same XCD at about
  // the same time, so the chunk comes from HBM once and from that XCD's L2
  // for the others.  Work unit u = (key/value head, chunk); ids past the
  // units (padding to a multiple of 8) exit.
  const int blk = (int)__builtin_amdgcn_workgroup_id_x();
  const int slot = blk >> 3;
  const int gq = slot % group;
  const int unit = (slot / group) * 8 + (blk & 7);
  if (unit >= units) return;
  const int kvh = unit / nchunk, chunk = unit - kvh * nchunk;  // kvh = b * Hkv + h_kv
  const int bh = kvh * group + gq;                              // query head b * Hq + h
  const int j0 = chunk * CH;
  const int n = min(CH, seq_len - j0);  // positions of this chunk (>= 1)
  const int64_t row0 = (int64_t)kvh * S_cap + j0;
  float* rec = ws + ((int64_t)bh * nchunk + chunk) * WS_FLOATS;
  if (n == CH)
    attention_chunk<true>(S, q, kc, ks, kz, vc, vs, vz, row0, bh, n, sm2, cnorm, rec);
  else
    attention_chunk<false>(S, q, kc, ks, kz, vc, vs, vz, row0, bh, n, sm2, cnorm, rec);
}

// Pass 2: merge the chunk records of one (b, h).  The chunk maxima are read
// by all lanes at once (a chain of dependent loads over the chunks would cost
// far more than the data), the factors 2^(m_i - m) go through LDS, and every
// thread then sums its dimension over the chunks with independent loads.
constexpr int CT = 1024;  // chunk factors held in LDS per round

// QUANT: the head's output row, rounded to bf16, is also quantized as one
// group of the quantizer (Eq. 1, no rotation): codes two per byte (element
// 2k in the low nibble), fp16 scale and int16 zero-point per (b, h), the
// layout offq_rotate_quantize writes for a [B, Hq * 128] input with g = 128;
// out may then be NULL.
template <bool QUANT>
__global__ __launch_bounds__(DH) void kv_attention_combine_kernel(
    const float* __restrict__ ws, int nchunk, int v_had, float cnorm, uint16_t* __restrict__ out,
    uint8_t* __restrict__ qcodes, uint16_t* __restrict__ qscale, int16_t* __restrict__ qzero) {
  __shared__ float s_e[CT];
  __shared__ float s_red[2][DH / 64];
  __shared__ float s_o[DH];
  const int d = (int)__builtin_amdgcn_workitem_id_x();
  const int lane = d & 63, wave = d >> 6;
  const int bh = (int)__builtin_amdgcn_workgroup_id_x();
  const float* w = ws + (int64_t)bh * nchunk * WS_FLOATS;

  float m = -__builtin_inff();
  for (int i = d; i < nchunk; i += DH) m = fmaxf(m, w[(int64_t)i * WS_FLOATS]);
  m = wave_max(m);
  if (lane == 0) s_red[0][wave] = m;
  __syncthreads();
  m = fmaxf(s_red[0][0], s_red[0][1]);

  float l = 0.0f, o = 0.0f;
  for (int i0 = 0; i0 < nchunk; i0 += CT) {
    const int nt = min(CT, nchunk - i0);
    __syncthreads();  // the previous round's factors are consumed
    for (int i = d; i < nt; i += DH) {
      const float* r = w + (int64_t)(i0 + i) * WS_FLOATS;
      const float e = __builtin_amdgcn_exp2f(r[0] - m);
      s_e[i] = e;
      l = __builtin_fmaf(e, r[1], l);
    }
    __syncthreads();
    const float* od = w + (int64_t)i0 * WS_FLOATS + 2 + d;
    int i = 0;
    for (; i + 8 <= nt; i += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = od[(int64_t)(i + u) * WS_FLOATS];
#pragma unroll
      for (int u = 0; u < 8; ++u) o = __builtin_fmaf(s_e[i + u], v[u], o);
    }
    for (; i < nt; ++i) o = __builtin_fmaf(s_e[i], od[(int64_t)i * WS_FLOATS], o);
  }
  l = wave_sum(l);
  if (lane == 0) s_red[1][wave] = l;
  __syncthreads();
  l = s_red[1][0] + s_red[1][1];
  o = o / l;
  if (v_had) {
    s_o[d] = o;
    __syncthreads();
    float a = 0.0f;
    for (int i = 0; i < DH; ++i)
      a = __builtin_fmaf(s_o[i], (__builtin_popcount(i & d) & 1) ? -1.0f : 1.0f, a);
    o = a * cnorm;
  }
  const uint16_t ob = f32_to_bf16_rne(o);
  if (out) out[(int64_t)bh * DH + d] = ob;
  if constexpr (QUANT) {
    const float y = bf16_lo(ob);
    const float mx = wave_max(y), mn = wave_min(y);
    __syncthreads();  // s_red's sums are consumed
    if (lane == 0) {
      s_red[0][wave] = mx;
      s_red[1][wave] = mn;
    }
    __syncthreads();
    const QParams P = quant_params(fmaxf(s_red[0][0], s_red[0][1]), fminf(s_red[1][0], s_red[1][1]));
    const uint32_t c = quant_bits(y, P) - __float_as_uint(P.lo);  // the code, 0..15
    const uint32_t c1 = __shfl_down(c, 1);                         // element d + 1's
    if (!(d & 1)) qcodes[(int64_t)bh * (DH / 2) + (d >> 1)] = (uint8_t)(c | (c1 << 4));
    if (d == 0) {
      qscale[bh] = P.s16;
      qzero[bh] = P.z;
    }
  }
}

}  // namespace

int64_t kv_attention_workspace_floats(int64_t BH, int64_t seq_len) {
  // one record per (query head, chunk); the grouped-head path uses the
  // smaller chunks, so their count bounds both paths
  return BH * ((seq_len + CHG - 1) / CHG) * WS_FLOATS;
}

hipError_t launch_kv_attention_decode(const uint16_t* q, const uint8_t* k_codes,
                                      const uint16_t* k_scale, const int16_t* k_zero,
                                      const uint8_t* v_codes, const uint16_t* v_scale,
                                      const int16_t* v_zero, int64_t BH, int64_t group,
                                      int64_t S_cap, int64_t seq_len, float sm_scale,
                                      bool v_hadamard, uint16_t* out, uint8_t* qcodes,
                                      uint16_t* qscale, int16_t* qzero, float* workspace,
                                      hipStream_t stream) {
  const float cnorm = (float)(1.0 / __builtin_sqrt((double)DH));
  auto combine = [&](int nchunk) {
    if (qcodes)
      hipLaunchKernelGGL(kv_attention_combine_kernel<true>, dim3((unsigned)BH), dim3(DH), 0, stream,
                         workspace, nchunk, v_hadamard ? 1 : 0, cnorm, out, qcodes, qscale, qzero);
    else
      hipLaunchKernelGGL(kv_attention_combine_kernel<false>, dim3((unsigned)BH), dim3(DH), 0,
                         stream, workspace, nchunk, v_hadamard ? 1 : 0, cnorm, out, nullptr,
                         nullptr, nullptr);
  };
  if (group == 2 || group == 4) {
    const int nchunk = (int)((seq_len + CHG - 1) / CHG);
    const int64_t units = BH / group * nchunk;  // (key/value head, chunk) pairs
    // the query heads of a key/value head in one workgroup
#define OFFQ_GQA(G_)                                                                        \
  hipLaunchKernelGGL(kv_attention_gqa_kernel<G_>, dim3((unsigned)units), dim3(THREADS), 0,  \
                     stream, q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, S_cap, \
                     (int)seq_len, nchunk, (int)units, sm_scale * LOG2E, cnorm, workspace)
    if (group == 2) OFFQ_GQA(2);
    else OFFQ_GQA(4);
#undef OFFQ_GQA
    combine(nchunk);
  } else {
    const int nchunk = (int)((seq_len + CH - 1) / CH);
    const int64_t units = BH / group * nchunk;  // (key/value head, chunk) pairs
    const int64_t grid = (units + 7) / 8 * 8 * group;
    hipLaunchKernelGGL(kv_attention_chunk_kernel, dim3((unsigned)grid), dim3(THREADS), 0, stream,
                       q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, S_cap, (int)seq_len,
                       nchunk, (int)units, (int)group, sm_scale * LOG2E, cnorm, workspace);
    combine(nchunk);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// The same step for callers that cannot allocate: the chunk records live in a
// file-scope device array instead of a caller-owned workspace.  Host code
// never passes the array's name to a kernel (on the host it only names the
// symbol); it passes the device address hipGetSymbolAddress returns, looked
// up once per device with that device current.  Every call on a device shares
// that device's array: calls that overlap on one device race.  Nothing in it
// needs to start at zero: pass 1 writes every record that pass 2 reads.
namespace {

static __device__ __align__(256) float scratch[kKvScratchBytes / sizeof(float)];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

hipError_t kv_attention_scratch(float** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = static_cast<float*>(p);
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace offq
