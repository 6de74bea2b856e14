// Causal prefill attention over the 4-bit KV cache (gfx950).
//
// The prefill of T new tokens per sequence: query t sits at position past + t
// and attends to cache positions 0 .. past + t (the cache already holds the
// T new rows, written by the RoPE + KV4 step).  Per row the arithmetic is
// that of the decode kernel (sec. 3.3 step 2(3): the query meets the keys in
// the H3-rotated basis; sec. 4.2: one quantizer group per cache row):
//
//   q_r  = bf16_rne(fl32(c * fl32(H q)))             c = fl32(1 / sqrt(128))
//   s_j  = sm_scale * sk_j * (sum_d q_r[d] ck_j[d] - zk_j sum_d q_r[d])
//   o[d] = (sum_j w_j cv_j[d] - sum_j w_j zv_j) / sum_j p_j,
//          p_j = 2^(s_j log2 e - m),  w_j = fp16(p_j sv_j)
//   (then c * H o if asked)
//
// With many queries per key the work is a dense contraction, so both
// products run on the fp16 MFMA (v_mfma_f32_32x32x16_f16):
// * the 4-bit codes enter as fp16 subnormals: an AND of a code word leaves
//   the code c (or 16 c) in a 16-bit half, which is the fp16 value c 2^-24;
//   the matrix cores take subnormal inputs exactly, so every product
//   q c 2^-24 is exact in fp32 and unpacking costs one AND per two codes;
// * scores are formed transposed, S^T = K Q^T (keys x queries): a lane
//   holds 16 keys of one query per 32 x 32 tile, so the softmax max and sum
//   run inside the lane plus one exchange with lane ^ 32, and the tile is
//   already in the operand layout of the next product, O^T = V^T W^T;
// * per-key parameters (score slope and offset, sv, zv) reach the lane that
//   needs them through DPP row_newbcast, folded into the arithmetic
//   instruction that uses them;
// * K and V are unpacked once per workgroup into LDS as fp16 code values,
//   K in the operand order of the score product, V transposed (keys
//   permuted to match the accumulator rows of S^T), shared by all waves.
//
// Organisation: one workgroup of 8 waves per (sequence b, kv head, 256 / G
// query positions); wave w takes query head w % G of the kv head
// (grouped-query attention) at the 32 positions of sub-tile w / G, so a
// staged key block serves 256 queries and its staging work is split over
// 512 threads (keys in one half, values in the other).  Keys stream in
// blocks of 64 through a double-buffered LDS stage; a wave skips the blocks
// past its last query and masks the diagonal ones, and takes a block's two
// 32-key tiles one after the other (the first tile's softmax runs while the
// second tile's score products are on the matrix cores).  The output rescale
// is lazy: a row's reference maximum moves only when a tile's maximum passes
// it by more than tau (at most 8, and small enough that every weight p sv
// stays finite in fp16).  Workgroups with the most keys launch first.
#include <type_traits>

#include "common.h"
#include "internal.h"

namespace offq {
namespace {

constexpr int PD = 128;     // head dimension
constexpr int KB = 64;      // keys per block
constexpr int KROW = 272;   // LDS bytes per key row: 128 fp16 code values + 16 padding
constexpr int VROW = 144;   // LDS bytes per dimension row of V^T (64 fp16 + 16 padding)
constexpr float PLOG2E = 1.4426950408889634f;
constexpr float TAU = 8.0f;  // lazy rescaling: a reference maximum may lag by up to 2^8

typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef float f16v_t __attribute__((ext_vector_type(16)));

struct Stage {
  uint8_t k[KB * KROW];   // key codes as fp16 c 2^-24 (16 c 2^-24), operand order
  uint8_t vt[PD * VROW];  // V^T: per dimension, the 64 keys' codes as fp16 c 2^-24
  float4 sc[KB];          // per key: (score slope, score offset / sum q, sv, zv)
  float tau;              // how far a row maximum may pass its reference unrescaled
};

__device__ __forceinline__ uint32_t pk_f16(float a, float b) {
  const h2_t h = {(_Float16)a, (_Float16)b};
  return __builtin_bit_cast(uint32_t, h);
}

// The value lane 16 (lane / 16) + R holds: each row of 16 lanes reads its own
// lane R (gfx90a+ DPP row_newbcast).
template <int R>
__device__ __forceinline__ float bcast(float v) {
  return __builtin_bit_cast(float,
                            __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x150 + R, 0xf, 0xf, true));
}

// position of key k of a block inside V^T's rows: key 16 a + 8 b + 4 h + i
// sits at 16 a + 8 h + 4 b + i, so that the 8 keys lane half h of the value
// product needs for k-step a are 8 consecutive fp16
__device__ __forceinline__ int vt_pos(int k) {
  return (k & ~15) | ((k & 4) << 1) | ((k & 8) >> 1) | (k & 3);
}

#define PF_FOR16(X) X(0) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15)

template <int G>
__global__ __launch_bounds__(512, 1) void kv_prefill_kernel(
    const uint16_t* __restrict__ q, int B, int T, int Hq, int Hkv, int past,
    const uint8_t* __restrict__ kc, const uint16_t* __restrict__ ks,
    const int16_t* __restrict__ kz, const uint8_t* __restrict__ vc,
    const uint16_t* __restrict__ vs, const int16_t* __restrict__ vz, int64_t s_cap, float sm2,
    float cnorm, int v_had, uint16_t* __restrict__ out) {
  constexpr int NW = 8;
  constexpr int TP = 32 * NW / G;  // query positions per workgroup
  __shared__ Stage st[2];
  __shared__ float red[NW];

  const int tid = (int)__builtin_amdgcn_workitem_id_x();
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int gq = wave % G, ps = wave / G;
  const int h = lane >> 5, ql = lane & 31;

  const int nbh = B * Hkv;
  const int ntile = (T + TP - 1) / TP;
  const int bid = (int)__builtin_amdgcn_workgroup_id_x();
  const int tile = ntile - 1 - bid / nbh;  // the longest key ranges first
  const int bh = bid - (bid / nbh) * nbh;  // b * Hkv + kv head
  const int b = bh / Hkv, hk = bh - b * Hkv;
  const int q0 = tile * TP;
  const int nk = past + min(q0 + TP, T);  // keys the workgroup reads
  const int nb = (nk + KB - 1) / KB;
  const int tw = q0 + 32 * ps;            // the wave's first query
  const bool live = tw < T;
  const int pmin = past + tw;
  const int pmax = past + min(tw + 31, T - 1);
  const int t = min(tw + ql, T - 1);
  const int pq = past + t;                // this lane's query position
  const int hq = hk * G + gq;

  // ---- the query: FWHT (dims 64 h .. 64 h + 63 in the lane), bf16 q_r ----
  float x[64];
  {
    const uint4* src =
        reinterpret_cast<const uint4*>(q + ((int64_t)(b * T + t) * Hq + hq) * PD + 64 * h);
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const uint4 v = src[c];
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        x[8 * c + 2 * u] = bf16_lo(w[u]);
        x[8 * c + 2 * u + 1] = __uint_as_float(w[u] & 0xFFFF0000u);
      }
    }
  }
#pragma unroll
  for (int s = 1; s < 64; s <<= 1)
#pragma unroll
    for (int i = 0; i < 64; ++i)
      if (!(i & s)) {
        const float a = x[i], c = x[i + s];
        x[i] = a + c;
        x[i + s] = a - c;
      }
  float qs = 0.0f, qm = 0.0f;
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    const float p = __shfl_xor(x[i], 32);
    const float y = h ? p - x[i] : x[i] + p;
    x[i] = bf16_lo(f32_to_bf16_rne(cnorm * y));
    qs += x[i];
    qm = fmaxf(qm, fabsf(x[i]));
  }
  const float qsum = qs + __shfl_xor(qs, 32);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) qm = fmaxf(qm, __shfl_xor(qm, o));
  if (lane == 0) red[wave] = qm;
  __syncthreads();
  qm = red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) qm = fmaxf(qm, red[w]);
  // scale so that the workgroup's max |q_r| lies in [2^14, 2^15): fp16 holds
  // the bf16 values; dims meeting a high nibble (16 c) are divided by 16
  const int e = __builtin_amdgcn_frexp_expf(qm);
  uint32_t qb[8][4];  // B operand of the score product, k-step s: dims 64 h + 8 s + ...
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const float* v = x + 8 * s;
    qb[s][0] = pk_f16(__builtin_amdgcn_ldexpf(v[0], 15 - e), __builtin_amdgcn_ldexpf(v[4], 15 - e));
    qb[s][1] = pk_f16(__builtin_amdgcn_ldexpf(v[1], 11 - e), __builtin_amdgcn_ldexpf(v[5], 11 - e));
    qb[s][2] = pk_f16(__builtin_amdgcn_ldexpf(v[2], 15 - e), __builtin_amdgcn_ldexpf(v[6], 15 - e));
    qb[s][3] = pk_f16(__builtin_amdgcn_ldexpf(v[3], 11 - e), __builtin_amdgcn_ldexpf(v[7], 11 - e));
  }

  // ---- staging of one key block: keys by threads 0..255, values by 256..511 -
  const int64_t rowbase = (int64_t)bh * s_cap;
  const uint8_t* kcb = kc + rowbase * (PD / 2);
  const uint8_t* vcb = vc + rowbase * (PD / 2);
  uint4 kreg = make_uint4(0, 0, 0, 0);
  uint2 va = make_uint2(0, 0), vb = make_uint2(0, 0);
  uint16_t r_ks = 0, r_vs = 0;
  int16_t r_kz = 0, r_vz = 0;
  const int vid = tid - 256;  // value-staging thread index (0..255 for waves 4..7)
  auto load = [&](int kb) {
    const int k0 = kb * KB;
    if (tid >= 256) {
      const int kp = vid & 31, dc = vid >> 5;
      const int ka = min(k0 + 2 * kp, nk - 1), kb1 = min(k0 + 2 * kp + 1, nk - 1);
      va = *reinterpret_cast<const uint2*>(vcb + (int64_t)ka * (PD / 2) + 8 * dc);
      vb = *reinterpret_cast<const uint2*>(vcb + (int64_t)kb1 * (PD / 2) + 8 * dc);
    } else {
      const int key = min(k0 + (tid >> 2), nk - 1);
      kreg = *reinterpret_cast<const uint4*>(kcb + (int64_t)key * (PD / 2) + 16 * (tid & 3));
      if (tid < KB) {
        const int64_t r = rowbase + min(k0 + tid, nk - 1);
        r_ks = ks[r];
        r_kz = kz[r];
        r_vs = vs[r];
        r_vz = vz[r];
      }
    }
  };
  auto store = [&](int kb, Stage& S) {
    if (tid >= 256) {
      const int kp = vid & 31, dc = vid >> 5;
      uint32_t* vt = reinterpret_cast<uint32_t*>(S.vt + 16 * dc * VROW + 2 * vt_pos(2 * kp));
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const uint32_t a = u ? va.y : va.x, c = u ? vb.y : vb.x;
        // bytes (a0, a1, c0, c1) and (a2, a3, c2, c3): each AND then leaves
        // the two keys' codes of one dimension in the two fp16 halves
        const uint32_t t0 = __builtin_amdgcn_perm(c, a, 0x05040100u);
        const uint32_t t1 = __builtin_amdgcn_perm(c, a, 0x07060302u);
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          vt[(8 * u + m) * (VROW / 4)] = (t0 >> (4 * m)) & 0x000F000Fu;
          vt[(8 * u + 4 + m) * (VROW / 4)] = (t1 >> (4 * m)) & 0x000F000Fu;
        }
      }
    } else {
      // code word i of the key row (8 dims) -> the 8 fp16 operand values of
      // one k-step: (d0, d4), (16 d1, 16 d5), (d2, d6), (16 d3, 16 d7)
      uint4* kd = reinterpret_cast<uint4*>(S.k + (tid >> 2) * KROW + 64 * (tid & 3));
      const uint32_t kw4[4] = {kreg.x, kreg.y, kreg.z, kreg.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t u = kw4[i];
        kd[i] = make_uint4(u & 0x000F000Fu, u & 0x00F000F0u, (u >> 8) & 0x000F000Fu,
                           (u >> 8) & 0x00F000F0u);
      }
      if (tid < KB) {
        // log2-domain score = a dot + b sum(q_r), dot = 2^(-9-e) sum q_r c
        const bool valid = kb * KB + tid < nk;
        const float skm = sm2 * fp16_bits_to_f32(r_ks);
        const float svf = valid ? fp16_bits_to_f32(r_vs) : 0.0f;
        S.sc[tid] = valid ? make_float4(__builtin_amdgcn_ldexpf(skm, 9 + e), -skm * (float)r_kz,
                                        svf, (float)r_vz)
                          : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        // a weight p sv with p <= 2^tau stays below 65000 (finite in fp16)
        float mx = fabsf(svf);
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
        if (tid == 0) S.tau = fminf(TAU, mx > 0.0f ? __builtin_log2f(65000.0f / mx) : TAU);
      }
    }
  };

  // this lane's DPP source key within a 32-key tile: row R of the tile
  // (8 (R / 4) + 4 half + R % 4) as lane R of each row of 16 lanes sees it
  const int kap = 8 * ((lane & 15) >> 2) + 4 * (lane >> 5) + (lane & 3);

  f16v_t oacc[4];
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[d][r] = 0.0f;
  float m = -__builtin_inff(), l = 0.0f, zs = 0.0f;

  load(0);
  store(0, st[0]);
  __syncthreads();
  for (int kb = 0; kb < nb; ++kb) {
    if (kb + 1 < nb) load(kb + 1);
    const Stage& S = st[kb & 1];
    if (live && kb * KB <= pmax) {
      // ---- S^T = K Q^T: two 32-key tiles ---------------------------------
      f16v_t sacc[2];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[tt][r] = 0.0f;
      // tile 0's chain first, then tile 1's: tile 0's softmax can start
      // while tile 1's products are still on the matrix cores
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          // lane (key, half h), k-step s: code word 8 h + s of the key row
          const uint4 a = *reinterpret_cast<const uint4*>(S.k + (32 * tt + ql) * KROW +
                                                          16 * (8 * h + s));
          const uint32_t b4[4] = {qb[s][0], qb[s][1], qb[s][2], qb[s][3]};
          sacc[tt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(h8_t, a),
                                                            __builtin_bit_cast(h8_t, b4),
                                                            sacc[tt], 0, 0, 0);
        }

      // One 32-key tile: scores, causal mask, running maximum, the weights
      // w = fp16(p sv) as the B operand of O^T += V^T W^T and that product.
      // Tile by tile, so that one tile's VALU work overlaps the other's MFMAs.
      auto tile = [&](auto tile_c) {
        constexpr int TT = decltype(tile_c)::value;
        const float4 sc = S.sc[32 * TT + kap];
        float sv[16];
#define PF_SCORE(R) sv[R] = __builtin_fmaf(bcast<R>(sc.x), sacc[TT][R], bcast<R>(sc.y) * qsum);
        PF_FOR16(PF_SCORE)
#undef PF_SCORE
        if (kb * KB + 32 * TT + 31 > pmin) {
          const int kbase = kb * KB + 32 * TT + 4 * h - pq;  // key - pq = kbase + 8 (r / 4) + r % 4
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (kbase + 8 * (r >> 2) + (r & 3) > 0) sv[r] = -__builtin_inff();
        }
        float bm = sv[0];
#pragma unroll
        for (int r = 1; r < 16; ++r) bm = fmaxf(bm, sv[r]);
        bm = fmaxf(bm, __shfl_xor(bm, 32));
        // The reference m of a row only moves when the tile's maximum passes
        // it by more than tau (then every row moves to its own maximum): the
        // weights stay below 2^tau (finite in fp16 by the choice of tau),
        // their relative rounding is unchanged, and the O rescale runs rarely.
        if (__builtin_amdgcn_ballot_w64(bm > m + fmaxf(S.tau, 0.0f))) {
          const float mn = fmaxf(m, bm);
          const float f = __builtin_amdgcn_exp2f(m - mn);
#pragma unroll
          for (int d = 0; d < 4; ++d)
#pragma unroll
            for (int r = 0; r < 16; ++r) oacc[d][r] *= f;
          l *= f;
          zs *= f;
          m = mn;
        }
#define PF_WEIGHT(R)                                                          \
  {                                                                           \
    const float p = __builtin_amdgcn_exp2f(sv[R] - m);                        \
    l += p;                                                                   \
    float w = bcast<R>(sc.z) * p;                                             \
    asm volatile("" : "+v"(w)); /* keep the DPP multiply */                   \
    sv[R] = w;                                                                \
  }
        PF_FOR16(PF_WEIGHT)
#undef PF_WEIGHT
        uint32_t wb[2][4];
#pragma unroll
        for (int k = 0; k < 2; ++k)
#pragma unroll
          for (int j = 0; j < 4; ++j) wb[k][j] = pk_f16(sv[8 * k + 2 * j], sv[8 * k + 2 * j + 1]);
        // the zero-point term with the rounded weights
#define PF_ZSUM(R)                                                                    \
  {                                                                                   \
    const h2_t w2 = __builtin_bit_cast(h2_t, wb[(R) >> 3][((R) & 7) >> 1]);           \
    zs = __builtin_fmaf((float)((R) & 1 ? w2.y : w2.x), bcast<R>(sc.w), zs);          \
  }
        PF_FOR16(PF_ZSUM)
#undef PF_ZSUM
#pragma unroll
        for (int k = 0; k < 2; ++k)
#pragma unroll
          for (int d = 0; d < 4; ++d) {
            const uint4 v = *reinterpret_cast<const uint4*>(S.vt + (32 * d + ql) * VROW +
                                                            2 * (16 * (2 * TT + k) + 8 * h));
            oacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(h8_t, v),
                                                             __builtin_bit_cast(h8_t, wb[k]),
                                                             oacc[d], 0, 0, 0);
          }
      };
      tile(std::integral_constant<int, 0>{});
      tile(std::integral_constant<int, 1>{});
    }
    if (kb + 1 < nb) store(kb + 1, st[(kb + 1) & 1]);
    __syncthreads();
  }
  if (!live) return;

  // ---- normalise, optionally rotate back, store ---------------------------
  l += __shfl_xor(l, 32);
  zs += __shfl_xor(zs, 32);
  float y[64];  // y[16 d + r]: dim 32 d + 8 (r / 4) + 4 h + r % 4
  const float il = 1.0f / l;
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      y[16 * d + r] = (__builtin_amdgcn_ldexpf(oacc[d][r], 24) - zs) * il;
  if (v_had) {
#pragma unroll
    for (int s = 1; s < 64; s <<= 1)
#pragma unroll
      for (int i = 0; i < 64; ++i)
        if (!(i & s)) {
          const float a = y[i], c = y[i + s];
          y[i] = a + c;
          y[i + s] = a - c;
        }
#pragma unroll
    for (int i = 0; i < 64; ++i) {
      const float p = __shfl_xor(y[i], 32);
      y[i] = cnorm * (h ? p - y[i] : y[i] + p);
    }
  }
  if (tw + ql < T) {
    uint16_t* dst = out + ((int64_t)(b * T + t) * Hq + hq) * PD + 4 * h;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float* v = y + 16 * d + 4 * j;
        *reinterpret_cast<uint2*>(dst + 32 * d + 8 * j) =
            make_uint2(bf16x2_rne(v[0], v[1]), bf16x2_rne(v[2], v[3]));
      }
  }
}

#undef PF_FOR16

}  // namespace

hipError_t launch_kv_attention_prefill(const uint16_t* q, int64_t B, int64_t T, int64_t Hq,
                                       int64_t Hkv, int64_t past, const uint8_t* kc,
                                       const uint16_t* ks, const int16_t* kz, const uint8_t* vc,
                                       const uint16_t* vs, const int16_t* vz, int64_t s_cap,
                                       float sm_scale, bool v_had, uint16_t* out,
                                       hipStream_t stream) {
  const int G = (int)(Hq / Hkv);
  const float sm2 = sm_scale * PLOG2E;
  const float cnorm = (float)(1.0 / __builtin_sqrt((double)PD));
  const int NW = 8;
  const int64_t TP = 32 * NW / G;
  const int64_t grid = B * Hkv * ((T + TP - 1) / TP);
#define PF_LAUNCH(GG)                                                                          \
  hipLaunchKernelGGL(kv_prefill_kernel<GG>, dim3((unsigned)grid), dim3(64 * NW), 0, stream, q, \
                     (int)B, (int)T, (int)Hq, (int)Hkv, (int)past, kc, ks, kz, vc, vs, vz,      \
                     s_cap, sm2, cnorm, v_had ? 1 : 0, out)
  switch (G) {
    case 1: PF_LAUNCH(1); break;
    case 2: PF_LAUNCH(2); break;
    case 4: PF_LAUNCH(4); break;
    case 8: PF_LAUNCH(8); break;
    default: return hipErrorInvalidValue;
  }
#undef PF_LAUNCH
  return hipGetLastError();
}

}  // namespace offq
