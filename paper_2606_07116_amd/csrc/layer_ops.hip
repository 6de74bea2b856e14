// Decoder-layer kernels around the quantized linear layers, for one decode
// step (one new token per sequence):
// * add + RMSNorm of the residual stream (RMSNorm's scale is fused into the
//   following weights offline, sec. 3.1 "Why the L-infinity norm", so the
//   kernel only normalises);
// * RoPE on the query and key heads, the per-head online Hadamard H3 on the
//   key (sec. 3.3 step 2(3)) and the KV4 quantizer (Eq. 1, group = head
//   dimension, sec. 4.2) writing the new position into the cache;
// * SwiGLU between the up/gate and down projections (the grouping
//   permutation P4 is fused into the up/gate weights offline, sec. 3.3
//   step 2(4), so the kernel is elementwise).
#include "common.h"
#include "internal.h"

namespace offq {
namespace {

__device__ __forceinline__ float wsum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wmax(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wmin(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fminf(v, __shfl_xor(v, o));
  return v;
}

// ---------------------------------------------------------------- add + RMSNorm
constexpr int RN_THREADS = 256;

// h = bf16(fl32(x + res)) (h = x without res); y = bf16(h * fl32(1 / sqrt(mean(h^2) + eps))).
// One workgroup per row, 8 elements per 16-byte load.
__global__ __launch_bounds__(RN_THREADS) void add_rmsnorm_kernel(
    const uint16_t* __restrict__ x, int64_t ldx, const uint16_t* __restrict__ res, int64_t ldr,
    int D, float eps, uint16_t* __restrict__ h_out, int64_t ldh, uint16_t* __restrict__ y_out,
    int64_t ldy) {
  __shared__ float s_red[RN_THREADS / 64];
  const int tid = (int)__builtin_amdgcn_workitem_id_x();
  const int64_t row = __builtin_amdgcn_workgroup_id_x();
  const uint4* xr = reinterpret_cast<const uint4*>(x + row * ldx);
  const uint4* rr = res ? reinterpret_cast<const uint4*>(res + row * ldr) : nullptr;
  const int nc = D / 8;
  auto h8 = [&](int c, float* h) {
    const uint4 a = xr[c];
    const uint32_t aw[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      h[2 * k] = bf16_lo(aw[k]);
      h[2 * k + 1] = bf16_hi(aw[k]);
    }
    if (rr) {
      const uint4 b = rr[c];
      const uint32_t bw[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        h[2 * k] = bf16_lo(f32_to_bf16_rne(h[2 * k] + bf16_lo(bw[k])));
        h[2 * k + 1] = bf16_lo(f32_to_bf16_rne(h[2 * k + 1] + bf16_hi(bw[k])));
      }
    }
  };
  float ss = 0.0f;
  for (int c = tid; c < nc; c += RN_THREADS) {
    float h[8];
    h8(c, h);
#pragma unroll
    for (int k = 0; k < 8; ++k) ss = __builtin_fmaf(h[k], h[k], ss);
    if (h_out) {
      uint4 o;
      o.x = bf16x2_rne(h[0], h[1]);
      o.y = bf16x2_rne(h[2], h[3]);
      o.z = bf16x2_rne(h[4], h[5]);
      o.w = bf16x2_rne(h[6], h[7]);
      reinterpret_cast<uint4*>(h_out + row * ldh)[c] = o;
    }
  }
  if (!y_out) return;
  ss = wsum(ss);
  if ((tid & 63) == 0) s_red[tid >> 6] = ss;
  __syncthreads();
  ss = s_red[0] + s_red[1] + s_red[2] + s_red[3];
  const float inv = 1.0f / __builtin_sqrtf(ss / (float)D + eps);
  for (int c = tid; c < nc; c += RN_THREADS) {
    float h[8];
    h8(c, h);
    uint4 o;
    o.x = bf16x2_rne(h[0] * inv, h[1] * inv);
    o.y = bf16x2_rne(h[2] * inv, h[3] * inv);
    o.z = bf16x2_rne(h[4] * inv, h[5] * inv);
    o.w = bf16x2_rne(h[6] * inv, h[7] * inv);
    reinterpret_cast<uint4*>(y_out + row * ldy)[c] = o;
  }
}

// ---------------------------------------------------------------- SwiGLU
// out[m, f] = bf16(fl32(silu(g) * u)), silu(g) = g / (1 + exp(-g)) in fp32,
// g = gu[m, f], u = gu[m, F + f].  8 outputs per thread.
__global__ __launch_bounds__(256) void swiglu_kernel(const uint16_t* __restrict__ gu, int64_t ldg,
                                                     int F, uint16_t* __restrict__ out,
                                                     int64_t ldo, int64_t total8) {
  const int64_t i = (int64_t)__builtin_amdgcn_workgroup_id_x() * 256 +
                    (int)__builtin_amdgcn_workitem_id_x();
  if (i >= total8) return;
  const int per_row = F / 8;
  const int64_t m = i / per_row;
  const int c = (int)(i - m * per_row);
  const uint4 g = reinterpret_cast<const uint4*>(gu + m * ldg)[c];
  const uint4 u = reinterpret_cast<const uint4*>(gu + m * ldg + F)[c];
  const uint32_t gw[4] = {g.x, g.y, g.z, g.w}, uw[4] = {u.x, u.y, u.z, u.w};
  uint32_t ow[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float g0 = bf16_lo(gw[k]), g1 = bf16_hi(gw[k]);
    const float a0 = g0 / (1.0f + expf(-g0)), a1 = g1 / (1.0f + expf(-g1));
    ow[k] = bf16x2_rne(a0 * bf16_lo(uw[k]), a1 * bf16_hi(uw[k]));
  }
  reinterpret_cast<uint4*>(out + m * ldo)[c] = make_uint4(ow[0], ow[1], ow[2], ow[3]);
}

// ---------------------------------------------------------------- RoPE + KV append
constexpr int HD = 128;  // head dimension

struct RopeTable {
  float inv_freq[HD / 2];  // fl32(base^(-2i/128)), computed on the host in double
};

// One workgroup per (token m, GPW head slots): 16 slots (4 waves) when the
// step has many tokens, 4 (one wave) for a few tokens, so that a decode step
// still has enough workgroups; each group of 16 lanes takes one head slot j (j < Hq query heads, then Hkv key heads, then
// Hkv value heads of the projection row qkv[m]), lane l of a group holding
// dims 8 l .. 8 l + 7.  The token's 64 RoPE angles a_i = fl32(pos *
// inv_freq[i]) are computed once per workgroup into LDS.  RoPE pairs dims
// (i, i + 64), which sit in lanes l and l + 8 of the group:
//   x'[i] = x[i] cos(a_i) - x[i + 64] sin(a_i),  x'[i + 64] = x[i + 64] cos(a_i) + x[i] sin(a_i)
// Queries are stored as bf16; keys are rounded to bf16, rotated by c H
// (optional: butterflies over dim bits 0..2 in the lane, 3..6 across the
// group) and quantized; values are quantized (optionally after c H).  Token m
// belongs to sequence m / T (T = 1 for a decode step, T new tokens per
// sequence for a prefill); its cache row for kv head h is
// ((m / T) * Hkv + h) * s_cap + pos[m]; positions outside [0, s_cap) write
// nothing.
template <int GPW>
__global__ __launch_bounds__(16 * GPW) void rope_kv_append_kernel(
    const uint16_t* __restrict__ qkv, int64_t ldq, int M, int T, int Hq, int Hkv,
    const int32_t* __restrict__ positions, RopeTable tab, int k_had, int v_had,
    uint16_t* __restrict__ q_out, uint8_t* __restrict__ kc, uint16_t* __restrict__ ks,
    int16_t* __restrict__ kz, uint8_t* __restrict__ vc, uint16_t* __restrict__ vs,
    int16_t* __restrict__ vz, int64_t s_cap, float* __restrict__ k_dbg,
    float* __restrict__ v_dbg) {
  __shared__ float2 s_cs[HD / 2];  // (cos, sin) of the token's angles
  const int tid = (int)__builtin_amdgcn_workitem_id_x();
  const int slots = Hq + 2 * Hkv;
  const int nchunk = (slots + GPW - 1) / GPW;
  const int bid = (int)__builtin_amdgcn_workgroup_id_x();
  const int m = bid / nchunk;
  const int l16 = tid & 15, j = (bid - m * nchunk) * GPW + (tid >> 4);
  const int pos = positions[m];
  if (tid < HD / 2) {
    float sn, cs;
    sincosf((float)pos * tab.inv_freq[tid], &sn, &cs);
    s_cs[tid] = make_float2(cs, sn);
  }
  __syncthreads();
  // this lane's angles: pair indices 8 (l16 mod 8) .. + 7
  float cs8[8], sn8[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float2 v = s_cs[8 * (l16 & 7) + i];
    cs8[i] = v.x;
    sn8[i] = v.y;
  }
  const bool upper = l16 >= 8;  // holds dims 64 .. 127
  const uint16_t* row = qkv + (int64_t)m * ldq + 8 * l16;
  if (j < slots) {  // whole groups of 16 lanes leave together
    const uint4 w4 = *reinterpret_cast<const uint4*>(row + (int64_t)j * HD);
    const uint32_t wv[4] = {w4.x, w4.y, w4.z, w4.w};
    float x[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x[2 * k] = bf16_lo(wv[k]);
      x[2 * k + 1] = bf16_hi(wv[k]);
    }
    const bool is_v = j >= Hq + Hkv;
    if (!is_v) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float p = __shfl_xor(x[i], 8);
        x[i] = upper ? x[i] * cs8[i] + p * sn8[i] : x[i] * cs8[i] - p * sn8[i];
      }
      if (j < Hq) {
        *reinterpret_cast<uint4*>(q_out + ((int64_t)m * Hq + j) * HD + 8 * l16) =
            make_uint4(bf16x2_rne(x[0], x[1]), bf16x2_rne(x[2], x[3]), bf16x2_rne(x[4], x[5]),
                       bf16x2_rne(x[6], x[7]));
        return;
      }
      // the key after RoPE is a bf16 activation
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = bf16_lo(f32_to_bf16_rne(x[i]));
    }
    const int h = is_v ? j - Hq - Hkv : j - Hq;
    if (is_v ? v_had : k_had) {
      // 128-point FWHT: dim bits 0..2 inside the lane, bits 3..6 across the group
#pragma unroll
      for (int st = 1; st < 8; st <<= 1)
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (!(i & st)) {
            const float a = x[i], b = x[i + st];
            x[i] = a + b;
            x[i + st] = a - b;
          }
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        const bool up = (l16 >> st) & 1;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float o = __shfl_xor(x[i], 1 << st);
          x[i] = up ? o - x[i] : x[i] + o;
        }
      }
      const float c = 0.08838834764831845f;  // fl32(1 / sqrt(128))
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] *= c;
    }
    float* dbg = is_v ? v_dbg : k_dbg;
    if (dbg) {
      float4* d4 = reinterpret_cast<float4*>(dbg + ((int64_t)m * Hkv + h) * HD + 8 * l16);
      d4[0] = make_float4(x[0], x[1], x[2], x[3]);
      d4[1] = make_float4(x[4], x[5], x[6], x[7]);
    }
    float mx = x[0], mn = x[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) {
      mx = fmaxf(mx, x[i]);
      mn = fminf(mn, x[i]);
    }
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      mx = fmaxf(mx, __shfl_xor(mx, o));
      mn = fminf(mn, __shfl_xor(mn, o));
    }
    const QParams p = quant_params(mx, mn);
    const uint32_t lo = __float_as_uint(p.lo);
    uint32_t code = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) code |= (quant_bits(x[k], p) - lo) << (4 * k);
    if (pos < 0 || (int64_t)pos >= s_cap) return;
    const int64_t crow = ((int64_t)(m / T) * Hkv + h) * s_cap + pos;
    reinterpret_cast<uint32_t*>((is_v ? vc : kc) + crow * (HD / 2))[l16] = code;
    if (l16 == 0) {
      (is_v ? vs : ks)[crow] = p.s16;
      (is_v ? vz : kz)[crow] = p.z;
    }
  }
}

// ---------------------------------------------------------------- fused variants
// add + RMSNorm + the quantizer (no online rotation: the inputs of QKV and
// up/gate, whose rotations are fused offline): the same arithmetic as
// add_rmsnorm followed by rotate_quantize(apply_hadamard = 0) on the bf16 y,
// in one pass.  One workgroup per row; thread t holds the E = D / 256
// consecutive channels [t E, t E + E) (E a multiple of 8); a group of g
// channels spans g / E adjacent lanes (1 ... 64).
template <int E>
__global__ __launch_bounds__(RN_THREADS) void add_rmsnorm_quant_kernel(
    const uint16_t* __restrict__ x, int64_t ldx, const uint16_t* __restrict__ res, int64_t ldr,
    int D, float eps, int log2g, uint16_t* __restrict__ h_out, int64_t ldh,
    uint8_t* __restrict__ codes, uint16_t* __restrict__ scale, int16_t* __restrict__ zero,
    uint16_t* __restrict__ y_dbg, int64_t ldy) {
  __shared__ float s_red[RN_THREADS / 64];
  const int tid = (int)__builtin_amdgcn_workitem_id_x();
  const int64_t row = __builtin_amdgcn_workgroup_id_x();
  float h[E];
  const uint4* xr = reinterpret_cast<const uint4*>(x + row * ldx) + tid * (E / 8);
#pragma unroll
  for (int c = 0; c < E / 8; ++c) {
    const uint4 a = xr[c];
    const uint32_t aw[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      h[8 * c + 2 * k] = bf16_lo(aw[k]);
      h[8 * c + 2 * k + 1] = bf16_hi(aw[k]);
    }
  }
  if (res) {
    const uint4* rr = reinterpret_cast<const uint4*>(res + row * ldr) + tid * (E / 8);
#pragma unroll
    for (int c = 0; c < E / 8; ++c) {
      const uint4 b = rr[c];
      const uint32_t bw[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        h[8 * c + 2 * k] = bf16_lo(f32_to_bf16_rne(h[8 * c + 2 * k] + bf16_lo(bw[k])));
        h[8 * c + 2 * k + 1] = bf16_lo(f32_to_bf16_rne(h[8 * c + 2 * k + 1] + bf16_hi(bw[k])));
      }
    }
  }
  if (h_out) {
    uint4* ho = reinterpret_cast<uint4*>(h_out + row * ldh) + tid * (E / 8);
#pragma unroll
    for (int c = 0; c < E / 8; ++c)
      ho[c] = make_uint4(bf16x2_rne(h[8 * c], h[8 * c + 1]), bf16x2_rne(h[8 * c + 2], h[8 * c + 3]),
                         bf16x2_rne(h[8 * c + 4], h[8 * c + 5]),
                         bf16x2_rne(h[8 * c + 6], h[8 * c + 7]));
  }
  float ss = 0.0f;
#pragma unroll
  for (int k = 0; k < E; ++k) ss = __builtin_fmaf(h[k], h[k], ss);
  ss = wsum(ss);
  if ((tid & 63) == 0) s_red[tid >> 6] = ss;
  __syncthreads();
  ss = s_red[0] + s_red[1] + s_red[2] + s_red[3];
  const float inv = 1.0f / __builtin_sqrtf(ss / (float)D + eps);
  float y[E];
#pragma unroll
  for (int k = 0; k < E; ++k) y[k] = bf16_lo(f32_to_bf16_rne(h[k] * inv));
  if (y_dbg) {
    uint4* yo = reinterpret_cast<uint4*>(y_dbg + row * ldy) + tid * (E / 8);
#pragma unroll
    for (int c = 0; c < E / 8; ++c)
      yo[c] = make_uint4(bf16x2_rne(y[8 * c], y[8 * c + 1]), bf16x2_rne(y[8 * c + 2], y[8 * c + 3]),
                         bf16x2_rne(y[8 * c + 4], y[8 * c + 5]),
                         bf16x2_rne(y[8 * c + 6], y[8 * c + 7]));
  }
  // group min / max over the g / E lanes of the group
  float mx = y[0], mn = y[0];
#pragma unroll
  for (int k = 1; k < E; ++k) {
    mx = fmaxf(mx, y[k]);
    mn = fminf(mn, y[k]);
  }
  const int lanes = (1 << log2g) / E;
  for (int o = 1; o < lanes; o <<= 1) {
    mx = fmaxf(mx, __shfl_xor(mx, o));
    mn = fminf(mn, __shfl_xor(mn, o));
  }
  const QParams p = quant_params(mx, mn);
  const uint32_t lo = __float_as_uint(p.lo);
  uint32_t cw[E / 8];
#pragma unroll
  for (int c = 0; c < E / 8; ++c) {
    uint32_t w = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) w |= (quant_bits(y[8 * c + k], p) - lo) << (4 * k);
    cw[c] = w;
  }
  uint32_t* co = reinterpret_cast<uint32_t*>(codes + row * (D / 2)) + tid * (E / 8);
#pragma unroll
  for (int c = 0; c < E / 8; ++c) co[c] = cw[c];
  if ((tid & (lanes - 1)) == 0) {
    const int64_t gi = row * (D >> log2g) + (int64_t)tid * E / (1 << log2g);
    scale[gi] = p.s16;
    zero[gi] = p.z;
  }
}

// SwiGLU + the online 128-point Hadamard H4 + the quantizer (g = 128) for
// the down-projection input: a = bf16(fl32(silu(gate) * up)) with silu from
// the hardware exp2 and reciprocal (swiglu_kernel divides exactly; the two
// can differ by one bf16 ulp next to a rounding midpoint), then y = c H a
// per group of 128 (fp32 butterflies, c = fl32(1/sqrt(128))
// after them) and the codes of Eq. 1.  A group is 16 lanes x 8 channels:
// butterfly stages over channel bits 0..2 inside the lane, bits 3..6 across
// the lanes.  Workgroup: 16 groups of one row.
constexpr float SW_LOG2E = 1.4426950408889634f;

__global__ __launch_bounds__(256) void swiglu_rq_kernel(const uint16_t* __restrict__ gu,
                                                        int64_t ldg, int F,
                                                        uint8_t* __restrict__ codes,
                                                        uint16_t* __restrict__ scale,
                                                        int16_t* __restrict__ zero,
                                                        float* __restrict__ y_dbg,
                                                        int64_t groups_per_row, int64_t M) {
  const int tid = (int)__builtin_amdgcn_workitem_id_x();
  const int64_t gidx = (int64_t)__builtin_amdgcn_workgroup_id_x() * 16 + (tid >> 4);
  const int64_t m = gidx / groups_per_row;
  const int grp = (int)(gidx - m * groups_per_row);
  if (m >= M) return;  // whole groups of 16 lanes leave together
  const int l16 = tid & 15;
  const int c0 = grp * 128 + l16 * 8;  // first channel of this lane
  const uint4 g4 = *reinterpret_cast<const uint4*>(gu + m * ldg + c0);
  const uint4 u4 = *reinterpret_cast<const uint4*>(gu + m * ldg + F + c0);
  const uint32_t gw[4] = {g4.x, g4.y, g4.z, g4.w}, uw[4] = {u4.x, u4.y, u4.z, u4.w};
  float v[8];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float g0 = bf16_lo(gw[k]), g1 = bf16_hi(gw[k]);
    // silu with the hardware exp2 and reciprocal (about 1 ulp each): the
    // product rounds to bf16, so an error of a few fp32 ulps can only move a
    // value that lies next to a rounding midpoint to the other neighbour
    const float a0 = g0 * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(g0 * -SW_LOG2E));
    const float a1 = g1 * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(g1 * -SW_LOG2E));
    const uint32_t ab = bf16x2_rne(a0 * bf16_lo(uw[k]), a1 * bf16_hi(uw[k]));
    v[2 * k] = bf16_lo(ab);
    v[2 * k + 1] = bf16_hi(ab);
  }
  // butterflies over channel bits 0, 1, 2 (inside the lane)
#pragma unroll
  for (int h = 1; h < 8; h <<= 1)
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (!(i & h)) {
        const float a = v[i], b = v[i + h];
        v[i] = a + b;
        v[i + h] = a - b;
      }
  // bits 3 .. 6: across the 16 lanes of the group (lane bit 0 .. 3)
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const bool up = (l16 >> s) & 1;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float o = __shfl_xor(v[i], 1 << s);
      v[i] = up ? o - v[i] : v[i] + o;
    }
  }
  const float c = 0.08838834764831845f;  // fl32(1 / sqrt(128))
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] *= c;
  if (y_dbg) {
    float4* yo = reinterpret_cast<float4*>(y_dbg + m * F + c0);
    yo[0] = make_float4(v[0], v[1], v[2], v[3]);
    yo[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
  float mx = v[0], mn = v[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) {
    mx = fmaxf(mx, v[i]);
    mn = fminf(mn, v[i]);
  }
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) {
    mx = fmaxf(mx, __shfl_xor(mx, o));
    mn = fminf(mn, __shfl_xor(mn, o));
  }
  const QParams p = quant_params(mx, mn);
  const uint32_t lo = __float_as_uint(p.lo);
  uint32_t w = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) w |= (quant_bits(v[k], p) - lo) << (4 * k);
  reinterpret_cast<uint32_t*>(codes + m * (F / 2))[c0 / 8] = w;
  if (l16 == 0) {
    scale[m * groups_per_row + grp] = p.s16;
    zero[m * groups_per_row + grp] = p.z;
  }
}

}  // namespace

hipError_t launch_add_rmsnorm_quant(const uint16_t* x, int64_t ldx, const uint16_t* res,
                                    int64_t ldr, int64_t M, int64_t D, float eps, int log2g,
                                    uint16_t* h_out, int64_t ldh, uint8_t* codes, uint16_t* scale,
                                    int16_t* zero, uint16_t* y_dbg, int64_t ldy,
                                    hipStream_t stream) {
  const int E = (int)(D / RN_THREADS);
#define OFFQ_ARQ(E_)                                                                         \
  hipLaunchKernelGGL(add_rmsnorm_quant_kernel<E_>, dim3((unsigned)M), dim3(RN_THREADS), 0,   \
                     stream, x, ldx, res, ldr, (int)D, eps, log2g, h_out, ldh, codes, scale, \
                     zero, y_dbg, ldy)
  switch (E) {
    case 8: OFFQ_ARQ(8); break;
    case 16: OFFQ_ARQ(16); break;
    case 32: OFFQ_ARQ(32); break;
    case 64: OFFQ_ARQ(64); break;
    default: return hipErrorInvalidValue;
  }
#undef OFFQ_ARQ
  return hipGetLastError();
}

hipError_t launch_swiglu_rq(const uint16_t* gu, int64_t ldg, int64_t M, int64_t F, uint8_t* codes,
                            uint16_t* scale, int16_t* zero, float* y_dbg, hipStream_t stream) {
  const int64_t gpr = F / 128;
  const int64_t groups = M * gpr;
  hipLaunchKernelGGL(swiglu_rq_kernel, dim3((unsigned)((groups + 15) / 16)), dim3(256), 0, stream,
                     gu, ldg, (int)F, codes, scale, zero, y_dbg, gpr, M);
  return hipGetLastError();
}

hipError_t launch_add_rmsnorm(const uint16_t* x, int64_t ldx, const uint16_t* res, int64_t ldr,
                              int64_t M, int64_t D, float eps, uint16_t* h_out, int64_t ldh,
                              uint16_t* y_out, int64_t ldy, hipStream_t stream) {
  hipLaunchKernelGGL(add_rmsnorm_kernel, dim3((unsigned)M), dim3(RN_THREADS), 0, stream, x, ldx,
                     res, ldr, (int)D, eps, h_out, ldh, y_out, ldy);
  return hipGetLastError();
}

hipError_t launch_swiglu(const uint16_t* gu, int64_t ldg, int64_t M, int64_t F, uint16_t* out,
                         int64_t ldo, hipStream_t stream) {
  const int64_t total8 = M * (F / 8);
  hipLaunchKernelGGL(swiglu_kernel, dim3((unsigned)((total8 + 255) / 256)), dim3(256), 0, stream,
                     gu, ldg, (int)F, out, ldo, total8);
  return hipGetLastError();
}

hipError_t launch_rope_kv_append(const uint16_t* qkv, int64_t ldq, int64_t M, int64_t T,
                                 int64_t Hq, int64_t Hkv, const int32_t* positions, double rope_base,
                                 bool k_had, bool v_had, uint16_t* q_out, uint8_t* kc,
                                 uint16_t* ks, int16_t* kz, uint8_t* vc, uint16_t* vs,
                                 int16_t* vz, int64_t s_cap, float* k_dbg, float* v_dbg,
                                 hipStream_t stream) {
  RopeTable tab;
  for (int i = 0; i < HD / 2; ++i)
    tab.inv_freq[i] = (float)__builtin_pow(rope_base, -2.0 * i / (double)HD);
  // 16 head slots per workgroup with many tokens, 4 with few
  const int gpw = M >= 256 ? 16 : 4;
  const int64_t nchunk = (Hq + 2 * Hkv + gpw - 1) / gpw;
  hipLaunchKernelGGL(gpw == 16 ? rope_kv_append_kernel<16> : rope_kv_append_kernel<4>,
                     dim3((unsigned)(M * nchunk)), dim3(16 * gpw), 0, stream, qkv, ldq, (int)M,
                     (int)T, (int)Hq, (int)Hkv, positions, tab, k_had ? 1 : 0, v_had ? 1 : 0,
                     q_out, kc, ks, kz, vc, vs, vz, s_cap, k_dbg, v_dbg);
  return hipGetLastError();
}

}  // namespace offq
