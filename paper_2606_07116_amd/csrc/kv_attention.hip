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
//   q_r  = bf16_rne(c * H q)                         c = fl32(1 / sqrt(128))
//   s_j  = sm_scale * sk_j * sum_d q_r[d] (ck_j[d] - zk_j)
//   p    = softmax_j(s)
//   o[d] = sum_j p_j * sv_j * (cv_j[d] - zv_j)       (then c * H o if asked)
//
// Organisation (split over the sequence, as in flash decoding)
// * Pass 1: one workgroup of 4 waves per (b, h, chunk of CH positions).
//   Scores: a lane owns whole positions; it reads the position's 64 code bytes
//   and forms the dot product with v_dot2_f32_bf16 against pairs of query
//   values: a pair of codes (c, c') becomes the bf16 pair (128 + c, 128 + c')
//   with one and-or, so sum q (128 + c) - 128 sum q = sum q c.  Softmax
//   statistics of the chunk through DPP and LDS; the weights p_j sv_j go to
//   LDS.  Values: a lane owns 8 dimensions (one code dword of a row) and a
//   quarter of the positions of its wave; codes are widened with
//   v_cvt_f32_ubyte and accumulated in fp32.  The chunk's maximum, sum and
//   unnormalised output go to the workspace.
// * Pass 2: one workgroup per (b, h) merges the chunks (rescaled by
//   exp(m_i - m)), divides by the sum, optionally rotates back, and stores
//   bf16.
#include "common.h"
#include "internal.h"

namespace offq {
namespace {

constexpr int DH = 128;       // head dimension
constexpr int CH = 1024;      // positions per chunk (pass 1 workgroup)
constexpr int THREADS = 256;  // 4 waves
constexpr int PPL = CH / THREADS;  // positions per lane in the score phase
constexpr float LOG2E = 1.4426950408889634f;

// acc + a.lo * b.lo + a.hi * b.hi for two packed bf16 pairs (fp32 result).
// Through the builtin, not inline asm: a dot result read by another VALU
// within a few cycles needs wait states that only the compiler's hazard
// tracking inserts.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float dot2_bf16_acc(uint32_t a, uint32_t b, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), acc, false);
}

// byte K of w as a float (v_cvt_f32_ubyteK)
template <int K>
__device__ __forceinline__ float ubyte(uint32_t w) {
  return (float)((w >> (8 * K)) & 0xFFu);
}

// (-1)^popcount(i & j): entry (i, j) of the Sylvester Hadamard matrix
__device__ __forceinline__ float had_sign(int i, int j) {
  return (__builtin_popcount(i & j) & 1) ? -1.0f : 1.0f;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Workspace per (b, h, chunk): m, l, then o[128] (fp32).
constexpr int WS_FLOATS = 2 + DH;

__global__ __launch_bounds__(THREADS) void kv_attention_chunk_kernel(
    const uint16_t* __restrict__ q, const uint8_t* __restrict__ kc, const uint16_t* __restrict__ ks,
    const int16_t* __restrict__ kz, const uint8_t* __restrict__ vc, const uint16_t* __restrict__ vs,
    const int16_t* __restrict__ vz, int64_t S_cap, int seq_len, int nchunk, float sm_scale,
    float cnorm, float* __restrict__ ws) {
  __shared__ float s_q[DH];                     // query (fp32)
  __shared__ float s_qr[DH];                    // H q (fp32)
  __shared__ uint32_t s_qp[DH / 2];             // rotated query as bf16 pairs
  __shared__ float s_qsum;                      // sum of the bf16 query values
  __shared__ float s_red[2][THREADS / 64];      // per-wave max / sum
  __shared__ float s_w[CH];                     // p_j * sv_j of the chunk
  __shared__ float s_o[THREADS / 64][DH];       // per-wave partial outputs
  __shared__ float s_zw[THREADS / 64];          // per-wave sum of p_j sv_j zv_j

  const int tid = (int)__builtin_amdgcn_workitem_id_x();
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int blk = (int)__builtin_amdgcn_workgroup_id_x();
  const int bh = blk / nchunk, chunk = blk - bh * nchunk;
  const int j0 = chunk * CH;
  const int n = min(CH, seq_len - j0);          // positions of this chunk (>= 1)
  const int64_t row0 = (int64_t)bh * S_cap + j0;

  // ---- query: q_r = bf16(c H q), as pairs (d, d + 4) of each group of 8 ----
  if (tid < DH) s_q[tid] = bf16_lo(q[(int64_t)bh * DH + tid]);
  __syncthreads();
  if (tid < DH) {
    float acc = 0.0f;
    for (int i = 0; i < DH; ++i) acc = __builtin_fmaf(s_q[i], had_sign(i, tid), acc);
    s_qr[tid] = acc;
  }
  __syncthreads();
  if (tid < DH / 2) {
    // pair p = 4 i + j (i = 0..15, j = 0..3): dimensions 8 i + j and 8 i + j + 4
    const int i = tid >> 2, j = tid & 3;
    const float a = s_qr[8 * i + j] * cnorm, b = s_qr[8 * i + j + 4] * cnorm;
    s_qp[tid] = bf16x2_rne(a, b);
  }
  __syncthreads();
  if (tid == 0) {
    float t = 0.0f;
    for (int p = 0; p < DH / 2; ++p) t += bf16_lo(s_qp[p]) + bf16_hi(s_qp[p]);
    s_qsum = t;
  }
  __syncthreads();

  // ---- scores: lane owns positions wave*256 + it*64 + lane -----------------
  uint32_t qp[DH / 2];
#pragma unroll
  for (int p = 0; p < DH / 2; ++p) qp[p] = s_qp[p];
  const float qsum = s_qsum;
  float sc[PPL];
  float mloc = -__builtin_inff();
  {
    uint4 kr[PPL][4];
    float ksc[PPL];
    int kzz[PPL];
#pragma unroll
    for (int it = 0; it < PPL; ++it) {
      const int jl = wave * (CH / 4) + it * 64 + lane;
      const int jj = min(jl, n - 1);  // past the chunk: a valid row, result unused
      const uint4* src = reinterpret_cast<const uint4*>(kc + (row0 + jj) * (DH / 2));
#pragma unroll
      for (int c = 0; c < 4; ++c) kr[it][c] = src[c];
      ksc[it] = fp16_bits_to_f32(ks[row0 + jj]);
      kzz[it] = kz[row0 + jj];
    }
#pragma unroll
    for (int it = 0; it < PPL; ++it) {
      float dot = 0.0f;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t w4[4] = {kr[it][c].x, kr[it][c].y, kr[it][c].z, kr[it][c].w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int i = 4 * c + u;  // dims 8 i .. 8 i + 7
          const uint32_t w = w4[u];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const uint32_t pr = ((w >> (4 * j)) & 0x000F000Fu) | 0x43004300u;  // (128 + c, 128 + c')
            dot = dot2_bf16_acc(qp[4 * i + j], pr, dot);
          }
        }
      }
      const int jl = wave * (CH / 4) + it * 64 + lane;
      const float s = sm_scale * ksc[it] * (dot - (128.0f + (float)kzz[it]) * qsum);
      sc[it] = jl < n ? s : -__builtin_inff();
      mloc = fmaxf(mloc, sc[it]);
    }
  }
  mloc = wave_max(mloc);
  if (lane == 0) s_red[0][wave] = mloc;
  __syncthreads();
  const float m = fmaxf(fmaxf(s_red[0][0], s_red[0][1]), fmaxf(s_red[0][2], s_red[0][3]));

  // ---- probabilities and value weights -------------------------------------
  float lsum = 0.0f, zsum = 0.0f;
#pragma unroll
  for (int it = 0; it < PPL; ++it) {
    const int jl = wave * (CH / 4) + it * 64 + lane;
    const int jj = min(jl, n - 1);
    const float p = jl < n ? __builtin_amdgcn_exp2f((sc[it] - m) * LOG2E) : 0.0f;
    const float w = p * fp16_bits_to_f32(vs[row0 + jj]);
    lsum += p;
    zsum = __builtin_fmaf(w, (float)vz[row0 + jj], zsum);
    s_w[jl] = w;
  }
  lsum = wave_sum(lsum);
  zsum = wave_sum(zsum);
  if (lane == 0) {
    s_red[1][wave] = lsum;
    s_zw[wave] = zsum;
  }
  __syncthreads();

  // ---- values: lane (dg, pg) owns dims 8 dg .. 8 dg + 7 and the positions
  // jl = wave * 256 + 4 t + pg of its wave's quarter ---------------------------
  const int dg = lane & 15, pg = lane >> 4;
  float acc[8] = {};
  {
    const uint32_t* vrow = reinterpret_cast<const uint32_t*>(vc + row0 * (DH / 2)) + dg;
    constexpr int NT = CH / 4 / 4;  // positions per lane (64)
    constexpr int BT = 16;          // loads in flight
#pragma unroll 1
    for (int t0 = 0; t0 < NT; t0 += BT) {
      uint32_t cw[BT];
#pragma unroll
      for (int t = 0; t < BT; ++t) {
        const int jl = wave * (CH / 4) + 4 * (t0 + t) + pg;
        cw[t] = vrow[(int64_t)min(jl, n - 1) * (DH / 8)];
      }
#pragma unroll
      for (int t = 0; t < BT; ++t) {
        const int jl = wave * (CH / 4) + 4 * (t0 + t) + pg;
        const float w = jl < n ? s_w[jl] : 0.0f;
        const uint32_t lo = cw[t] & 0x0F0F0F0Fu, hi = (cw[t] >> 4) & 0x0F0F0F0Fu;
        // byte k of lo: dim 8 dg + 2 k; byte k of hi: dim 8 dg + 2 k + 1
        acc[0] = __builtin_fmaf(w, ubyte<0>(lo), acc[0]);
        acc[1] = __builtin_fmaf(w, ubyte<0>(hi), acc[1]);
        acc[2] = __builtin_fmaf(w, ubyte<1>(lo), acc[2]);
        acc[3] = __builtin_fmaf(w, ubyte<1>(hi), acc[3]);
        acc[4] = __builtin_fmaf(w, ubyte<2>(lo), acc[4]);
        acc[5] = __builtin_fmaf(w, ubyte<2>(hi), acc[5]);
        acc[6] = __builtin_fmaf(w, ubyte<3>(lo), acc[6]);
        acc[7] = __builtin_fmaf(w, ubyte<3>(hi), acc[7]);
      }
    }
  }
  // sum over the four position groups of the wave, then over the waves
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    acc[k] += __shfl_xor(acc[k], 16);
    acc[k] += __shfl_xor(acc[k], 32);
  }
  if (pg == 0) {
#pragma unroll
    for (int k = 0; k < 8; ++k) s_o[wave][8 * dg + k] = acc[k];
  }
  __syncthreads();
  float* const out = ws + (int64_t)blk * WS_FLOATS;
  if (tid < DH) {
    const float zw = s_zw[0] + s_zw[1] + s_zw[2] + s_zw[3];
    out[2 + tid] = s_o[0][tid] + s_o[1][tid] + s_o[2][tid] + s_o[3][tid] - zw;
  }
  if (tid == 0) {
    out[0] = m;
    out[1] = s_red[1][0] + s_red[1][1] + s_red[1][2] + s_red[1][3];
  }
}

__global__ __launch_bounds__(DH) void kv_attention_combine_kernel(const float* __restrict__ ws,
                                                                  int nchunk, int v_had,
                                                                  float cnorm,
                                                                  uint16_t* __restrict__ out) {
  __shared__ float s_o[DH];
  const int d = (int)__builtin_amdgcn_workitem_id_x();
  const int bh = (int)__builtin_amdgcn_workgroup_id_x();
  const float* w = ws + (int64_t)bh * nchunk * WS_FLOATS;
  float m = -__builtin_inff();
  for (int i = 0; i < nchunk; ++i) m = fmaxf(m, w[i * WS_FLOATS]);
  float l = 0.0f, o = 0.0f;
  for (int i = 0; i < nchunk; ++i) {
    const float e = __builtin_amdgcn_exp2f((w[i * WS_FLOATS] - m) * LOG2E);
    l = __builtin_fmaf(e, w[i * WS_FLOATS + 1], l);
    o = __builtin_fmaf(e, w[i * WS_FLOATS + 2 + d], o);
  }
  o = o / l;
  if (v_had) {
    s_o[d] = o;
    __syncthreads();
    float a = 0.0f;
    for (int i = 0; i < DH; ++i) a = __builtin_fmaf(s_o[i], had_sign(i, d), a);
    o = a * cnorm;
  }
  out[(int64_t)bh * DH + d] = f32_to_bf16_rne(o);
}

}  // namespace

int64_t kv_attention_workspace_floats(int64_t BH, int64_t seq_len) {
  return BH * ((seq_len + CH - 1) / CH) * WS_FLOATS;
}

hipError_t launch_kv_attention_decode(const uint16_t* q, const uint8_t* k_codes,
                                      const uint16_t* k_scale, const int16_t* k_zero,
                                      const uint8_t* v_codes, const uint16_t* v_scale,
                                      const int16_t* v_zero, int64_t BH, int64_t S_cap,
                                      int64_t seq_len, float sm_scale, bool v_hadamard,
                                      uint16_t* out, float* workspace, hipStream_t stream) {
  const int nchunk = (int)((seq_len + CH - 1) / CH);
  const float cnorm = (float)(1.0 / __builtin_sqrt((double)DH));
  hipLaunchKernelGGL(kv_attention_chunk_kernel, dim3((unsigned)(BH * nchunk)), dim3(THREADS), 0,
                     stream, q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, S_cap,
                     (int)seq_len, nchunk, sm_scale, cnorm, workspace);
  hipLaunchKernelGGL(kv_attention_combine_kernel, dim3((unsigned)BH), dim3(DH), 0, stream,
                     workspace, nchunk, v_hadamard ? 1 : 0, cnorm, out);
  return hipGetLastError();
}

}  // namespace offq
