// Offline calibration on the GPU: the steps that turn calibration activations
// into the rotations and permutations the online path relies on.
//
// * top-1 selection (sec. 3.1 "Top-1 PCA"): per calibration sequence, the
//   token with the largest L-infinity norm;
// * C = X^T X / N over the selected tokens (Eq. 2), in fp64;
// * the eigendecomposition C = U Lambda U^T, eigenvalues descending (Eq. 2),
//   by parallel cyclic Jacobi in fp64 (see below);
// * the grouping permutation (sec. 3.2 "Group-Wise Offsetting"): the G
//   channels with the largest statistic lead the G groups in descending order,
//   the rest fill the groups in ascending order ("sorted grouping", sec. 4.3);
// * the rotation R = U P blockdiag(H_g / sqrt(g)) (sec. 3.3 step 2(1)) and
//   its fusion into the weights W' = W R, rows permuted for P4 (step 2(4)),
//   before the per-channel 4-bit packing (offq_pack_weights).
//
// Jacobi: each step rotates D/2 disjoint index pairs at once, each rotation
// zeroing its pair's off-diagonal entry (the symmetric 2x2 Schur rotation):
// A <- J^T A J, V <- V J, written out of place (ping-pong buffers) and with
// the slots permuted by one move of the round-robin (circle) tournament, so
// that the pairs are always the adjacent slots (2k, 2k+1) and D - 1 steps
// meet every pair once (a sweep).  Sweeps repeat until the off-diagonal norm
// is below tol times the Frobenius norm.
#include "common.h"
#include "internal.h"

namespace offq {
namespace {

__device__ __forceinline__ float cmax(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// ---------------------------------------------------------------- top-1 tokens
// L-infinity norm of every token row (one wave per token; D % 8 == 0).
__global__ __launch_bounds__(256) void token_linf_kernel(const uint16_t* __restrict__ x,
                                                         int64_t ld_tok, int64_t ld_seq, int L,
                                                         int D, int64_t ntok,
                                                         float* __restrict__ linf) {
  const int lane = threadIdx.x & 63;
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= ntok) return;
  const int64_t seq = w / L, t = w - seq * L;
  const uint4* row = reinterpret_cast<const uint4*>(x + seq * ld_seq + t * ld_tok);
  float m = 0.0f;
  for (int c = lane; c < D / 8; c += 64) {
    const uint4 v = row[c];
    const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int k = 0; k < 4; ++k)
      m = fmaxf(m, fmaxf(fabsf(bf16_lo(u[k])), fabsf(bf16_hi(u[k]))));
  }
  m = cmax(m);
  if (lane == 0) linf[w] = m;
}

// Per sequence: the first token of largest norm; its row copied as fp32.
__global__ __launch_bounds__(256) void top1_gather_kernel(const uint16_t* __restrict__ x,
                                                          int64_t ld_tok, int64_t ld_seq, int L,
                                                          int D, const float* __restrict__ linf,
                                                          int32_t* __restrict__ idx,
                                                          float* __restrict__ X, int64_t ldX) {
  __shared__ float sv[4];
  __shared__ int si[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t seq = blockIdx.x;
  float bv = -1.0f;
  int bi = 0x7fffffff;
  for (int t = tid; t < L; t += 256) {
    const float v = linf[seq * L + t];
    if (v > bv) {  // t increases: the first maximum of this thread stays
      bv = v;
      bi = t;
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float ov = __shfl_xor(bv, o);
    const int oi = __shfl_xor(bi, o);
    if (ov > bv || (ov == bv && oi < bi)) {
      bv = ov;
      bi = oi;
    }
  }
  if (lane == 0) {
    sv[wave] = bv;
    si[wave] = bi;
  }
  __syncthreads();
  bv = sv[0];
  bi = si[0];
  for (int w = 1; w < 4; ++w)
    if (sv[w] > bv || (sv[w] == bv && si[w] < bi)) {
      bv = sv[w];
      bi = si[w];
    }
  if (tid == 0) idx[seq] = bi;
  const uint16_t* row = x + seq * ld_seq + (int64_t)bi * ld_tok;
  for (int c = tid; c < D; c += 256) X[seq * ldX + c] = bf16_lo(row[c]);
}

// Per-channel maximum of |x| over rows (the statistic that picks the outlier
// channels of the down-projection input, sec. 3.3 step 2(4)).  Block of 256
// channels x 16 row slices; column maxima combined through LDS.
__global__ __launch_bounds__(256) void channel_absmax_kernel(const uint16_t* __restrict__ x,
                                                             int64_t rows, int D, int64_t ldx,
                                                             double* __restrict__ out) {
  const int c = (int)blockIdx.x * 256 + (int)threadIdx.x;
  if (c >= D) return;
  float m = 0.0f;
  for (int64_t r = 0; r < rows; ++r) m = fmaxf(m, fabsf(bf16_lo(x[r * ldx + c])));
  out[c] = (double)m;
}

// ---------------------------------------------------------------- C = X^T X / N
// 64 x 64 output tiles of the upper triangle (tile row <= tile column), each
// thread 4 x 4 outputs; k in slices of 16 rows staged as fp64 in LDS.  Tiles
// below the diagonal are written as the transposes of those above, so C is
// exactly symmetric.
__global__ __launch_bounds__(256) void gram_kernel(const float* __restrict__ X, int N, int D,
                                                   int64_t ldX, double* __restrict__ C,
                                                   int64_t ldC) {
  const int ti = blockIdx.y, tj = blockIdx.x;
  if (ti > tj) return;
  __shared__ double As[16][64], Bs[16][64];
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const int i0 = ti * 64, j0 = tj * 64;
  double acc[4][4] = {};
  for (int n0 = 0; n0 < N; n0 += 16) {
    for (int e = tid; e < 16 * 64; e += 256) {
      const int k = e >> 6, c = e & 63;
      const int n = n0 + k;
      As[k][c] = (n < N && i0 + c < D) ? (double)X[(int64_t)n * ldX + i0 + c] : 0.0;
      Bs[k][c] = (n < N && j0 + c < D) ? (double)X[(int64_t)n * ldX + j0 + c] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      double a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a[u] = As[k][ty * 4 + u];
        b[u] = Bs[k][tx * 4 + u];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = __builtin_fma(a[u], b[v], acc[u][v]);
    }
    __syncthreads();
  }
  const double inv = 1.0 / (double)N;
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int i = i0 + ty * 4 + u, j = j0 + tx * 4 + v;
      if (i < D && j < D && i <= j) {
        const double c = acc[u][v] * inv;
        C[(int64_t)i * ldC + j] = c;
        C[(int64_t)j * ldC + i] = c;
      }
    }
}

// ---------------------------------------------------------------- Jacobi
// Slot of the circle tournament after one round (P = D / 2 pairs; slot 2k is
// the "top" player of pair k, 2k + 1 the "bottom" one).  Slot 0 stays; the
// others move one place around the ring 1 -> 2 -> 4 -> ... -> 2P-2 ->
// 2P-1 -> 2P-3 -> ... -> 3 -> 1.
__device__ __forceinline__ int next_slot(int x, int P) {
  if (x == 0 || P == 1) return x;  // D = 2: one pair, nothing moves
  if (x & 1) return x == 1 ? 2 : x - 2;
  return x == 2 * P - 2 ? 2 * P - 1 : x + 2;
}

// (c, s) of the rotation that zeroes a[p][q] of pair k (Golub & Van Loan's
// symmetric Schur decomposition of a 2 x 2 block); identity when the entry is
// negligible against the diagonal.
__device__ __forceinline__ double2 jacobi_rotation(const double* __restrict__ A, int64_t ldA,
                                                   int k) {
  const double app = A[(int64_t)(2 * k) * ldA + 2 * k];
  const double aqq = A[(int64_t)(2 * k + 1) * ldA + 2 * k + 1];
  const double apq = A[(int64_t)(2 * k) * ldA + 2 * k + 1];
  double c = 1.0, s = 0.0;
  if (fabs(apq) > 1e-300 && fabs(apq) > 1e-18 * __builtin_sqrt(fabs(app * aqq))) {
    const double tau = (aqq - app) / (2.0 * apq);
    const double t = (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + __builtin_sqrt(1.0 + tau * tau));
    c = 1.0 / __builtin_sqrt(1.0 + t * t);
    s = t * c;
  }
  return make_double2(c, s);
}

// One Jacobi step, A_out = perm(J^T A_in J), on the upper triangle: the
// matrices hold (and the steps read and write) only the entries (r, c) with
// r <= c; the lower ones are left stale.  A workgroup takes a 16 x 16 tile of
// 2 x 2 blocks (pair rows bi, pair columns bj >= bi); block (i, j), i <= j,
// becomes B' = R_i^T B R_j with R = [[c, s], [-s, c]].  The rotations come
// from A_in's diagonal blocks, which every workgroup reads (the step writes
// A_out only), and the diagonal tiles store them for the eigenvector update.
// An entry moved to (r', c') with r' > c' is stored at (c', r'); the rotated
// tile is staged in LDS and written by rows.
__global__ __launch_bounds__(256) void jacobi_a_tile_kernel(const double* __restrict__ A,
                                                            int64_t ld, int P,
                                                            double2* __restrict__ cs_out,
                                                            double* __restrict__ Ao) {
  // workgroup b -> tile (bi, bj) of the upper triangle, b = bj (bj + 1) / 2 + bi
  const int b = blockIdx.x;
  int bj = (int)((__builtin_sqrtf(8.0f * (float)b + 1.0f) - 1.0f) * 0.5f);
  while ((bj + 1) * (bj + 2) / 2 <= b) ++bj;
  while (bj * (bj + 1) / 2 > b) --bj;
  const int bi = b - bj * (bj + 1) / 2;
  __shared__ double2 s_r[2][16];
  __shared__ double s_t[32][33];
  const int tid = threadIdx.x;
  const int pi = tid >> 4, pj = tid & 15;
  const int i = bi * 16 + pi, j = bj * 16 + pj;
  const bool ok = i < P && j < P;
  double b00 = 0.0, b01 = 0.0, b10 = 0.0, b11 = 0.0;
  if (ok && i <= j) {
    const double* a0 = A + (int64_t)(2 * i) * ld + 2 * j;
    b00 = a0[0];
    b01 = a0[1];
    b10 = i == j ? b01 : a0[ld];  // (2i + 1, 2i) is below the diagonal
    b11 = a0[ld + 1];
  }
  if (tid < 32) {
    const int k = (tid < 16 ? bi : bj) * 16 + (tid & 15);
    if (k < P) {
      const double2 r = jacobi_rotation(A, ld, k);
      s_r[tid >> 4][tid & 15] = r;
      if (bi == bj && tid < 16) cs_out[k] = r;
    }
  }
  __syncthreads();
  double n00 = 0.0, n01 = 0.0, n10 = 0.0, n11 = 0.0;
  if (ok) {
    const double2 ri = s_r[0][pi], rj = s_r[1][pj];
    const double t00 = b00 * rj.x - b01 * rj.y, t01 = b00 * rj.y + b01 * rj.x;
    const double t10 = b10 * rj.x - b11 * rj.y, t11 = b10 * rj.y + b11 * rj.x;
    n00 = ri.x * t00 - ri.y * t10;
    n01 = ri.x * t01 - ri.y * t11;
    n10 = ri.y * t00 + ri.x * t10;
    n11 = ri.y * t01 + ri.x * t11;
    if (i == j) {
      n01 = 0.0;  // what the rotation is for
      n10 = 0.0;
    }
  }
  s_t[2 * pi][2 * pj] = n00;
  s_t[2 * pi][2 * pj + 1] = n01;
  s_t[2 * pi + 1][2 * pj] = n10;
  s_t[2 * pi + 1][2 * pj + 1] = n11;
  __syncthreads();
  // writes: 32 lanes per tile row, 8 rows per pass; in a diagonal tile only
  // the entries on and above the diagonal
  const int ec = tid & 31;
  const int D = 2 * P;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int er = (tid >> 5) + 8 * u;
    const int gr = bi * 32 + er, gc = bj * 32 + ec;
    if (gr < D && gc < D && (bi != bj || er <= ec)) {
      const int r1 = next_slot(gr, P), c1 = next_slot(gc, P);
      Ao[(int64_t)min(r1, c1) * ld + max(r1, c1)] = s_t[er][ec];
    }
  }
}

__global__ __launch_bounds__(256) void identity_kernel(double* __restrict__ V, int64_t ldV, int D) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int64_t r = blockIdx.y;
  if (c < D) V[r * ldV + c] = (c == r) ? 1.0 : 0.0;
}

// The slots other than 0 form one ring under next_slot: R = 1, 2, 4, ...,
// 2P-2, 2P-1, 2P-3, ..., 3.  ring_index(x) is x's place in it; ring_slot is
// the inverse.
__device__ __forceinline__ int ring_index(int x, int P) {
  if (x == 1) return 0;
  if (!(x & 1)) return x >> 1;
  return x == 2 * P - 1 ? P : 2 * P - 1 - (x >> 1);
}
__device__ __forceinline__ int ring_slot(int i, int P) {
  if (i == 0) return 1;
  return i < P ? 2 * i : 4 * P - 1 - 2 * i;
}
// Where the entry that sits in slot x after t steps of a batch was at the
// batch's start (every step moves slot R[i] to R[i + 1]); t = steps mod
// (2P - 1), the length of the ring.
__device__ __forceinline__ int batch_loc(int x, int t, int P) {
  if (x == 0) return 0;
  int i = ring_index(x, P) - t;
  if (i < 0) i += 2 * P - 1;
  return ring_slot(i, P);
}

// LDS position of slot x of a row: even slots first, then odd ones, so that
// the pair members of consecutive pairs are consecutive (unit-stride LDS
// accesses).
__device__ __forceinline__ int lds_pos(int x, int P) { return (x & 1) * P + (x >> 1); }

// V <- V J_1 ... J_S for S steps at once: a workgroup holds NR rows of V in
// LDS at their batch-start slots; step tau rotates the pairs (2k, 2k+1) of
// that step's slots, found through batch_loc, so nothing moves until the
// rows are written back in the slot order after the S steps.  V is read and
// written once per S steps instead of once per step, and each rotation and
// slot lookup serves the NR rows.
template <int NR>
__global__ __launch_bounds__(512) void jacobi_v_batch_kernel(const double* __restrict__ V,
                                                             int64_t ldV, int D, int P,
                                                             const double2* __restrict__ cs,
                                                             int S, double* __restrict__ Vo) {
  extern __shared__ double rows[];
  const int64_t r0 = (int64_t)blockIdx.x * NR;
  const int nr = (int)min((int64_t)NR, (int64_t)D - r0);
  const int tid = threadIdx.x;
  const int L = 2 * P - 1;
  for (int q = 0; q < nr; ++q)
    for (int c = tid; c < D; c += 512) rows[q * D + lds_pos(c, P)] = V[(r0 + q) * ldV + c];
  __syncthreads();
  for (int tau = 0; tau < S; ++tau) {
    const double2* rot = cs + (int64_t)tau * P;
    const int t = tau % L;
    // the pairs of a step are disjoint: up to 4 per thread are all loaded
    // before any is stored, so the LDS latencies overlap
    for (int k0 = tid; k0 < P; k0 += 4 * 512) {
      int lp[4], lq[4];
      double2 rk[4];
      double vp[4][NR], vq[4][NR];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int k = k0 + u * 512;
        if (k < P) {
          lp[u] = lds_pos(batch_loc(2 * k, t, P), P);
          lq[u] = lds_pos(batch_loc(2 * k + 1, t, P), P);
          rk[u] = rot[k];
#pragma unroll
          for (int q = 0; q < NR; ++q) {
            vp[u][q] = rows[q * D + lp[u]];
            vq[u][q] = rows[q * D + lq[u]];
          }
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (k0 + u * 512 < P) {
#pragma unroll
          for (int q = 0; q < NR; ++q) {
            rows[q * D + lp[u]] = vp[u][q] * rk[u].x - vq[u][q] * rk[u].y;
            rows[q * D + lq[u]] = vp[u][q] * rk[u].y + vq[u][q] * rk[u].x;
          }
        }
      }
    }
    __syncthreads();
  }
  const int t = S % L;
  for (int q = 0; q < nr; ++q)
    for (int c = tid; c < D; c += 512)
      Vo[(r0 + q) * ldV + c] = rows[q * D + lds_pos(batch_loc(c, t, P), P)];
}

// Partial sums of the off-diagonal and total squares of a symmetric A held in
// its upper triangle (one per row).
__global__ __launch_bounds__(256) void offnorm_kernel(const double* __restrict__ A, int64_t ldA,
                                                      int D, double* __restrict__ part) {
  __shared__ double s_off[4], s_all[4];
  const int64_t r = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  double off = 0.0, all = 0.0;
  for (int c = (int)r + tid; c < D; c += 256) {
    const double v = A[r * ldA + c];
    if (c != r) off = __builtin_fma(v, v, off);
    else all = v * v;
  }
  off *= 2.0;  // (r, c) and (c, r)
  all += off;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    off += __shfl_xor(off, o);
    all += __shfl_xor(all, o);
  }
  if (lane == 0) {
    s_off[wave] = off;
    s_all[wave] = all;
  }
  __syncthreads();
  if (tid == 0) {
    part[2 * r] = s_off[0] + s_off[1] + s_off[2] + s_off[3];
    part[2 * r + 1] = s_all[0] + s_all[1] + s_all[2] + s_all[3];
  }
}

__global__ __launch_bounds__(256) void offnorm_total_kernel(const double* __restrict__ part,
                                                            int D, double* __restrict__ tot) {
  __shared__ double s_off[4], s_all[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  double off = 0.0, all = 0.0;
  for (int r = tid; r < D; r += 256) {
    off += part[2 * r];
    all += part[2 * r + 1];
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    off += __shfl_xor(off, o);
    all += __shfl_xor(all, o);
  }
  if (lane == 0) {
    s_off[wave] = off;
    s_all[wave] = all;
  }
  __syncthreads();
  if (tid == 0) {
    tot[0] = s_off[0] + s_off[1] + s_off[2] + s_off[3];
    tot[1] = s_all[0] + s_all[1] + s_all[2] + s_all[3];
  }
}

// rank[i] = #{j : key[j] > key[i], or key[j] == key[i] and j < i}: the
// position of i in descending order, ties by index (O(D^2) comparisons).
__global__ __launch_bounds__(256) void rank_desc_kernel(const double* __restrict__ key,
                                                        int64_t stride, int D,
                                                        int32_t* __restrict__ rank) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= D) return;
  const double ki = key[(int64_t)i * stride];
  int r = 0;
  for (int j = 0; j < D; ++j) {
    const double kj = key[(int64_t)j * stride];
    r += (kj > ki || (kj == ki && j < i)) ? 1 : 0;
  }
  rank[i] = r;
}

// Sorted eigenpairs: evals[k] = diag slot with descending rank k; column k of
// U = that slot's column of V, its sign making the largest |entry| (first
// such) positive.
__global__ __launch_bounds__(256) void eig_gather_kernel(const double* __restrict__ A,
                                                         int64_t ldA, const double* __restrict__ V,
                                                         int64_t ldV, int D,
                                                         const int32_t* __restrict__ rank,
                                                         double* __restrict__ evals,
                                                         double* __restrict__ U, int64_t ldU) {
  __shared__ double s_v[4];
  __shared__ int s_i[4];
  const int slot = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int k = rank[slot];
  // sign: the entry of largest magnitude, first index on ties
  double bv = -1.0;
  int bi = 0x7fffffff;
  for (int r = tid; r < D; r += 256) {
    const double a = fabs(V[(int64_t)r * ldV + slot]);
    if (a > bv) {
      bv = a;
      bi = r;
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const double ov = __shfl_xor(bv, o);
    const int oi = __shfl_xor(bi, o);
    if (ov > bv || (ov == bv && oi < bi)) {
      bv = ov;
      bi = oi;
    }
  }
  if (lane == 0) {
    s_v[wave] = bv;
    s_i[wave] = bi;
  }
  __syncthreads();
  bv = s_v[0];
  bi = s_i[0];
  for (int w = 1; w < 4; ++w)
    if (s_v[w] > bv || (s_v[w] == bv && s_i[w] < bi)) {
      bv = s_v[w];
      bi = s_i[w];
    }
  const double sg = V[(int64_t)bi * ldV + slot] < 0.0 ? -1.0 : 1.0;
  for (int r = tid; r < D; r += 256) U[(int64_t)r * ldU + k] = sg * V[(int64_t)r * ldV + slot];
  if (tid == 0) evals[k] = A[(int64_t)slot * ldA + slot];
}

// ---------------------------------------------------------------- grouping
// Sorted grouping: descending rank r < G -> head of group r (slot r g);
// the rest, ranked ascending among themselves (ties by index), fill the other
// g - 1 slots of the groups in order.
__global__ __launch_bounds__(256) void group_perm_kernel(const double* __restrict__ key, int D,
                                                         int g, const int32_t* __restrict__ rank,
                                                         int32_t* __restrict__ perm) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= D) return;
  const int G = D / g;
  const int r = rank[i];
  if (r < G) {
    perm[r * g] = i;
    return;
  }
  const double ki = key[i];
  int a = 0;  // ascending position among the non-heads
  for (int j = 0; j < D; ++j) {
    if (rank[j] < G) continue;
    const double kj = key[j];
    a += (kj < ki || (kj == ki && j < i)) ? 1 : 0;
  }
  perm[(a / (g - 1)) * g + 1 + a % (g - 1)] = i;
}

// ---------------------------------------------------------------- rotation
// R[r][c] = sum_t U[r][perm[gc + t]] H_g[t][c - gc] / sqrt(g) for column c in
// group gc (U = identity if null, perm = identity if null, no Hadamard if
// g == 1): one workgroup per row, the gathered row in LDS, fp64 butterflies.
__global__ __launch_bounds__(256) void rotation_kernel(const double* __restrict__ U, int64_t ldU,
                                                       int D, const int32_t* __restrict__ perm,
                                                       int log2g, float* __restrict__ R,
                                                       int64_t ldR) {
  extern __shared__ double row[];
  const int64_t r = blockIdx.x;
  const int tid = threadIdx.x;
  for (int c = tid; c < D; c += 256) {
    const int src = perm ? perm[c] : c;
    // an index outside [0, D) (not a permutation) contributes zero
    row[c] = (src < 0 || src >= D) ? 0.0 : U ? U[r * ldU + src] : (src == r ? 1.0 : 0.0);
  }
  __syncthreads();
  for (int h = 1; h < (1 << log2g); h <<= 1) {
    for (int b = tid; b < D / 2; b += 256) {
      // butterfly b: indices (x, x + h) with x having bit h clear
      const int x = ((b & ~(h - 1)) << 1) | (b & (h - 1));
      const double u = row[x], v = row[x + h];
      row[x] = u + v;
      row[x + h] = u - v;
    }
    __syncthreads();
  }
  const double scale = 1.0 / __builtin_sqrt((double)(1 << log2g));
  for (int c = tid; c < D; c += 256) R[r * ldR + c] = (float)(row[c] * scale);
}

// W_out = W R (fp32; 64 x 64 output tiles, 4 x 4 per thread, k slices of 16).
__global__ __launch_bounds__(256) void fuse_gemm_kernel(const float* __restrict__ W, int64_t ldW,
                                                        int N, int K, const float* __restrict__ R,
                                                        int64_t ldR, float* __restrict__ Wo,
                                                        int64_t ldo) {
  __shared__ float As[16][65], Bs[16][64];
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const int n0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int e = tid; e < 16 * 64; e += 256) {
      const int rr = e >> 4, kk = e & 15;   // W tile: 64 rows x 16 k
      const int n = n0 + rr, k = k0 + kk;
      As[kk][rr] = (n < N && k < K) ? W[(int64_t)n * ldW + k] : 0.0f;
      const int kb = e >> 6, cb = e & 63;   // R tile: 16 k x 64 columns
      Bs[kb][cb] = (k0 + kb < K && c0 + cb < K) ? R[(int64_t)(k0 + kb) * ldR + c0 + cb] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      float a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a[u] = As[k][ty * 4 + u];
        b[u] = Bs[k][tx * 4 + u];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = __builtin_fmaf(a[u], b[v], acc[u][v]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int n = n0 + ty * 4 + u, c = c0 + tx * 4 + v;
      if (n < N && c < K) Wo[(int64_t)n * ldo + c] = acc[u][v];
    }
}

__global__ __launch_bounds__(256) void permute_rows_kernel(const float* __restrict__ W,
                                                           int64_t ldW, int N, int K,
                                                           const int32_t* __restrict__ perm,
                                                           float* __restrict__ Wo, int64_t ldo) {
  const int64_t s = blockIdx.x;
  const int p = perm[s];
  const bool ok = p >= 0 && p < N;  // an index outside the rows gives a zero row
  const float* src = W + (int64_t)(ok ? p : 0) * ldW;
  for (int c = threadIdx.x; c < K; c += 256) Wo[s * ldo + c] = ok ? src[c] : 0.0f;
}

}  // namespace

hipError_t launch_top1_select(const uint16_t* x, int64_t n_seq, int64_t L, int64_t D,
                              int64_t ld_tok, int64_t ld_seq, int32_t* idx, float* X, int64_t ldX,
                              float* linf, hipStream_t stream) {
  const int64_t ntok = n_seq * L;
  hipLaunchKernelGGL(token_linf_kernel, dim3((unsigned)((ntok + 3) / 4)), dim3(256), 0, stream, x,
                     ld_tok, ld_seq, (int)L, (int)D, ntok, linf);
  hipLaunchKernelGGL(top1_gather_kernel, dim3((unsigned)n_seq), dim3(256), 0, stream, x, ld_tok,
                     ld_seq, (int)L, (int)D, linf, idx, X, ldX);
  return hipGetLastError();
}

hipError_t launch_channel_absmax(const uint16_t* x, int64_t rows, int64_t D, int64_t ldx,
                                 double* out, hipStream_t stream) {
  hipLaunchKernelGGL(channel_absmax_kernel, dim3((unsigned)((D + 255) / 256)), dim3(256), 0,
                     stream, x, rows, (int)D, ldx, out);
  return hipGetLastError();
}

hipError_t launch_gram(const float* X, int64_t N, int64_t D, int64_t ldX, double* C, int64_t ldC,
                       hipStream_t stream) {
  const unsigned T = (unsigned)((D + 63) / 64);
  hipLaunchKernelGGL(gram_kernel, dim3(T, T), dim3(256), 0, stream, X, (int)N, (int)D, ldX, C,
                     ldC);
  return hipGetLastError();
}

constexpr int JB = 64;  // Jacobi steps per batch of V updates

int64_t eigh_workspace_doubles(int64_t D) {
  // A, A', V, V'; partial norms (2 D) and totals (2); the rotations of a
  // batch (JB steps of D / 2 pairs, 2 doubles each); ranks (D int32)
  return 4 * D * D + 2 * D + 2 + (int64_t)JB * D + D / 2 + 2;
}

hipError_t launch_eigh(const double* C, int64_t ldC, int64_t D, double* evals, double* U,
                       int64_t ldU, double* ws, int max_sweeps, double tol, int* sweeps_done,
                       double* rel_off, hipStream_t stream) {
  const int P = (int)(D / 2);
  double* A0 = ws;
  double* A1 = A0 + D * D;
  double* V0 = A1 + D * D;
  double* V1 = V0 + D * D;
  double* part = V1 + D * D;          // 2 D
  double* tot = part + 2 * D;         // 2
  double2* cs = reinterpret_cast<double2*>(tot + 2);  // JB x P pairs (16-byte aligned)
  int32_t* rank = reinterpret_cast<int32_t*>(cs + (int64_t)JB * P);  // D ints
  hipError_t e;
  e = hipMemcpy2DAsync(A0, D * sizeof(double), C, ldC * sizeof(double), D * sizeof(double), D,
                       hipMemcpyDeviceToDevice, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(identity_kernel, dim3((unsigned)((D + 255) / 256), (unsigned)D), dim3(256), 0,
                     stream, V0, D, (int)D);
  const unsigned nt = (unsigned)((P + 15) / 16);
  const dim3 ga(nt * (nt + 1) / 2);  // tiles of the upper triangle
  // V rows per workgroup of the batched update: as many as 128 KB of LDS hold, at most 4
  const int nr = D <= 4096 ? 4 : 2;  // D <= 8192
  double h_tot[2] = {0.0, 0.0};
  int sweeps = 0;
  double rel = 0.0;
  for (;;) {
    hipLaunchKernelGGL(offnorm_kernel, dim3((unsigned)D), dim3(256), 0, stream, A0, D, (int)D, part);
    hipLaunchKernelGGL(offnorm_total_kernel, dim3(1), dim3(256), 0, stream, part, (int)D, tot);
    e = hipMemcpyAsync(h_tot, tot, sizeof(h_tot), hipMemcpyDeviceToHost, stream);
    if (e != hipSuccess) return e;
    e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return e;
    rel = h_tot[1] > 0.0 ? __builtin_sqrt(h_tot[0] / h_tot[1]) : 0.0;
    if (rel <= tol || sweeps >= max_sweeps) break;
    for (int step = 0; step < D - 1; step += JB) {
      const int nb = (int)std::min<int64_t>(JB, D - 1 - step);
      for (int tau = 0; tau < nb; ++tau) {
        double2* cst = cs + (int64_t)tau * P;
        hipLaunchKernelGGL(jacobi_a_tile_kernel, ga, dim3(256), 0, stream, A0, D, P, cst, A1);
        std::swap(A0, A1);
      }
      const dim3 gv((unsigned)((D + nr - 1) / nr)), bv(512);
      const size_t lv = (size_t)(nr * D) * sizeof(double);
      if (nr == 4)
        hipLaunchKernelGGL(jacobi_v_batch_kernel<4>, gv, bv, lv, stream, V0, D, (int)D, P, cs, nb,
                           V1);
      else if (nr == 2)
        hipLaunchKernelGGL(jacobi_v_batch_kernel<2>, gv, bv, lv, stream, V0, D, (int)D, P, cs, nb,
                           V1);
      else
        hipLaunchKernelGGL(jacobi_v_batch_kernel<1>, gv, bv, lv, stream, V0, D, (int)D, P, cs, nb,
                           V1);
      std::swap(V0, V1);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    ++sweeps;
  }
  if (sweeps_done) *sweeps_done = sweeps;
  if (rel_off) *rel_off = rel;
  // eigenvalues descending: rank the diagonal (stride ldA + 1)
  hipLaunchKernelGGL(rank_desc_kernel, dim3((unsigned)((D + 255) / 256)), dim3(256), 0, stream, A0,
                     D + 1, (int)D, rank);
  hipLaunchKernelGGL(eig_gather_kernel, dim3((unsigned)D), dim3(256), 0, stream, A0, D, V0, D,
                     (int)D, rank, evals, U, ldU);
  return hipGetLastError();
}

hipError_t launch_group_permutation(const double* key, int64_t D, int64_t g, int32_t* perm,
                                    int32_t* rank, hipStream_t stream) {
  const dim3 grid((unsigned)((D + 255) / 256));
  hipLaunchKernelGGL(rank_desc_kernel, grid, dim3(256), 0, stream, key, (int64_t)1, (int)D, rank);
  hipLaunchKernelGGL(group_perm_kernel, grid, dim3(256), 0, stream, key, (int)D, (int)g, rank,
                     perm);
  return hipGetLastError();
}

hipError_t launch_build_rotation(const double* U, int64_t ldU, int64_t D, const int32_t* perm,
                                 int log2g, float* R, int64_t ldR, hipStream_t stream) {
  hipLaunchKernelGGL(rotation_kernel, dim3((unsigned)D), dim3(256), (size_t)D * sizeof(double),
                     stream, U, ldU, (int)D, perm, log2g, R, ldR);
  return hipGetLastError();
}

hipError_t launch_fuse_weights(const float* W, int64_t ldW, int64_t N, int64_t K, const float* R,
                               int64_t ldR, float* Wo, int64_t ldo, hipStream_t stream) {
  hipLaunchKernelGGL(fuse_gemm_kernel, dim3((unsigned)((K + 63) / 64), (unsigned)((N + 63) / 64)),
                     dim3(256), 0, stream, W, ldW, (int)N, (int)K, R, ldR, Wo, ldo);
  return hipGetLastError();
}

hipError_t launch_permute_rows(const float* W, int64_t ldW, int64_t N, int64_t K,
                               const int32_t* perm, float* Wo, int64_t ldo, hipStream_t stream) {
  hipLaunchKernelGGL(permute_rows_kernel, dim3((unsigned)N), dim3(256), 0, stream, W, ldW, (int)N,
                     (int)K, perm, Wo, ldo);
  return hipGetLastError();
}

}  // namespace offq
