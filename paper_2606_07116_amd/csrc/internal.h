// Host-side launchers shared between the kernel files and the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace offq {

// Fused rotate + quantize over n_groups groups of g channels.  Group q lives at
// row q / G, channels [(q % G) * g, (q % G + 1) * g) of x (row stride ldx).
hipError_t launch_rotate_quantize(const uint16_t* x, int64_t n_groups, int G,
                                  int64_t ldx, int log2g, bool hadamard,
                                  uint8_t* codes, int64_t ldc_bytes,
                                  uint16_t* scale, int16_t* zero, float* y_debug,
                                  int64_t ldy, hipStream_t stream);

hipError_t launch_w4a4_gemm(const uint8_t* a_codes, const uint16_t* a_scale,
                            const int16_t* a_zero, const uint8_t* w_codes,
                            const uint16_t* w_scale, const int32_t* w_colsum,
                            int64_t M, int64_t N, int64_t K, int log2g,
                            uint16_t* y, int64_t ldy, int32_t* acc_debug,
                            hipStream_t stream);

// Several groups per row (g < K, g >= 128): MFMA GEMM with per-group fold.
bool gemm_grouped_supported(int64_t M, int64_t N, int64_t K, int log2g);
hipError_t launch_w4a4_gemm_grouped(const uint8_t* a_codes, const uint16_t* a_scale,
                                    const int16_t* a_zero, const uint8_t* w_codes,
                                    const uint16_t* w_scale, const int32_t* w_colsum, int64_t M,
                                    int64_t N, int64_t K, int log2g, uint16_t* y, int64_t ldy,
                                    int32_t* acc_debug, hipStream_t stream);

// Decode (M <= 16) on MFMA: 16-channel row tiles, K split over 4 waves.
bool gemv_mfma_supported(int64_t M, int64_t N, int64_t K, int log2g);
hipError_t launch_w4a4_gemv_mfma(const uint8_t* a_codes, const uint16_t* a_scale,
                                 const int16_t* a_zero, const uint8_t* w_codes,
                                 const uint16_t* w_scale, const int32_t* w_colsum, int64_t M,
                                 int64_t N, int64_t K, int log2g, uint16_t* y, int64_t ldy,
                                 int32_t* acc_debug, hipStream_t stream);

hipError_t launch_w4a4_gemv(const uint8_t* a_codes, const uint16_t* a_scale,
                            const int16_t* a_zero, const uint8_t* w_codes,
                            const uint16_t* w_scale, const int32_t* w_colsum,
                            int64_t M, int64_t N, int64_t K, int log2g,
                            uint16_t* y, int64_t ldy, int32_t* acc_debug,
                            hipStream_t stream);

hipError_t launch_pack_weights(const float* w, int64_t N, int64_t K, int log2g,
                               uint8_t* w_codes, uint16_t* w_scale,
                               int32_t* w_colsum, hipStream_t stream);

// One decode step of attention over the 4-bit KV cache (head_dim 128).
int64_t kv_attention_workspace_floats(int64_t BH, int64_t seq_len);
hipError_t launch_kv_attention_decode(const uint16_t* q, const uint8_t* k_codes,
                                      const uint16_t* k_scale, const int16_t* k_zero,
                                      const uint8_t* v_codes, const uint16_t* v_scale,
                                      const int16_t* v_zero, int64_t BH, int64_t group,
                                      int64_t S_cap, int64_t seq_len, float sm_scale,
                                      bool v_hadamard, uint16_t* out, uint8_t* qcodes,
                                      uint16_t* qscale, int16_t* qzero, float* workspace,
                                      hipStream_t stream);

// The same step's chunk records in a static device array (16 MiB per device,
// kept until the process ends) for callers that cannot allocate:
// kv_attention_scratch gives the current device's address of that array.
constexpr int64_t kKvScratchBytes = int64_t(16) << 20;
hipError_t kv_attention_scratch(float** ptr);

// decoder-layer kernels (layer_ops.hip)
hipError_t launch_add_rmsnorm(const uint16_t* x, int64_t ldx, const uint16_t* res, int64_t ldr,
                              int64_t M, int64_t D, float eps, uint16_t* h_out, int64_t ldh,
                              uint16_t* y_out, int64_t ldy, hipStream_t stream);
hipError_t launch_swiglu(const uint16_t* gu, int64_t ldg, int64_t M, int64_t F, uint16_t* out,
                         int64_t ldo, hipStream_t stream);
hipError_t launch_add_rmsnorm_quant(const uint16_t* x, int64_t ldx, const uint16_t* res,
                                    int64_t ldr, int64_t M, int64_t D, float eps, int log2g,
                                    uint16_t* h_out, int64_t ldh, uint8_t* codes, uint16_t* scale,
                                    int16_t* zero, uint16_t* y_dbg, int64_t ldy,
                                    hipStream_t stream);
hipError_t launch_swiglu_rq(const uint16_t* gu, int64_t ldg, int64_t M, int64_t F, uint8_t* codes,
                            uint16_t* scale, int16_t* zero, float* y_dbg, hipStream_t stream);
hipError_t launch_kv_attention_prefill(const uint16_t* q, int64_t B, int64_t T, int64_t Hq,
                                       int64_t Hkv, int64_t past, const uint8_t* kc,
                                       const uint16_t* ks, const int16_t* kz, const uint8_t* vc,
                                       const uint16_t* vs, const int16_t* vz, int64_t s_cap,
                                       float sm_scale, bool v_had, uint16_t* out,
                                       hipStream_t stream);
hipError_t launch_rope_kv_append(const uint16_t* qkv, int64_t ldq, int64_t M, int64_t T,
                                 int64_t Hq, int64_t Hkv, const int32_t* positions, double rope_base,
                                 bool k_had, bool v_had, uint16_t* q_out, uint8_t* kc,
                                 uint16_t* ks, int16_t* kz, uint8_t* vc, uint16_t* vs,
                                 int16_t* vz, int64_t s_cap, float* k_dbg, float* v_dbg,
                                 hipStream_t stream);

// offline calibration (calibration.hip)
hipError_t launch_top1_select(const uint16_t* x, int64_t n_seq, int64_t L, int64_t D,
                              int64_t ld_tok, int64_t ld_seq, int32_t* idx, float* X, int64_t ldX,
                              float* linf, hipStream_t stream);
hipError_t launch_channel_absmax(const uint16_t* x, int64_t rows, int64_t D, int64_t ldx,
                                 double* out, hipStream_t stream);
hipError_t launch_gram(const float* X, int64_t N, int64_t D, int64_t ldX, double* C, int64_t ldC,
                       hipStream_t stream);
int64_t eigh_workspace_doubles(int64_t D);
hipError_t launch_eigh(const double* C, int64_t ldC, int64_t D, double* evals, double* U,
                       int64_t ldU, double* ws, int max_sweeps, double tol, int* sweeps_done,
                       double* rel_off, hipStream_t stream);
hipError_t launch_group_permutation(const double* key, int64_t D, int64_t g, int32_t* perm,
                                    int32_t* rank, hipStream_t stream);
hipError_t launch_build_rotation(const double* U, int64_t ldU, int64_t D, const int32_t* perm,
                                 int log2g, float* R, int64_t ldR, hipStream_t stream);
hipError_t launch_fuse_weights(const float* W, int64_t ldW, int64_t N, int64_t K, const float* R,
                               int64_t ldR, float* Wo, int64_t ldo, hipStream_t stream);
hipError_t launch_permute_rows(const float* W, int64_t ldW, int64_t N, int64_t K,
                               const int32_t* perm, float* Wo, int64_t ldo, hipStream_t stream);

}  // namespace offq
