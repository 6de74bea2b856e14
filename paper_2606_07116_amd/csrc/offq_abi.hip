// C ABI of the OffQ library: argument validation, device check, dispatch.
// Every entry point validates on the host before enqueuing anything and
// returns a status code; nothing here allocates device memory.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "../../include/offq.h"
#include "common.h"
#include "internal.h"

namespace {

thread_local char g_last_error[512] = "";

offq_status_t fail(offq_status_t status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

offq_status_t ok() {
  g_last_error[0] = '\0';
  return OFFQ_OK;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int ilog2_pow2(int64_t v) {
  if (v <= 0 || (v & (v - 1))) return -1;
  int l = 0;
  while ((int64_t(1) << l) < v) ++l;
  return l;
}

// The kernels are built for gfx950 only; refuse other devices up front.
offq_status_t check_device() {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(OFFQ_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  static thread_local int cached_dev = -1;
  static thread_local bool cached_ok = false;
  if (dev != cached_dev) {
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess)
      return fail(OFFQ_ERR_HIP, "hipGetDeviceProperties: %s", hipGetErrorString(e));
    cached_dev = dev;
    cached_ok = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    if (!cached_ok)
      return fail(OFFQ_ERR_UNSUPPORTED, "device %d is %s; this library is built for gfx950",
                  dev, prop.gcnArchName);
  }
  if (!cached_ok) return fail(OFFQ_ERR_UNSUPPORTED, "device %d is not gfx950", dev);
  return OFFQ_OK;
}

offq_status_t launched(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(OFFQ_ERR_HIP, "%s launch: %s", what, hipGetErrorString(e));
  return ok();
}

constexpr int64_t kMaxGroups = int64_t(1) << 31;

}  // namespace

extern "C" {

int offq_abi_version(void) { return OFFQ_ABI_VERSION; }

const char* offq_status_string(offq_status_t status) {
  switch (status) {
    case OFFQ_OK: return "OFFQ_OK";
    case OFFQ_ERR_INVALID: return "OFFQ_ERR_INVALID";
    case OFFQ_ERR_UNSUPPORTED: return "OFFQ_ERR_UNSUPPORTED";
    case OFFQ_ERR_HIP: return "OFFQ_ERR_HIP";
    default: return "OFFQ_ERR_UNKNOWN";
  }
}

const char* offq_last_error(void) { return g_last_error; }

offq_status_t offq_rotate_quantize(const uint16_t* x, int64_t M, int64_t K, int64_t ldx, int32_t g,
                         int32_t apply_hadamard, uint8_t* codes, uint16_t* scale,
                         int16_t* zero, float* y_debug, void* stream) {
  if (M < 0 || K <= 0) return fail(OFFQ_ERR_INVALID, "M must be >= 0 and K > 0");
  const int lg = ilog2_pow2(g);
  if (lg < 0) return fail(OFFQ_ERR_INVALID, "g = %d is not a power of two", g);
  if (lg < 4 || lg > 13) return fail(OFFQ_ERR_UNSUPPORTED, "g = %d outside [16, 8192]", g);
  if (K % g) return fail(OFFQ_ERR_INVALID, "K = %lld is not a multiple of g = %d", (long long)K, g);
  if (ldx < K || ldx % 8) return fail(OFFQ_ERR_INVALID, "ldx must be >= K and a multiple of 8");
  if (apply_hadamard != 0 && apply_hadamard != 1)
    return fail(OFFQ_ERR_INVALID, "apply_hadamard must be 0 or 1");
  if (M == 0) return ok();  // empty: pointers may be NULL
  if (!x || !codes || !scale || !zero) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(x, 16) || !aligned(codes, 4) || !aligned(scale, 2) || !aligned(zero, 2) ||
      (y_debug && !aligned(y_debug, 16)))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer (x, y_debug: 16 B; codes: 4 B)");
  if (M * (K / g) >= kMaxGroups) return fail(OFFQ_ERR_UNSUPPORTED, "too many groups");
  if (offq_status_t s = check_device()) return s;
  return launched(offq::launch_rotate_quantize(x, M * (K / g), (int)(K / g), ldx, lg,
                                               apply_hadamard != 0, codes, K / 2, scale, zero,
                                               y_debug, K, (hipStream_t)stream),
                  "rotate_quantize");
}

offq_status_t offq_kv_quantize(const uint16_t* kv, int64_t rows, int32_t head_dim, int64_t row_stride,
                     int32_t apply_hadamard, uint8_t* codes, uint16_t* scale, int16_t* zero,
                     float* y_debug, void* stream) {
  if (rows < 0) return fail(OFFQ_ERR_INVALID, "rows must be >= 0");
  const int lg = ilog2_pow2(head_dim);
  if (lg < 0) return fail(OFFQ_ERR_INVALID, "head_dim = %d is not a power of two", head_dim);
  if (lg < 4 || lg > 13) return fail(OFFQ_ERR_UNSUPPORTED, "head_dim outside [16, 8192]");
  if (row_stride < head_dim || row_stride % 8)
    return fail(OFFQ_ERR_INVALID, "row_stride must be >= head_dim and a multiple of 8");
  if (apply_hadamard != 0 && apply_hadamard != 1)
    return fail(OFFQ_ERR_INVALID, "apply_hadamard must be 0 or 1");
  if (rows == 0) return ok();  // empty: pointers may be NULL
  if (!kv || !codes || !scale || !zero) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(kv, 16) || !aligned(codes, 4) || !aligned(scale, 2) || !aligned(zero, 2) ||
      (y_debug && !aligned(y_debug, 16)))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer (kv, y_debug: 16 B; codes: 4 B)");
  if (rows >= kMaxGroups) return fail(OFFQ_ERR_UNSUPPORTED, "too many rows");
  if (offq_status_t s = check_device()) return s;
  return launched(offq::launch_rotate_quantize(kv, rows, 1, row_stride, lg, apply_hadamard != 0,
                                               codes, head_dim / 2, scale, zero, y_debug,
                                               head_dim, (hipStream_t)stream),
                  "kv_quantize");
}

offq_status_t offq_w4a4_gemm(const uint8_t* a_codes, const uint16_t* a_scale, const int16_t* a_zero,
                   const uint8_t* w_codes, const uint16_t* w_scale, const int32_t* w_colsum,
                   int64_t M, int64_t N, int64_t K, int32_t g, uint16_t* y, int64_t ldy,
                   int32_t* acc_debug, void* stream) {
  if (M < 0 || N <= 0 || K <= 0) return fail(OFFQ_ERR_INVALID, "need M >= 0, N > 0, K > 0");
  const int lg = ilog2_pow2(g);
  if (lg < 0) return fail(OFFQ_ERR_INVALID, "g = %d is not a power of two", g);
  if (lg < 6 || lg > 13) return fail(OFFQ_ERR_UNSUPPORTED, "g = %d outside [64, 8192]", g);
  if (K % g) return fail(OFFQ_ERR_INVALID, "K = %lld is not a multiple of g = %d", (long long)K, g);
  if (ldy < N) return fail(OFFQ_ERR_INVALID, "ldy must be >= N");
  if (M > (1 << 30) || N > (1 << 30) || K > (1 << 30))
    return fail(OFFQ_ERR_UNSUPPORTED, "dimension too large");
  if (M == 0) return ok();  // empty: pointers may be NULL
  if (!a_codes || !a_scale || !a_zero || !w_codes || !w_scale || !w_colsum || !y)
    return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(a_codes, 16) || !aligned(w_codes, 16) || !aligned(a_scale, 2) ||
      !aligned(a_zero, 2) || !aligned(w_scale, 2) || !aligned(w_colsum, 4) || !aligned(y, 2) ||
      (acc_debug && !aligned(acc_debug, 4)))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer (codes: 16 B)");
  if (offq_status_t s = check_device()) return s;
  hipError_t e;
  if (M <= 16 && offq::gemv_mfma_supported(M, N, K, lg))
    e = offq::launch_w4a4_gemv_mfma(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N,
                                    K, lg, y, ldy, acc_debug, (hipStream_t)stream);
  else if (M <= 16)
    e = offq::launch_w4a4_gemv(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K, lg,
                               y, ldy, acc_debug, (hipStream_t)stream);
  else
    e = offq::launch_w4a4_gemm(a_codes, a_scale, a_zero, w_codes, w_scale, w_colsum, M, N, K, lg,
                               y, ldy, acc_debug, (hipStream_t)stream);
  return launched(e, M <= 16 ? "w4a4_gemv" : "w4a4_gemm");
}

int64_t offq_weight_codes_bytes(int64_t N, int64_t K) {
  if (N <= 0 || K <= 0 || N > (1 << 30) || K > (1 << 30)) return 0;
  return offq::wblk_bytes(N, K);
}

offq_status_t offq_pack_weights(const float* w, int64_t N, int64_t K, int32_t g, uint8_t* w_codes,
                      uint16_t* w_scale, int32_t* w_colsum, void* stream) {
  if (N <= 0 || K <= 0) return fail(OFFQ_ERR_INVALID, "need N > 0, K > 0");
  const int lg = ilog2_pow2(g);
  if (lg < 0) return fail(OFFQ_ERR_INVALID, "g = %d is not a power of two", g);
  if (lg < 6 || lg > 13) return fail(OFFQ_ERR_UNSUPPORTED, "g = %d outside [64, 8192]", g);
  if (K % g) return fail(OFFQ_ERR_INVALID, "K = %lld is not a multiple of g = %d", (long long)K, g);
  if (K / g > 512) return fail(OFFQ_ERR_UNSUPPORTED, "K / g must be <= 512");
  if (N >= kMaxGroups) return fail(OFFQ_ERR_UNSUPPORTED, "N too large");
  if (!w || !w_codes || !w_scale || !w_colsum) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(w, 16) || !aligned(w_codes, 4) || !aligned(w_scale, 2) || !aligned(w_colsum, 4))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer (w: 16 B; w_codes: 4 B)");
  if (offq_status_t s = check_device()) return s;
  return launched(offq::launch_pack_weights(w, N, K, lg, w_codes, w_scale, w_colsum,
                                            (hipStream_t)stream),
                  "pack_weights");
}


int64_t offq_kv_attention_workspace_bytes(int64_t B, int64_t H, int64_t seq_len) {
  if (B <= 0 || H <= 0 || seq_len <= 0 || B * H > (1 << 24) || seq_len > (int64_t(1) << 30))
    return 0;
  return offq::kv_attention_workspace_floats(B * H, seq_len) * (int64_t)sizeof(float);
}

namespace {
offq_status_t kv_attention_checked(const uint16_t* q, const uint8_t* k_codes, const uint16_t* k_scale,
                         const int16_t* k_zero, const uint8_t* v_codes, const uint16_t* v_scale,
                         const int16_t* v_zero, int64_t B, int64_t Hq, int64_t Hkv, int64_t s_cap,
                         int64_t seq_len, int32_t head_dim, float sm_scale, int32_t v_hadamard,
                         uint16_t* out, uint8_t* qcodes, uint16_t* qscale, int16_t* qzero,
                         void* workspace, int64_t workspace_bytes, void* stream) {
  if (B <= 0 || Hq <= 0 || Hkv <= 0) return fail(OFFQ_ERR_INVALID, "need B, Hq, Hkv > 0");
  if (Hq % Hkv) return fail(OFFQ_ERR_INVALID, "Hq = %lld is not a multiple of Hkv = %lld",
                            (long long)Hq, (long long)Hkv);
  if (head_dim != 128) return fail(OFFQ_ERR_UNSUPPORTED, "head_dim = %d (only 128)", head_dim);
  if (seq_len < 1 || seq_len > s_cap)
    return fail(OFFQ_ERR_INVALID, "need 1 <= seq_len <= s_cap");
  if (B * Hq > (1 << 24) || seq_len > (int64_t(1) << 30) ||
      s_cap > (int64_t(1) << 40) / (B * Hkv) || B * Hq * ((seq_len + 511) / 512) > (1 << 24))
    return fail(OFFQ_ERR_UNSUPPORTED, "sizes too large (B Hq ceil(seq_len / 512) <= 2^24)");
  if (v_hadamard != 0 && v_hadamard != 1) return fail(OFFQ_ERR_INVALID, "v_hadamard must be 0 or 1");
  if (!(sm_scale == sm_scale)) return fail(OFFQ_ERR_INVALID, "sm_scale is NaN");
  if (!q || !k_codes || !k_scale || !k_zero || !v_codes || !v_scale || !v_zero || !workspace ||
      (!out && !qcodes) || (qcodes && (!qscale || !qzero)))
    return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(q, 2) || !aligned(k_codes, 16) || !aligned(v_codes, 16) || !aligned(k_scale, 2) ||
      !aligned(k_zero, 2) || !aligned(v_scale, 2) || !aligned(v_zero, 2) || !aligned(out, 2) ||
      !aligned(qscale, 2) || !aligned(qzero, 2) || !aligned(workspace, 4))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer (codes: 16 B; workspace: 4 B)");
  const int64_t need = offq_kv_attention_workspace_bytes(B, Hq, seq_len);
  if (workspace_bytes < need)
    return fail(OFFQ_ERR_INVALID, "workspace of %lld bytes, need %lld", (long long)workspace_bytes,
                (long long)need);
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_kv_attention_decode(q, k_codes, k_scale, k_zero, v_codes, v_scale,
                                                   v_zero, B * Hq, Hq / Hkv, s_cap, seq_len,
                                                   sm_scale, v_hadamard != 0, out, qcodes,
                                                   qscale, qzero, static_cast<float*>(workspace),
                                                   (hipStream_t)stream),
                  "kv_attention_decode");
}
}  // namespace

offq_status_t offq_kv_attention_decode_gqa(const uint16_t* q, const uint8_t* k_codes,
                                 const uint16_t* k_scale, const int16_t* k_zero,
                                 const uint8_t* v_codes, const uint16_t* v_scale,
                                 const int16_t* v_zero, int64_t B, int64_t Hq, int64_t Hkv,
                                 int64_t s_cap, int64_t seq_len, int32_t head_dim, float sm_scale,
                                 int32_t v_hadamard, uint16_t* out, void* workspace,
                                 int64_t workspace_bytes, void* stream) {
  if (!out) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  return kv_attention_checked(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, B, Hq, Hkv,
                              s_cap, seq_len, head_dim, sm_scale, v_hadamard, out, nullptr, nullptr,
                              nullptr, workspace, workspace_bytes, stream);
}

offq_status_t offq_kv_attention_decode_quantize(const uint16_t* q, const uint8_t* k_codes,
                                      const uint16_t* k_scale, const int16_t* k_zero,
                                      const uint8_t* v_codes, const uint16_t* v_scale,
                                      const int16_t* v_zero, int64_t B, int64_t Hq, int64_t Hkv,
                                      int64_t s_cap, int64_t seq_len, int32_t head_dim,
                                      float sm_scale, int32_t v_hadamard, uint16_t* out,
                                      uint8_t* out_codes, uint16_t* out_scale, int16_t* out_zero,
                                      void* workspace, int64_t workspace_bytes, void* stream) {
  if (!out_codes) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  return kv_attention_checked(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, B, Hq, Hkv,
                              s_cap, seq_len, head_dim, sm_scale, v_hadamard, out, out_codes,
                              out_scale, out_zero, workspace, workspace_bytes, stream);
}

offq_status_t offq_kv_attention_decode(const uint16_t* q, const uint8_t* k_codes, const uint16_t* k_scale,
                             const int16_t* k_zero, const uint8_t* v_codes,
                             const uint16_t* v_scale, const int16_t* v_zero, int64_t B,
                             int64_t H, int64_t s_cap, int64_t seq_len, int32_t head_dim,
                             float sm_scale, int32_t v_hadamard, uint16_t* out, void* workspace,
                             int64_t workspace_bytes, void* stream) {
  return offq_kv_attention_decode_gqa(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, B, H,
                                      H, s_cap, seq_len, head_dim, sm_scale, v_hadamard, out,
                                      workspace, workspace_bytes, stream);
}

offq_status_t offq_kv_attention_decode_noalloc(const uint16_t* q, const uint8_t* k_codes,
                                               const uint16_t* k_scale, const int16_t* k_zero,
                                               const uint8_t* v_codes, const uint16_t* v_scale,
                                               const int16_t* v_zero, int64_t B, int64_t Hq,
                                               int64_t Hkv, int64_t s_cap, int64_t seq_len,
                                               int32_t head_dim, float sm_scale,
                                               int32_t v_hadamard, uint16_t* out, void* stream) {
  if (!out) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (B > 0 && Hq > 0 && seq_len > 0) {
    const int64_t need = offq_kv_attention_workspace_bytes(B, Hq, seq_len);
    if (need > offq::kKvScratchBytes)
      return fail(OFFQ_ERR_UNSUPPORTED,
                  "B Hq ceil(seq_len / 512) = %lld chunk records need %lld bytes; the static "
                  "scratch holds %lld",
                  (long long)(need / (130 * 4)), (long long)need,
                  (long long)offq::kKvScratchBytes);
  }
  // the other checks (sizes, pointers, device) are the plain call's, with the
  // scratch standing in for the workspace
  if (offq_status_t st = check_device()) return st;
  float* ws = nullptr;
  const hipError_t e = offq::kv_attention_scratch(&ws);
  if (e != hipSuccess)
    return fail(OFFQ_ERR_HIP, "static scratch address: %s", hipGetErrorString(e));
  return kv_attention_checked(q, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, B, Hq, Hkv,
                              s_cap, seq_len, head_dim, sm_scale, v_hadamard, out, nullptr,
                              nullptr, nullptr, ws, offq::kKvScratchBytes, stream);
}

offq_status_t offq_add_rmsnorm(const uint16_t* x, int64_t ldx, const uint16_t* res, int64_t ldr, int64_t M,
                     int64_t D, float eps, uint16_t* h_out, int64_t ldh, uint16_t* y_out,
                     int64_t ldy, void* stream) {
  if (M < 0) return fail(OFFQ_ERR_INVALID, "M < 0");
  if (D < 8 || D % 8) return fail(OFFQ_ERR_INVALID, "D = %lld must be a positive multiple of 8",
                                  (long long)D);
  if (D > (1 << 20) || M > (int64_t(1) << 31) - 1)
    return fail(OFFQ_ERR_UNSUPPORTED, "sizes too large");
  if (!(eps >= 0.0f) || eps > 1e30f) return fail(OFFQ_ERR_INVALID, "eps must be finite and >= 0");
  if (!x || (!h_out && !y_out)) return fail(OFFQ_ERR_INVALID, "need x and at least one output");
  if (ldx < D || ldx % 8 || (res && (ldr < D || ldr % 8)) || (h_out && (ldh < D || ldh % 8)) ||
      (y_out && (ldy < D || ldy % 8)))
    return fail(OFFQ_ERR_INVALID, "row strides must be >= D and multiples of 8");
  if (!aligned(x, 16) || (res && !aligned(res, 16)) || (h_out && !aligned(h_out, 16)) ||
      (y_out && !aligned(y_out, 16)))
    return fail(OFFQ_ERR_INVALID, "pointers must be 16-byte aligned");
  if (M == 0) return ok();
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_add_rmsnorm(x, ldx, res, ldr, M, D, eps, h_out, ldh, y_out, ldy,
                                           (hipStream_t)stream),
                  "add_rmsnorm");
}

offq_status_t offq_swiglu(const uint16_t* gu, int64_t ldg, int64_t M, int64_t F, uint16_t* out, int64_t ldo,
                void* stream) {
  if (M < 0) return fail(OFFQ_ERR_INVALID, "M < 0");
  if (F < 8 || F % 8) return fail(OFFQ_ERR_INVALID, "F must be a positive multiple of 8");
  if (ldg < 2 * F || ldg % 8 || ldo < F || ldo % 8)
    return fail(OFFQ_ERR_INVALID, "need ldg >= 2F, ldo >= F, both multiples of 8");
  if (F > (1 << 24) || M * (F / 8) > (int64_t(1) << 38))
    return fail(OFFQ_ERR_UNSUPPORTED, "sizes too large");
  if (!gu || !out) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(gu, 16) || !aligned(out, 16))
    return fail(OFFQ_ERR_INVALID, "pointers must be 16-byte aligned");
  if (M == 0) return ok();
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_swiglu(gu, ldg, M, F, out, ldo, (hipStream_t)stream), "swiglu");
}

namespace {
// Shared by the decode (T = 1) and prefill forms: M = B T rows, row m of
// sequence m / T.
offq_status_t rope_kv(const uint16_t* qkv, int64_t ldq, int64_t B, int64_t T, int64_t Hq,
                      int64_t Hkv, int32_t head_dim, const int32_t* positions, double rope_base,
                      int32_t k_hadamard, int32_t v_hadamard, uint16_t* q_out, uint8_t* k_codes,
                      uint16_t* k_scale, int16_t* k_zero, uint8_t* v_codes, uint16_t* v_scale,
                      int16_t* v_zero, int64_t s_cap, float* k_y_debug, float* v_y_debug,
                      void* stream, const char* what) {
  if (B < 0 || T < 1 || Hq <= 0 || Hkv <= 0)
    return fail(OFFQ_ERR_INVALID, "need rows >= 0, T >= 1, Hq, Hkv > 0");
  if (head_dim != 128) return fail(OFFQ_ERR_UNSUPPORTED, "head_dim = %d (only 128)", head_dim);
  if (ldq < (Hq + 2 * Hkv) * 128 || ldq % 8)
    return fail(OFFQ_ERR_INVALID, "ldq must be >= (Hq + 2 Hkv) * 128 and a multiple of 8");
  if (s_cap < 1) return fail(OFFQ_ERR_INVALID, "s_cap must be >= 1");
  if (!(rope_base > 1.0) || rope_base > 1e30) return fail(OFFQ_ERR_INVALID, "rope_base must be > 1");
  if ((k_hadamard != 0 && k_hadamard != 1) || (v_hadamard != 0 && v_hadamard != 1))
    return fail(OFFQ_ERR_INVALID, "k_hadamard / v_hadamard must be 0 or 1");
  if (T > (int64_t(1) << 31) || B > (int64_t(1) << 32) / T)
    return fail(OFFQ_ERR_UNSUPPORTED, "sizes too large");
  const int64_t M = B * T;
  if (M * (Hq + 2 * Hkv) > (int64_t(1) << 32) || Hq + 2 * Hkv > (1 << 20) ||
      s_cap > (int64_t(1) << 40) / (B > 0 ? B * Hkv : 1))
    return fail(OFFQ_ERR_UNSUPPORTED, "sizes too large");
  if (!qkv || !positions || !q_out || !k_codes || !k_scale || !k_zero || !v_codes || !v_scale ||
      !v_zero)
    return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(qkv, 16) || !aligned(positions, 4) || !aligned(q_out, 16) ||
      !aligned(k_codes, 4) || !aligned(v_codes, 4) || !aligned(k_scale, 2) ||
      !aligned(k_zero, 2) || !aligned(v_scale, 2) || !aligned(v_zero, 2) ||
      (k_y_debug && !aligned(k_y_debug, 16)) || (v_y_debug && !aligned(v_y_debug, 16)))
    return fail(OFFQ_ERR_INVALID,
                "misaligned pointer (qkv, q_out, debug: 16 B; codes, positions: 4 B)");
  if (M == 0) return ok();
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_rope_kv_append(qkv, ldq, M, T, Hq, Hkv, positions, rope_base,
                                              k_hadamard != 0, v_hadamard != 0, q_out, k_codes,
                                              k_scale, k_zero, v_codes, v_scale, v_zero, s_cap,
                                              k_y_debug, v_y_debug, (hipStream_t)stream),
                  what);
}
}  // namespace

offq_status_t offq_rope_kv_append(const uint16_t* qkv, int64_t ldq, int64_t M, int64_t Hq, int64_t Hkv,
                        int32_t head_dim, const int32_t* positions, double rope_base,
                        int32_t k_hadamard, int32_t v_hadamard, uint16_t* q_out,
                        uint8_t* k_codes, uint16_t* k_scale, int16_t* k_zero, uint8_t* v_codes,
                        uint16_t* v_scale, int16_t* v_zero, int64_t s_cap, float* k_y_debug,
                        float* v_y_debug, void* stream) {
  return rope_kv(qkv, ldq, M, 1, Hq, Hkv, head_dim, positions, rope_base, k_hadamard, v_hadamard,
                 q_out, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, s_cap, k_y_debug,
                 v_y_debug, stream, "rope_kv_append");
}

offq_status_t offq_rope_kv_prefill(const uint16_t* qkv, int64_t ldq, int64_t B, int64_t T,
                        int64_t Hq, int64_t Hkv, int32_t head_dim, const int32_t* positions,
                        double rope_base, int32_t k_hadamard, int32_t v_hadamard,
                        uint16_t* q_out, uint8_t* k_codes, uint16_t* k_scale, int16_t* k_zero,
                        uint8_t* v_codes, uint16_t* v_scale, int16_t* v_zero, int64_t s_cap,
                        float* k_y_debug, float* v_y_debug, void* stream) {
  return rope_kv(qkv, ldq, B, T, Hq, Hkv, head_dim, positions, rope_base, k_hadamard, v_hadamard,
                 q_out, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, s_cap, k_y_debug,
                 v_y_debug, stream, "rope_kv_prefill");
}

offq_status_t offq_kv_attention_prefill(const uint16_t* q, int64_t B, int64_t T, int64_t Hq,
                        int64_t Hkv, int32_t head_dim, int64_t past, const uint8_t* k_codes,
                        const uint16_t* k_scale, const int16_t* k_zero, const uint8_t* v_codes,
                        const uint16_t* v_scale, const int16_t* v_zero, int64_t s_cap,
                        float sm_scale, int32_t v_hadamard, uint16_t* out, void* stream) {
  if (B < 0 || T < 0 || Hq <= 0 || Hkv <= 0 || past < 0)
    return fail(OFFQ_ERR_INVALID, "need B, T, past >= 0 and Hq, Hkv > 0");
  if (head_dim != 128) return fail(OFFQ_ERR_UNSUPPORTED, "head_dim = %d (only 128)", head_dim);
  if (Hq % Hkv) return fail(OFFQ_ERR_INVALID, "Hq = %lld is not a multiple of Hkv = %lld",
                            (long long)Hq, (long long)Hkv);
  const int64_t G = Hq / Hkv;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(OFFQ_ERR_UNSUPPORTED, "Hq / Hkv = %lld (supported: 1, 2, 4, 8)", (long long)G);
  if (past + T > s_cap) return fail(OFFQ_ERR_INVALID, "past + T exceeds s_cap");
  if (v_hadamard != 0 && v_hadamard != 1) return fail(OFFQ_ERR_INVALID, "v_hadamard must be 0 or 1");
  if (!(sm_scale > 0.0f) || sm_scale > 1e30f) return fail(OFFQ_ERR_INVALID, "sm_scale must be > 0");
  if (past + T > (int64_t(1) << 30) || Hq > (1 << 16) ||
      B * T > (int64_t(1) << 31) / Hq || B * Hkv * ((T + 31) / 32) > (int64_t(1) << 31) ||
      s_cap > (int64_t(1) << 40) / (B > 0 ? B * Hkv : 1))
    return fail(OFFQ_ERR_UNSUPPORTED, "sizes too large");
  if (B == 0 || T == 0) return ok();
  if (!q || !k_codes || !k_scale || !k_zero || !v_codes || !v_scale || !v_zero || !out)
    return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(q, 16) || !aligned(out, 16) || !aligned(k_codes, 16) || !aligned(v_codes, 16) ||
      !aligned(k_scale, 2) || !aligned(k_zero, 2) || !aligned(v_scale, 2) || !aligned(v_zero, 2))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer (q, out, codes: 16 B; scales: 2 B)");
  const int64_t n = B * T * Hq * 128 * 2;
  const uintptr_t qa = (uintptr_t)q, oa = (uintptr_t)out;
  if (n > 0 && qa < oa + (uintptr_t)n && oa < qa + (uintptr_t)n)
    return fail(OFFQ_ERR_INVALID, "out overlaps q");
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_kv_attention_prefill(q, B, T, Hq, Hkv, past, k_codes, k_scale,
                                                    k_zero, v_codes, v_scale, v_zero, s_cap,
                                                    sm_scale, v_hadamard != 0, out,
                                                    (hipStream_t)stream),
                  "kv_attention_prefill");
}

int64_t offq_top1_workspace_bytes(int64_t n_seq, int64_t seq_len) {
  if (n_seq <= 0 || seq_len <= 0 || n_seq > (int64_t(1) << 31) / seq_len) return 0;
  return n_seq * seq_len * (int64_t)sizeof(float);
}

offq_status_t offq_top1_select(const uint16_t* x, int64_t n_seq, int64_t seq_len, int64_t D, int64_t ld_tok,
                     int64_t ld_seq, int32_t* idx, float* X, int64_t ldX, void* workspace,
                     int64_t workspace_bytes, void* stream) {
  if (n_seq <= 0 || seq_len <= 0) return fail(OFFQ_ERR_INVALID, "need n_seq, seq_len > 0");
  if (D < 8 || D % 8 || ld_tok < D || ld_tok % 8 || ld_seq % 8 || ldX < D)
    return fail(OFFQ_ERR_INVALID, "D, ld_tok, ld_seq must be multiples of 8 with ld_tok >= D, ldX >= D");
  if (ld_seq < (seq_len - 1) * ld_tok + D && n_seq > 1)
    return fail(OFFQ_ERR_INVALID, "sequences overlap (ld_seq too small)");
  if (D > (1 << 20) || n_seq > (1 << 24) || n_seq * seq_len > (int64_t(1) << 31))
    return fail(OFFQ_ERR_UNSUPPORTED, "sizes too large");
  if (!x || !idx || !X || !workspace) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(x, 16) || !aligned(idx, 4) || !aligned(X, 4) || !aligned(workspace, 4))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer (x: 16 B)");
  if (workspace_bytes < offq_top1_workspace_bytes(n_seq, seq_len))
    return fail(OFFQ_ERR_INVALID, "workspace too small");
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_top1_select(x, n_seq, seq_len, D, ld_tok, ld_seq, idx, X, ldX,
                                           static_cast<float*>(workspace), (hipStream_t)stream),
                  "top1_select");
}

offq_status_t offq_channel_absmax(const uint16_t* x, int64_t rows, int64_t D, int64_t ldx, double* out,
                        void* stream) {
  if (rows <= 0 || D <= 0 || ldx < D) return fail(OFFQ_ERR_INVALID, "need rows, D > 0, ldx >= D");
  if (D > (1 << 24)) return fail(OFFQ_ERR_UNSUPPORTED, "D too large");
  if (!x || !out) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(x, 2) || !aligned(out, 8)) return fail(OFFQ_ERR_INVALID, "misaligned pointer");
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_channel_absmax(x, rows, D, ldx, out, (hipStream_t)stream),
                  "channel_absmax");
}

offq_status_t offq_gram(const float* X, int64_t N, int64_t D, int64_t ldX, double* C, int64_t ldC,
              void* stream) {
  if (N <= 0 || D <= 0 || ldX < D || ldC < D)
    return fail(OFFQ_ERR_INVALID, "need N, D > 0, ldX >= D, ldC >= D");
  if (D > 65536 || N > (int64_t(1) << 30)) return fail(OFFQ_ERR_UNSUPPORTED, "sizes too large");
  if (!X || !C) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(X, 4) || !aligned(C, 8)) return fail(OFFQ_ERR_INVALID, "misaligned pointer");
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_gram(X, N, D, ldX, C, ldC, (hipStream_t)stream), "gram");
}

int64_t offq_eigh_workspace_bytes(int64_t D) {
  if (D < 2 || D > 8192 || D % 2) return 0;
  return offq::eigh_workspace_doubles(D) * (int64_t)sizeof(double);
}

offq_status_t offq_eigh(const double* C, int64_t D, int64_t ldC, double* evals, double* U, int64_t ldU,
              void* workspace, int64_t workspace_bytes, int32_t max_sweeps, double tol,
              int32_t* sweeps, double* rel_off, void* stream) {
  if (D < 2 || D % 2) return fail(OFFQ_ERR_INVALID, "D must be even and >= 2");
  if (D > 8192) return fail(OFFQ_ERR_UNSUPPORTED, "D = %lld > 8192", (long long)D);
  if (ldC < D || ldU < D) return fail(OFFQ_ERR_INVALID, "row strides must be >= D");
  if (max_sweeps < 0 || !(tol >= 0.0)) return fail(OFFQ_ERR_INVALID, "need max_sweeps >= 0, tol >= 0");
  if (!C || !evals || !U || !workspace) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(C, 8) || !aligned(evals, 8) || !aligned(U, 8) || !aligned(workspace, 16))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer (workspace: 16 B)");
  if (workspace_bytes < offq_eigh_workspace_bytes(D))
    return fail(OFFQ_ERR_INVALID, "workspace of %lld bytes, need %lld", (long long)workspace_bytes,
                (long long)offq_eigh_workspace_bytes(D));
  if (offq_status_t st = check_device()) return st;
  int sw = 0;
  double ro = 0.0;
  const hipError_t e = offq::launch_eigh(C, ldC, D, evals, U, ldU, static_cast<double*>(workspace),
                                         max_sweeps, tol, &sw, &ro, (hipStream_t)stream);
  if (sweeps) *sweeps = sw;
  if (rel_off) *rel_off = ro;
  return launched(e, "eigh");
}

offq_status_t offq_group_permutation(const double* key, int64_t D, int32_t g, int32_t* perm,
                           void* workspace, int64_t workspace_bytes, void* stream) {
  if (D <= 0 || g <= 0 || D % g) return fail(OFFQ_ERR_INVALID, "need D > 0 a multiple of g > 0");
  if (D > (1 << 20)) return fail(OFFQ_ERR_UNSUPPORTED, "D too large");
  if (!key || !perm || !workspace) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(key, 8) || !aligned(perm, 4) || !aligned(workspace, 4))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer");
  if (workspace_bytes < D * 4) return fail(OFFQ_ERR_INVALID, "workspace too small (D int32)");
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_group_permutation(key, D, g, perm, static_cast<int32_t*>(workspace),
                                                 (hipStream_t)stream),
                  "group_permutation");
}

offq_status_t offq_build_rotation(const double* U, int64_t ldU, int64_t D, const int32_t* perm, int32_t g,
                        int32_t apply_hadamard, float* R, int64_t ldR, void* stream) {
  if (D <= 0 || D > 8192) return fail(OFFQ_ERR_UNSUPPORTED, "need 0 < D <= 8192");
  if (apply_hadamard != 0 && apply_hadamard != 1)
    return fail(OFFQ_ERR_INVALID, "apply_hadamard must be 0 or 1");
  int lg = 0;
  if (apply_hadamard) {
    lg = ilog2_pow2(g);
    if (lg < 0 || D % g) return fail(OFFQ_ERR_INVALID, "g must be a power of two dividing D");
  }
  if ((U && ldU < D) || ldR < D) return fail(OFFQ_ERR_INVALID, "row strides must be >= D");
  if (!R) return fail(OFFQ_ERR_INVALID, "null output");
  if ((U && !aligned(U, 8)) || (perm && !aligned(perm, 4)) || !aligned(R, 4))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer");
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_build_rotation(U, ldU, D, perm, lg, R, ldR, (hipStream_t)stream),
                  "build_rotation");
}

offq_status_t offq_fuse_weights(const float* W, int64_t ldW, int64_t N, int64_t K, const float* R,
                      int64_t ldR, float* W_out, int64_t ldo, void* stream) {
  if (N <= 0 || K <= 0 || ldW < K || ldR < K || ldo < K)
    return fail(OFFQ_ERR_INVALID, "need N, K > 0 and row strides >= K");
  if (N > (1 << 24) || K > 65536) return fail(OFFQ_ERR_UNSUPPORTED, "sizes too large");
  if (!W || !R || !W_out) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(W, 4) || !aligned(R, 4) || !aligned(W_out, 4))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer");
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_fuse_weights(W, ldW, N, K, R, ldR, W_out, ldo, (hipStream_t)stream),
                  "fuse_weights");
}

offq_status_t offq_permute_rows(const float* W, int64_t ldW, int64_t N, int64_t K, const int32_t* perm,
                      float* W_out, int64_t ldo, void* stream) {
  if (N <= 0 || K <= 0 || ldW < K || ldo < K)
    return fail(OFFQ_ERR_INVALID, "need N, K > 0 and row strides >= K");
  if (N > (int64_t(1) << 31) - 1) return fail(OFFQ_ERR_UNSUPPORTED, "N too large");
  if (!W || !perm || !W_out) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(W, 4) || !aligned(perm, 4) || !aligned(W_out, 4))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer");
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_permute_rows(W, ldW, N, K, perm, W_out, ldo, (hipStream_t)stream),
                  "permute_rows");
}

offq_status_t offq_add_rmsnorm_quantize(const uint16_t* x, int64_t ldx, const uint16_t* res, int64_t ldr,
                              int64_t M, int64_t D, float eps, int32_t g, uint16_t* h_out,
                              int64_t ldh, uint8_t* codes, uint16_t* scale, int16_t* zero,
                              uint16_t* y_debug, int64_t ldy, void* stream) {
  if (M < 0) return fail(OFFQ_ERR_INVALID, "M < 0");
  const int64_t E = D / 256;
  if (D % 256 || (E != 8 && E != 16 && E != 32 && E != 64))
    return fail(OFFQ_ERR_UNSUPPORTED, "D = %lld (D / 256 must be 8, 16, 32 or 64)", (long long)D);
  const int lg = ilog2_pow2(g);
  if (lg < 0 || g < E || g > D / 4 || D % g)
    return fail(OFFQ_ERR_UNSUPPORTED, "g = %d (a power of two with D/256 <= g <= D/4)", g);
  if (!(eps >= 0.0f) || eps > 1e30f) return fail(OFFQ_ERR_INVALID, "eps must be finite and >= 0");
  if (!x || !codes || !scale || !zero) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (ldx < D || ldx % 8 || (res && (ldr < D || ldr % 8)) || (h_out && (ldh < D || ldh % 8)) ||
      (y_debug && (ldy < D || ldy % 8)))
    return fail(OFFQ_ERR_INVALID, "row strides must be >= D and multiples of 8");
  if (!aligned(x, 16) || (res && !aligned(res, 16)) || (h_out && !aligned(h_out, 16)) ||
      (y_debug && !aligned(y_debug, 16)) || !aligned(codes, 16) || !aligned(scale, 2) ||
      !aligned(zero, 2))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer (rows and codes: 16 B)");
  if (M > (int64_t(1) << 31) - 1) return fail(OFFQ_ERR_UNSUPPORTED, "M too large");
  if (M == 0) return ok();
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_add_rmsnorm_quant(x, ldx, res, ldr, M, D, eps, lg, h_out, ldh,
                                                 codes, scale, zero, y_debug, ldy,
                                                 (hipStream_t)stream),
                  "add_rmsnorm_quantize");
}

offq_status_t offq_swiglu_rotate_quantize(const uint16_t* gu, int64_t ldg, int64_t M, int64_t F,
                                uint8_t* codes, uint16_t* scale, int16_t* zero, float* y_debug,
                                void* stream) {
  if (M < 0) return fail(OFFQ_ERR_INVALID, "M < 0");
  if (F < 128 || F % 128) return fail(OFFQ_ERR_INVALID, "F must be a positive multiple of 128");
  if (ldg < 2 * F || ldg % 8) return fail(OFFQ_ERR_INVALID, "need ldg >= 2F, a multiple of 8");
  if (F > (1 << 24) || M * (F / 128) > (int64_t(1) << 34))
    return fail(OFFQ_ERR_UNSUPPORTED, "sizes too large");
  if (!gu || !codes || !scale || !zero) return fail(OFFQ_ERR_INVALID, "null pointer argument");
  if (!aligned(gu, 16) || !aligned(codes, 4) || !aligned(scale, 2) || !aligned(zero, 2) ||
      (y_debug && !aligned(y_debug, 16)))
    return fail(OFFQ_ERR_INVALID, "misaligned pointer (gu: 16 B)");
  if (M == 0) return ok();
  if (offq_status_t st = check_device()) return st;
  return launched(offq::launch_swiglu_rq(gu, ldg, M, F, codes, scale, zero, y_debug,
                                         (hipStream_t)stream),
                  "swiglu_rotate_quantize");
}

}  // extern "C"
