// host.hpp -- host-side helpers shared by the translation units of libllmv:
// error reporting, workspace checks and the shape constants of Sec. 2.1.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <mutex>

#include "llmv.h"

namespace llmv {
namespace host {

// Message of the calling thread's last failure (llmv_last_error).
inline thread_local char g_err[512] = "";

inline int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

inline int hip_fail(hipError_t e, const char* what) {
  return fail(LLMV_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                       \
  do {                                            \
    hipError_t e_ = (expr);                       \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

constexpr size_t kAlign = 256;

inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Compute units of the current device (cached per device).
inline int device_cus(int* out) {
  static std::mutex m;
  static int cache[64] = {0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(LLMV_EDEVICE, "device index %d out of range", dev);
  std::lock_guard<std::mutex> g(m);
  if (!cache[dev]) {
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    cache[dev] = cus > 0 ? cus : 1;
  }
  *out = cache[dev];
  return LLMV_OK;
}

// Shape constants S0..S3 of Sec. 2.1 (documented with llmv_shape_constants).
inline int shape_constants(const llmv_shape* sh, double S[4]) {
  if (!sh) {
    S[0] = S[1] = S[2] = S[3] = 1.0;
    return LLMV_OK;
  }
  const int32_t f[9] = {sh->n_layers, sh->hidden, sh->n_q_heads, sh->n_kv_heads, sh->head_dim,
                        sh->ffn, sh->vocab, sh->weight_bytes, sh->kv_bytes};
  for (int i = 0; i < 9; ++i)
    if (f[i] <= 0) return fail(LLMV_EINVAL, "shape field %d is %d; every field must be > 0", i, f[i]);
  // All products in int64: at most a few 2^31-bounded fields each; the
  // results are checked against 2^53 so they convert to fp64 exactly.
  const long double Ld = sh->n_layers, hd = sh->hidden, hq = sh->n_q_heads, hkv = sh->n_kv_heads,
                    dd = sh->head_dim, ff = sh->ffn, vv = sh->vocab, wb = sh->weight_bytes,
                    kb = sh->kv_bytes;
  const long double layer = hd * dd * (2 * hq + 2 * hkv) + 3 * hd * ff;
  const long double c0 = wb * (Ld * layer + vv * hd), c1 = 2 * Ld * layer,
                    c2 = 2 * Ld * hkv * dd * kb, c3 = 2 * Ld * hq * dd;
  const long double lim = 9007199254740992.0L;  // 2^53
  if (c0 >= lim || c1 >= lim || c2 >= lim || c3 >= lim)
    return fail(LLMV_EINVAL, "shape constants exceed 2^53");
  const int64_t L = sh->n_layers, h = sh->hidden, q = sh->n_q_heads, kv = sh->n_kv_heads,
                d = sh->head_dim;
  const int64_t p_layer = h * d * (2 * q + 2 * kv) + 3 * h * (int64_t)sh->ffn;
  S[0] = (double)((int64_t)sh->weight_bytes * (L * p_layer + (int64_t)sh->vocab * h));
  S[1] = (double)(2 * L * p_layer);
  S[2] = (double)(2 * L * kv * d * (int64_t)sh->kv_bytes);
  S[3] = (double)(2 * L * q * d);
  return LLMV_OK;
}

// Constants of the extended model's two extra features: S[0..3] as
// shape_constants, S[4] = 4*L*Hq*head_dim (FLOPs per processed token and
// cached key), S[5] = 2*vocab*hidden (output-projection FLOPs per request);
// all ones for the unit shape.
inline int shape_constants_ext(const llmv_shape* sh, double S[6]) {
  int rc = shape_constants(sh, S);
  if (rc) return rc;
  if (!sh) {
    S[4] = S[5] = 1.0;
    return LLMV_OK;
  }
  const int64_t s5 = 4 * (int64_t)sh->n_layers * sh->n_q_heads * sh->head_dim;
  const int64_t s6 = 2 * (int64_t)sh->vocab * sh->hidden;
  const int64_t lim = (int64_t)1 << 53;
  if (s5 >= lim || s6 >= lim) return fail(LLMV_EINVAL, "shape constants exceed 2^53");
  S[4] = (double)s5;
  S[5] = (double)s6;
  return LLMV_OK;
}

inline int check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return LLMV_OK;
  if (!ws) return fail(LLMV_EWORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (((uintptr_t)ws & (kAlign - 1)) != 0) return fail(LLMV_EWORKSPACE, "workspace not 256-byte aligned");
  if (ws_bytes < need)
    return fail(LLMV_EWORKSPACE, "workspace of %zu bytes, %zu needed", ws_bytes, need);
  return LLMV_OK;
}

}  // namespace host
}  // namespace llmv
