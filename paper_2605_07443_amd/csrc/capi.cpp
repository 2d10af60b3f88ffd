// Host-side pieces of the C ABI: error reporting, status strings, shape
// checks and the RoPE table builder.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>

#include "rc_common.h"

namespace rc {

static thread_local char g_last_error[512] = "";

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

void clear_error() { g_last_error[0] = '\0'; }

int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(RC_ERR_HIP, "%s: launch failed: %s", what, hipGetErrorString(e));
  return RC_OK;
}

int check_shape(const rc_shape* s, bool need_hq) {
  if (!s) return fail(RC_ERR_INVALID_ARG, "shape is NULL");
  if (s->B < 1 || s->N < 1 || s->Hkv < 1 || s->D < 1)
    return fail(RC_ERR_INVALID_ARG, "shape: B=%d N=%d Hkv=%d D=%d must be >= 1", s->B, s->N,
                s->Hkv, s->D);
  if (need_hq) {
    if (s->Hq < 1) return fail(RC_ERR_INVALID_ARG, "shape: Hq=%d must be >= 1", s->Hq);
    if (s->Hq % s->Hkv != 0)
      return fail(RC_ERR_INVALID_ARG, "shape: Hq=%d is not a multiple of Hkv=%d", s->Hq, s->Hkv);
  }
  if (s->dtype != RC_F32 && s->dtype != RC_BF16)
    return fail(RC_ERR_UNSUPPORTED, "dtype %d is not RC_F32 or RC_BF16", s->dtype);
  if (s->D != 64 && s->D != 128) return fail(RC_ERR_UNSUPPORTED, "head dim D=%d (64 or 128)", s->D);
  // element counts of the largest tensors must fit the kernels' 64-bit math,
  // and per-request row counts their 32-bit math
  if ((int64_t)s->N * s->Hkv * s->D >= (int64_t)1 << 31 ||
      (need_hq && (int64_t)s->N * s->Hq * s->D >= (int64_t)1 << 31))
    return fail(RC_ERR_UNSUPPORTED, "one request's tensor exceeds 2^31 elements");
  return RC_OK;
}

}  // namespace rc

extern "C" {

const char* rc_status_string(int status) {
  switch (status) {
    case RC_OK: return "RC_OK";
    case RC_ERR_INVALID_ARG: return "RC_ERR_INVALID_ARG";
    case RC_ERR_UNSUPPORTED: return "RC_ERR_UNSUPPORTED";
    case RC_ERR_HIP: return "RC_ERR_HIP";
    default: return "unknown rc_status";
  }
}

const char* rc_last_error(void) { return rc::g_last_error; }

// Angle pos * base^(-2j/D) in fp64; cos and sin rounded once to fp32.
int rc_rope_table(int32_t max_pos, int32_t D, double base, float* cos_out, float* sin_out) {
  rc::clear_error();
  if (!cos_out || !sin_out) return rc::fail(RC_ERR_INVALID_ARG, "rope table outputs are NULL");
  if (max_pos < 1 || D < 2 || (D & 1)) return rc::fail(RC_ERR_INVALID_ARG, "max_pos=%d D=%d", max_pos, D);
  if (!(base > 0.0) || !std::isfinite(base)) return rc::fail(RC_ERR_INVALID_ARG, "base must be > 0");
  const int half = D / 2;
  for (int32_t p = 0; p < max_pos; ++p) {
    for (int j = 0; j < half; ++j) {
      const double freq = std::pow(base, -(2.0 * j) / D);
      const double angle = static_cast<double>(p) * freq;
      cos_out[static_cast<size_t>(p) * half + j] = static_cast<float>(std::cos(angle));
      sin_out[static_cast<size_t>(p) * half + j] = static_cast<float>(std::sin(angle));
    }
  }
  return RC_OK;
}

}  // extern "C"
