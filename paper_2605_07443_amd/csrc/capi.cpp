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

// The local sliding window (Sec. III-C.2b): the last W positions of every
// request are recomputed like instruction tokens, so they become fresh
// segments. Segments before N - W are kept, the one crossing N - W is cut
// there, and the window is appended as fresh pieces -- as many as it takes
// for every request to end with the same segment count (tables are [B, S]).
int rc_segments_with_window(const rc_segment* segs_in, int32_t B, int32_t S, int32_t N,
                            int32_t W, rc_segment* segs_out, int32_t S_cap, int32_t* S_out) {
  rc::clear_error();
  if (!segs_in || !segs_out || !S_out) return rc::fail(RC_ERR_INVALID_ARG, "NULL table or S_out");
  if (B < 1 || S < 1 || N < 1) return rc::fail(RC_ERR_INVALID_ARG, "B=%d S=%d N=%d", B, S, N);
  if (W < 0 || W > N) return rc::fail(RC_ERR_INVALID_ARG, "window W=%d not in [0, N=%d]", W, N);
  const int32_t cut = N - W;
  // segments each request keeps before the window (cut ones count once)
  int32_t keep_max = 0;
  for (int32_t b = 0; b < B; ++b) {
    int32_t keep = 0, pos = 0;
    for (int32_t s = 0; s < S; ++s) {
      const rc_segment& g = segs_in[static_cast<size_t>(b) * S + s];
      if (g.dst_start != pos || g.len < 1)
        return rc::fail(RC_ERR_INVALID_ARG, "request %d: segments must tile [0, N) in order", b);
      if (g.dst_start < cut) ++keep;
      pos += g.len;
    }
    if (pos != N) return rc::fail(RC_ERR_INVALID_ARG, "request %d: segments cover %d of N=%d", b, pos, N);
    keep_max = keep > keep_max ? keep : keep_max;
  }
  const int32_t S_new = W > 0 ? keep_max + 1 : keep_max;
  if (S_new > S_cap) return rc::fail(RC_ERR_INVALID_ARG, "S_cap=%d < %d segments needed", S_cap, S_new);
  for (int32_t b = 0; b < B; ++b) {
    rc_segment* out = segs_out + static_cast<size_t>(b) * S_new;
    int32_t n = 0;
    for (int32_t s = 0; s < S; ++s) {
      rc_segment g = segs_in[static_cast<size_t>(b) * S + s];
      if (g.dst_start >= cut) break;
      if (g.dst_start + g.len > cut) g.len = cut - g.dst_start;
      out[n++] = g;
    }
    const int32_t pieces = S_new - n;  // >= 1 when W > 0
    if (pieces > W) return rc::fail(RC_ERR_INVALID_ARG, "window W=%d too short for %d pieces", W, pieces);
    int32_t pos = cut;
    for (int32_t i = 0; i < pieces; ++i) {
      const int32_t len = (i + 1 < pieces) ? 1 : N - pos;  // single tokens, then the rest
      out[n++] = rc_segment{pos, len, -1, 0};
      pos += len;
    }
  }
  *S_out = S_new;
  return RC_OK;
}

}  // extern "C"
