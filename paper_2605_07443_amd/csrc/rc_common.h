// Internal helpers shared by the HIP sources of librcllm (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rcllm.h"

namespace rc {

// ---------------------------------------------------------------- host side

// Record a failure message for rc_last_error() and return `status`.
int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
// Check hipGetLastError() after a launch; RC_OK or RC_ERR_HIP.
int check_launch(const char* what);
// Clear the thread's last error (called on entry of every API function).
void clear_error();

// Shape checks common to every call. `need_hq` also checks Hq/Hkv.
int check_shape(const rc_shape* s, bool need_hq);

inline int elem_size(int dtype) { return dtype == RC_F32 ? 4 : 2; }

constexpr int kMaxSegments = 1024;
constexpr int kMaxPools = 8;
constexpr int kMaxSelectN = 16384;

// Pools passed to kernels by value.
struct PoolArgs {
  const char* k[kMaxPools];
  const char* v[kMaxPools];
  int32_t num_blocks[kMaxPools];
  int32_t block_len[kMaxPools];
  int32_t n;
};

// -------------------------------------------------------------- device side

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// fp32 -> bf16 bits, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x0040u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
  return x;
}

__device__ __forceinline__ int wave_max_i(int x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x = max(x, __shfl_xor(x, off, 64));
  return x;
}

__device__ __forceinline__ int wave_min_i(int x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x = min(x, __shfl_xor(x, off, 64));
  return x;
}

using u32x4_t = uint32_t __attribute__((ext_vector_type(4)));

// sum over the elements of two 16-byte units of |a - b| (fp32 or bf16 storage)
template <int ES>
__device__ __forceinline__ float absdiff_sum(const u32x4_t& a, const u32x4_t& b) {
  float acc = 0.f;
  if constexpr (ES == 4) {
#pragma unroll
    for (int e = 0; e < 4; ++e) acc += fabsf(__uint_as_float(a[e]) - __uint_as_float(b[e]));
  } else {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      acc += fabsf(bf16_to_f32(static_cast<uint16_t>(a[w])) - bf16_to_f32(static_cast<uint16_t>(b[w])));
      acc += fabsf(bf16_to_f32(static_cast<uint16_t>(a[w] >> 16)) -
                   bf16_to_f32(static_cast<uint16_t>(b[w] >> 16)));
    }
  }
  return acc;
}

// Rotate E = 16/ES elements of the first half (a) and second half (b) of a
// head by the angle whose cos/sin are c[0..E), s[0..E).
//   a' = a*c - b*s,  b' = a*s + b*c   (fp32, no contraction), then RNE.
template <int ES>
__device__ __forceinline__ void rotate_unit(u32x4_t& a, u32x4_t& b, const float* c, const float* s) {
#pragma clang fp contract(off)
  if constexpr (ES == 4) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float x = __uint_as_float(a[e]);
      const float y = __uint_as_float(b[e]);
      const float xc = x * c[e], ys = y * s[e], xs = x * s[e], yc = y * c[e];
      a[e] = __float_as_uint(xc - ys);
      b[e] = __float_as_uint(xs + yc);
    }
  } else {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      uint32_t na = 0, nb = 0;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int e = 2 * w + h;
        const float x = bf16_to_f32(static_cast<uint16_t>(a[w] >> (16 * h)));
        const float y = bf16_to_f32(static_cast<uint16_t>(b[w] >> (16 * h)));
        const float xc = x * c[e], ys = y * s[e], xs = x * s[e], yc = y * c[e];
        na |= static_cast<uint32_t>(f32_to_bf16(xc - ys)) << (16 * h);
        nb |= static_cast<uint32_t>(f32_to_bf16(xs + yc)) << (16 * h);
      }
      a[w] = na;
      b[w] = nb;
    }
  }
}

// Segment of request-local position i: index of the last segment whose
// dst_start <= i (segments tile [0, N) in increasing order), or -1.
__device__ __forceinline__ int find_segment(const int4* segs, int S, int i) {
  int lo = 0, hi = S - 1, ans = -1;
  while (lo <= hi) {
    int mid = (lo + hi) >> 1;
    if (segs[mid].x <= i) {
      ans = mid;
      lo = mid + 1;
    } else {
      hi = mid - 1;
    }
  }
  if (ans >= 0 && i >= segs[ans].x + segs[ans].y) ans = -1;  // gap
  return ans;
}

}  // namespace rc
