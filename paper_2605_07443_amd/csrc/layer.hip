// Decoder-layer pieces for recomputing only the selected rows through a stack
// of layers (RcLLM, arXiv 2605.07443, Sec. III-C.2b: the first layer is
// computed in full, later layers recompute the heavy hitters and reuse the
// cached K/V of every other token). All four are HBM-bound row kernels:
//
//   rmsnorm_kernel     y = x * rsqrt(mean(x^2) + eps) * gamma per row (fp32
//                      statistics, one workgroup per row)
//   qkv_rope_kernel    splits a fused QKV projection row, rotates q and k by
//                      the row's absolute position (the gather's fp32
//                      operation order) and writes q, k, v at that position
//                      of [B, N, H, D] tensors -- for a cached layer this is
//                      the heavy-hitter update of its assembled K/V
//   silu_mul_kernel    SwiGLU activation silu(gate) * up
//   gather_rows_kernel dst[b, r] = src[b, rows[b, r]] (residual rows)
#include <cmath>

#include "rc_common.h"

namespace rc {
namespace {

using u32x4 = u32x4_t;
constexpr int kRowThreads = 256;
constexpr int kNormMaxUnits = 4;  // 16-byte units per thread kept in registers (H <= 8192)

__global__ __launch_bounds__(kRowThreads) void rmsnorm_kernel(const uint16_t* __restrict__ x,
                                                             const uint16_t* __restrict__ gamma,
                                                             int H, float eps,
                                                             uint16_t* __restrict__ y) {
  __shared__ float s_red[kRowThreads / 64];
  const size_t row = blockIdx.x;
  const int units = H / 8;
  const u32x4* xr = reinterpret_cast<const u32x4*>(x + row * H);
  u32x4 buf[kNormMaxUnits];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kNormMaxUnits; ++j) {
    const int u = threadIdx.x + j * kRowThreads;
    if (u < units) {
      buf[j] = xr[u];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float a = bf16_to_f32(static_cast<uint16_t>(buf[j][w]));
        const float b = bf16_to_f32(static_cast<uint16_t>(buf[j][w] >> 16));
        ss += a * a + b * b;
      }
    }
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kRowThreads / 64; ++w) tot += s_red[w];
  const float inv = 1.f / sqrtf(tot / static_cast<float>(H) + eps);
  const u32x4* gr = reinterpret_cast<const u32x4*>(gamma);
  u32x4* yr = reinterpret_cast<u32x4*>(y + row * H);
#pragma unroll
  for (int j = 0; j < kNormMaxUnits; ++j) {
    const int u = threadIdx.x + j * kRowThreads;
    if (u < units) {
      const u32x4 g = gr[u];
      u32x4 o;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float a = bf16_to_f32(static_cast<uint16_t>(buf[j][w])) * inv *
                        bf16_to_f32(static_cast<uint16_t>(g[w]));
        const float b = bf16_to_f32(static_cast<uint16_t>(buf[j][w] >> 16)) * inv *
                        bf16_to_f32(static_cast<uint16_t>(g[w] >> 16));
        o[w] = static_cast<uint32_t>(f32_to_bf16(a)) | (static_cast<uint32_t>(f32_to_bf16(b)) << 16);
      }
      yr[u] = o;
    }
  }
}

// One workgroup per projected row m = b * R + r; its position is rows[m]
// (or r when rows is NULL, R == N).
__global__ __launch_bounds__(kRowThreads) void qkv_rope_kernel(
    const uint16_t* __restrict__ qkv, const int32_t* __restrict__ rows, int R, int N, int Hq,
    int Hkv, int D, const float* __restrict__ cos_t, const float* __restrict__ sin_t, int max_pos,
    uint16_t* __restrict__ q_out, uint16_t* __restrict__ k_out, uint16_t* __restrict__ v_out) {
  const int m = blockIdx.x;
  const int b = m / R;
  const int r = m - b * R;
  const int pos = rows ? rows[m] : r;
  if (pos < 0 || pos >= N) return;
  const int half_units = D / 16;            // 16-byte units in half a head
  const int q_pairs = Hq * half_units;
  const int k_pairs = Hkv * half_units;
  const int v_units = Hkv * 2 * half_units;
  const bool rot = cos_t != nullptr && pos < max_pos;
  const u32x4* src = reinterpret_cast<const u32x4*>(qkv + static_cast<size_t>(m) * (Hq + 2 * Hkv) * D);
  const size_t row_q = (static_cast<size_t>(b) * N + pos) * Hq * D;
  const size_t row_kv = (static_cast<size_t>(b) * N + pos) * Hkv * D;
  for (int it = threadIdx.x; it < q_pairs + k_pairs + v_units; it += kRowThreads) {
    if (it < q_pairs + k_pairs) {
      const bool isq = it < q_pairs;
      const int p = isq ? it : it - q_pairs;
      const int head = p / half_units;
      const int u = p - head * half_units;
      const int base = (isq ? 0 : Hq * 2 * half_units) + head * 2 * half_units;  // units
      u32x4 a = src[base + u];
      u32x4 c = src[base + u + half_units];
      if (rot) {
        float cs[8], sn[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          cs[e] = cos_t[static_cast<size_t>(pos) * (D / 2) + u * 8 + e];
          sn[e] = sin_t[static_cast<size_t>(pos) * (D / 2) + u * 8 + e];
        }
        rotate_unit<2>(a, c, cs, sn);
      }
      u32x4* dst = reinterpret_cast<u32x4*>(isq ? q_out + row_q + static_cast<size_t>(head) * D
                                                : k_out + row_kv + static_cast<size_t>(head) * D);
      dst[u] = a;
      dst[u + half_units] = c;
    } else {
      const int u = it - q_pairs - k_pairs;
      reinterpret_cast<u32x4*>(v_out + row_kv)[u] = src[(Hq + Hkv) * 2 * half_units + u];
    }
  }
}

// out[m, i] = silu(gu[m, i]) * gu[m, I + i], 8 elements per thread
__global__ __launch_bounds__(kRowThreads) void silu_mul_kernel(const uint16_t* __restrict__ gu,
                                                              int64_t M, int I,
                                                              uint16_t* __restrict__ out) {
  const int upr = I / 8;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kRowThreads + threadIdx.x;
  if (idx >= M * upr) return;
  const int64_t m = idx / upr;
  const int u = static_cast<int>(idx - m * upr);
  const u32x4 g = reinterpret_cast<const u32x4*>(gu + m * 2 * I)[u];
  const u32x4 p = reinterpret_cast<const u32x4*>(gu + m * 2 * I + I)[u];
  u32x4 o;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t packed = 0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float a = bf16_to_f32(static_cast<uint16_t>(g[w] >> (16 * h)));
      const float b = bf16_to_f32(static_cast<uint16_t>(p[w] >> (16 * h)));
      const float s = a / (1.f + expf(-a));
      packed |= static_cast<uint32_t>(f32_to_bf16(s * b)) << (16 * h);
    }
    o[w] = packed;
  }
  reinterpret_cast<u32x4*>(out + m * I)[u] = o;
}

__global__ __launch_bounds__(kRowThreads) void gather_rows_kernel(const char* __restrict__ src,
                                                                 const int32_t* __restrict__ rows,
                                                                 int R, int Nsrc, int units,
                                                                 char* __restrict__ dst) {
  const int m = blockIdx.x;
  const int b = m / R;
  const int p = rows[m];
  if (p < 0 || p >= Nsrc) return;
  const u32x4* s = reinterpret_cast<const u32x4*>(src + (static_cast<size_t>(b) * Nsrc + p) * units * 16);
  u32x4* d = reinterpret_cast<u32x4*>(dst + static_cast<size_t>(m) * units * 16);
  for (int u = threadIdx.x; u < units; u += kRowThreads) d[u] = s[u];
}

}  // namespace
}  // namespace rc

extern "C" int rc_rmsnorm(int32_t M, int32_t H, const void* x, const void* gamma, float eps,
                          void* y, hipStream_t stream) {
  using namespace rc;
  clear_error();
  if (!x || !gamma || !y) return fail(RC_ERR_INVALID_ARG, "x, gamma and y must be non-NULL");
  if (M < 0 || H < 8 || H % 8) return fail(RC_ERR_INVALID_ARG, "M=%d H=%d (H a multiple of 8)", M, H);
  if (H > 8 * kNormMaxUnits * kRowThreads) return fail(RC_ERR_UNSUPPORTED, "H=%d exceeds 8192", H);
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(RC_ERR_INVALID_ARG, "eps must be finite and >= 0");
  if (M == 0) return RC_OK;
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(M), dim3(kRowThreads), 0, stream,
                     static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(gamma), H, eps,
                     static_cast<uint16_t*>(y));
  return check_launch("rc_rmsnorm");
}

extern "C" int rc_qkv_rope(const rc_shape* shape, const void* qkv, const int32_t* rows, int32_t R,
                           const float* rope_cos, const float* rope_sin, int32_t max_pos,
                           void* q_out, void* k_out, void* v_out, hipStream_t stream) {
  using namespace rc;
  clear_error();
  if (int st = check_shape(shape, true)) return st;
  if (shape->dtype != RC_BF16) return fail(RC_ERR_UNSUPPORTED, "rc_qkv_rope is implemented for bf16");
  if (!qkv || !q_out || !k_out || !v_out) return fail(RC_ERR_INVALID_ARG, "NULL tensor");
  if (!rows && R != shape->N) return fail(RC_ERR_INVALID_ARG, "rows NULL needs R == N");
  if (R < 0) return fail(RC_ERR_INVALID_ARG, "R=%d must be >= 0", R);
  if ((rope_cos == nullptr) != (rope_sin == nullptr))
    return fail(RC_ERR_INVALID_ARG, "rope_cos and rope_sin must both be given or both be NULL");
  if (rope_cos && max_pos < shape->N) return fail(RC_ERR_INVALID_ARG, "max_pos=%d < N=%d", max_pos, shape->N);
  const int64_t M = static_cast<int64_t>(shape->B) * R;
  if (M > 0x7fffffff) return fail(RC_ERR_UNSUPPORTED, "too many rows");
  if (M == 0) return RC_OK;
  hipLaunchKernelGGL(qkv_rope_kernel, dim3(static_cast<unsigned>(M)), dim3(kRowThreads), 0, stream,
                     static_cast<const uint16_t*>(qkv), rows, R, shape->N, shape->Hq, shape->Hkv,
                     shape->D, rope_cos, rope_sin, rope_cos ? max_pos : 0,
                     static_cast<uint16_t*>(q_out), static_cast<uint16_t*>(k_out),
                     static_cast<uint16_t*>(v_out));
  return check_launch("rc_qkv_rope");
}

extern "C" int rc_silu_mul(int64_t M, int32_t I, const void* gate_up, void* out, hipStream_t stream) {
  using namespace rc;
  clear_error();
  if (!gate_up || !out) return fail(RC_ERR_INVALID_ARG, "gate_up and out must be non-NULL");
  if (M < 0 || I < 8 || I % 8) return fail(RC_ERR_INVALID_ARG, "M=%lld I=%d (I a multiple of 8)",
                                           static_cast<long long>(M), I);
  const int64_t items = M * (I / 8);
  const int64_t blocks = (items + kRowThreads - 1) / kRowThreads;
  if (blocks > 0x7fffffff) return fail(RC_ERR_UNSUPPORTED, "too many elements");
  if (items == 0) return RC_OK;
  hipLaunchKernelGGL(silu_mul_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kRowThreads), 0,
                     stream, static_cast<const uint16_t*>(gate_up), M, I, static_cast<uint16_t*>(out));
  return check_launch("rc_silu_mul");
}

extern "C" int rc_gather_rows(int32_t B, int32_t Nsrc, int32_t R, int32_t row_bytes,
                              const void* src, const int32_t* rows, void* dst, hipStream_t stream) {
  using namespace rc;
  clear_error();
  if (!src || !rows || !dst) return fail(RC_ERR_INVALID_ARG, "src, rows and dst must be non-NULL");
  if (B < 1 || Nsrc < 1 || R < 0 || row_bytes < 16 || row_bytes % 16)
    return fail(RC_ERR_INVALID_ARG, "B=%d Nsrc=%d R=%d row_bytes=%d (a multiple of 16)", B, Nsrc, R,
                row_bytes);
  const int64_t M = static_cast<int64_t>(B) * R;
  if (M > 0x7fffffff) return fail(RC_ERR_UNSUPPORTED, "too many rows");
  if (M == 0) return RC_OK;
  hipLaunchKernelGGL(gather_rows_kernel, dim3(static_cast<unsigned>(M)), dim3(kRowThreads), 0, stream,
                     static_cast<const char*>(src), rows, R, Nsrc, row_bytes / 16,
                     static_cast<char*>(dst));
  return check_launch("rc_gather_rows");
}
