// Projections of a decoder layer (QKV, O, gate/up, down) for the multi-layer
// path: Y[M, n] = X[M, k] W[n, k]^T (+ residual), bf16 storage, fp32
// accumulation on the matrix cores (v_mfma_f32_16x16x32_bf16).
//
// Both operands are k-contiguous, which is the native operand order of the
// MFMA: a lane's A fragment is 8 consecutive k of one X row and its B
// fragment 8 consecutive k of one W row. A workgroup computes a 128 x 128
// tile of Y with 4 waves of 64 x 64 (4 x 4 accumulator blocks each); X and W
// tiles of 64 k stream through double-buffered LDS (rows padded to 144 bytes,
// so the 16-byte fragment reads of 16 consecutive rows are conflict-free),
// with the next tile's global loads in flight during the MFMAs. Tiles are
// ordered n-fastest within groups of 8 row tiles, so the workgroups running
// together share both operands in L2.
#include "rc_common.h"

namespace rc {
namespace {

using u32x4 = u32x4_t;
constexpr int kGThreads = 256;
constexpr int kGM = 128, kGN = 128, kGK = 64;
constexpr int kGPad = 8;
constexpr int kGGroup = 8;  // row tiles per ordering group
constexpr int kGUnits = kGK / 8;                              // 16-byte units per tile row
constexpr int kGPer = kGM * kGUnits / kGThreads;              // units per thread per operand (4)

struct GemmSmem {
  uint16_t a[2][kGM][kGK + kGPad];
  uint16_t b[2][kGN][kGK + kGPad];
};

__global__ __launch_bounds__(kGThreads) __attribute__((amdgpu_waves_per_eu(2)))
void gemm_bf16_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
                      const uint16_t* __restrict__ res, uint16_t* __restrict__ y, int64_t M, int n,
                      int k, int tiles_m, int tiles_n) {
  __shared__ GemmSmem sm;
  // ---- tile of this workgroup: groups of kGGroup row tiles, n fastest inside
  const int64_t bid = blockIdx.x;
  const int64_t per_group = static_cast<int64_t>(kGGroup) * tiles_n;
  const int64_t grp = bid / per_group;
  const int64_t in = bid - grp * per_group;
  const int64_t first_m = grp * kGGroup;
  const int64_t gm = min(static_cast<int64_t>(kGGroup), tiles_m - first_m);
  const int64_t tm = first_m + in % gm;
  const int tn = static_cast<int>(in / gm);
  const int64_t m0 = tm * kGM;
  const int n0 = tn * kGN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c16 = lane & 15;
  const int q4 = lane >> 4;
  const int wm = (wave >> 1) * 64;  // wave tile origin inside the workgroup tile
  const int wn = (wave & 1) * 64;

  // ---- staging: thread owns units u = tid + i*256: row u / 8, k offset (u % 8) * 8
  u32x4 ra[kGPer], rb[kGPer];
  const int n_kt = (k + kGK - 1) / kGK;
  auto load = [&](int kt) {
#pragma unroll
    for (int i = 0; i < kGPer; ++i) {
      const int u = tid + i * kGThreads;
      const int row = u / kGUnits;
      const int kk = kt * kGK + (u % kGUnits) * 8;
      const int64_t gr = m0 + row;
      const int gc = n0 + row;
      ra[i] = (gr < M && kk < k) ? *reinterpret_cast<const u32x4*>(x + gr * k + kk) : u32x4{0, 0, 0, 0};
      rb[i] = (gc < n && kk < k)
                  ? *reinterpret_cast<const u32x4*>(w + static_cast<int64_t>(gc) * k + kk)
                  : u32x4{0, 0, 0, 0};
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < kGPer; ++i) {
      const int u = tid + i * kGThreads;
      const int row = u / kGUnits;
      const int col = (u % kGUnits) * 8;
      *reinterpret_cast<u32x4*>(&sm.a[buf][row][col]) = ra[i];
      *reinterpret_cast<u32x4*>(&sm.b[buf][row][col]) = rb[i];
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  load(0);
  store(0);
  __syncthreads();
  if (n_kt > 1) load(1);
  for (int kt = 0; kt < n_kt; ++kt) {
    const int cur = kt & 1;
#pragma unroll
    for (int ks = 0; ks < kGK / 32; ++ks) {
      bf16x8 fa[4], fb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        fa[i] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(&sm.a[cur][wm + i * 16 + c16][ks * 32 + q4 * 8]));
        fb[i] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(&sm.b[cur][wn + i * 16 + c16][ks * 32 + q4 * 8]));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < n_kt) {
      store(cur ^ 1);
      if (kt + 2 < n_kt) load(kt + 2);
    }
    __syncthreads();
  }

  // ---- epilogue: lane holds rows q4*4 + r of column c16 of each 16 x 16 block
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int gc = n0 + wn + j * 16 + c16;
      if (gc >= n) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t gr = m0 + wm + i * 16 + q4 * 4 + r;
        if (gr >= M) continue;
        float v = acc[i][j][r];
        if (res) v += bf16_to_f32(res[gr * n + gc]);
        y[gr * n + gc] = f32_to_bf16(v);
      }
    }
}

}  // namespace
}  // namespace rc

extern "C" int rc_gemm_bf16(int64_t M, int32_t n, int32_t k, const void* x, const void* w,
                            const void* residual, void* y, hipStream_t stream) {
  using namespace rc;
  clear_error();
  if (!x || !w || !y) return fail(RC_ERR_INVALID_ARG, "x, w and y must be non-NULL");
  if (M < 0 || n < 1 || k < 8 || k % 8)
    return fail(RC_ERR_INVALID_ARG, "M=%lld n=%d k=%d (k a positive multiple of 8)",
                static_cast<long long>(M), n, k);
  if (residual == y) return fail(RC_ERR_INVALID_ARG, "residual must not alias y");
  if (M == 0) return RC_OK;
  const int64_t tiles_m = (M + kGM - 1) / kGM;
  const int tiles_n = (n + kGN - 1) / kGN;
  const int64_t blocks = tiles_m * tiles_n;
  if (blocks > 0x7fffffff) return fail(RC_ERR_UNSUPPORTED, "grid too large");
  hipLaunchKernelGGL(gemm_bf16_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kGThreads), 0,
                     stream, static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w),
                     static_cast<const uint16_t*>(residual), static_cast<uint16_t*>(y), M, n, k,
                     static_cast<int>(tiles_m), tiles_n);
  return check_launch("rc_gemm_bf16");
}
