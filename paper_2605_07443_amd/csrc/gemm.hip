// Projections of a decoder layer (QKV, O, gate/up, down) for the multi-layer
// path: Y[M, n] = X[M, k] W[n, k]^T (+ residual), bf16 storage, fp32
// accumulation on the matrix cores (v_mfma_f32_16x16x32_bf16).
//
// Both operands are k-contiguous, which is the native operand order of the
// MFMA: a lane's fragment is 8 consecutive k of one W row (the MFMA's A
// operand) or of one X row (its B operand). With W as A the accumulators hold
// Y^T, so each lane ends with 4 consecutive outputs of one row and the
// epilogue stores 8-byte packs instead of single values. A workgroup computes
// a 128 x 128 tile of Y with 4 waves of 64 x 64 (4 x 4 accumulator blocks
// each); X and W tiles of 64 k stream through double-buffered LDS (rows
// padded to 144 bytes, so the 16-byte fragment reads of 16 consecutive rows
// are conflict-free), with the next tile's global loads in flight during the
// MFMAs. Consecutive workgroups walk the 8 row tiles of a group before moving
// to the next column tile; as workgroups are dealt to the 8 XCDs in turn,
// each XCD keeps one row tile of X in its L2 while the column tiles of W
// stream past.
#include <type_traits>

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

using u32x2 = uint32_t __attribute__((ext_vector_type(2)));

// Epilogue of a wave tile of NI x NJ accumulator blocks. The W fragment is the
// MFMA's A operand and the X fragment its B operand, so block (i, j) holds
// Y^T and a lane holds columns q4*4 .. q4*4+3 of row c16: four consecutive
// outputs of one row, stored as one 8-byte pack when the row layout allows
// it (vec: n % 4 == 0 and 8-byte aligned y and residual), else one by one.
// The residual is added in fp32 before the single rounding.
template <int NI, int NJ>
__device__ __forceinline__ void store_wave_tile(const f32x4 (&acc)[NI][NJ], const uint16_t* __restrict__ res,
                                                uint16_t* __restrict__ y, int64_t M, int n, int64_t r0,
                                                int c0, int c16, int q4, bool vec) {
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int64_t gr = r0 + i * 16 + c16;
    if (gr >= M) continue;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int gc = c0 + j * 16 + q4 * 4;
      float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      if (vec && gc + 3 < n) {
        if (res) {
          const u32x2 rr = *reinterpret_cast<const u32x2*>(res + gr * n + gc);
          v[0] += bf16_to_f32(static_cast<uint16_t>(rr[0]));
          v[1] += bf16_to_f32(static_cast<uint16_t>(rr[0] >> 16));
          v[2] += bf16_to_f32(static_cast<uint16_t>(rr[1]));
          v[3] += bf16_to_f32(static_cast<uint16_t>(rr[1] >> 16));
        }
        const u32x2 o = {static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16),
                         static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16)};
        *reinterpret_cast<u32x2*>(y + gr * n + gc) = o;
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          if (gc + r >= n) continue;
          float t = v[r];
          if (res) t += bf16_to_f32(res[gr * n + gc + r]);
          y[gr * n + gc + r] = f32_to_bf16(t);
        }
      }
    }
  }
}

struct GemmSmem {
  uint16_t a[2][kGM][kGK + kGPad];
  uint16_t b[2][kGN][kGK + kGPad];
};

__global__ __launch_bounds__(kGThreads) __attribute__((amdgpu_waves_per_eu(2)))
void gemm_bf16_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
                      const uint16_t* __restrict__ res, uint16_t* __restrict__ y, int64_t M, int n,
                      int k, int tiles_m, int tiles_n, int vec) {
  __shared__ GemmSmem sm;
  // ---- tile of this workgroup: groups of kGGroup row tiles, row tile fastest inside
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
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < n_kt) {
      store(cur ^ 1);
      if (kt + 2 < n_kt) load(kt + 2);
    }
    __syncthreads();
  }

  store_wave_tile(acc, res, y, M, n, m0 + wm, n0 + wn, c16, q4, vec != 0);
}

// Large tiles for k % 64 == 0: a 256 x 256 tile per workgroup of 8 waves,
// each 128 x 64 (8 x 4 accumulator blocks), two waves per SIMD. X and W tiles
// of 64 k go straight from global memory into LDS (global_load_lds_dwordx4,
// 1 KB = 8 rows of 128 B per wave instruction), so the 16-byte chunks of a
// row are XOR-swizzled instead of padded: row r keeps data chunk c at chunk
// c ^ ((r >> 1) & 7), which puts the fragment reads of 16 consecutive rows on
// 16 distinct (bank half, chunk) pairs. The two LDS buffers are separate
// objects and every k tile knows its buffer at compile time, so loading one
// never waits on reading the other. Rows past M or n repeat the last row
// (finite values whose products are never stored).
constexpr int kBThreads = 512;
constexpr int kBM = 256, kBN = 256;
struct GemmBuf {
  uint16_t a[kBM * kGK];
  uint16_t b[kBN * kGK];
};

__global__ __launch_bounds__(kBThreads) __attribute__((amdgpu_waves_per_eu(2)))
void gemm_bf16_big_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
                          const uint16_t* __restrict__ res, uint16_t* __restrict__ y, int64_t M,
                          int n, int k, int tiles_m, int tiles_n, int vec) {
  __shared__ GemmBuf s0, s1;
  const int64_t bid = blockIdx.x;
  const int64_t per_group = static_cast<int64_t>(kGGroup) * tiles_n;
  const int64_t grp = bid / per_group;
  const int64_t in = bid - grp * per_group;
  const int64_t first_m = grp * kGGroup;
  const int64_t gm = min(static_cast<int64_t>(kGGroup), tiles_m - first_m);
  const int64_t tm = first_m + in % gm;
  const int tn = static_cast<int>(in / gm);
  const int64_t m0 = tm * kBM;
  const int n0 = tn * kBN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c16 = lane & 15;
  const int q4 = lane >> 4;
  const int wm = (wave >> 2) * 128;
  const int wn = (wave & 3) * 64;
  const int n_kt = k / kGK;

  // wave w fills rows 32w .. 32w+31 of both tiles, 8 rows per instruction
  auto issue = [&](int kt, auto buf_tag) {
    GemmBuf& dst = decltype(buf_tag)::value ? s1 : s0;
    const int ch = lane & 7;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = wave * 32 + j * 8 + (lane >> 3);
      const int dch = ch ^ ((row >> 1) & 7);
      const int64_t gr = min(m0 + row, M - 1);
      const int gc = min(n0 + row, n - 1);
      const int kk = kt * kGK + dch * 8;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(x + gr * k + kk),
                                       (__attribute__((address_space(3))) void*)(&dst.a[(wave * 32 + j * 8) * kGK]),
                                       16, 0, 0);
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void*)(w + static_cast<int64_t>(gc) * k + kk),
          (__attribute__((address_space(3))) void*)(&dst.b[(wave * 32 + j * 8) * kGK]), 16, 0, 0);
    }
  };

  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](auto buf_tag) {
    const GemmBuf& src = decltype(buf_tag)::value ? s1 : s0;
#pragma unroll
    for (int ks = 0; ks < kGK / 32; ++ks) {
      const int u = ks * 4 + q4;
      bf16x8 fb[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int rb = wn + j * 16 + c16;
        fb[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                                               &src.b[rb * kGK + ((u ^ ((rb >> 1) & 7)) * 8)]));
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int ra = wm + i * 16 + c16;
        const bf16x8 fa = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                                                       &src.a[ra * kGK + ((u ^ ((ra >> 1) & 7)) * 8)]));
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[j], fa, acc[i][j], 0, 0, 0);
      }
    }
  };
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;

  issue(0, B0{});
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  int kt = 0;
  // the scheduling barriers keep each tile's loads ahead of the MFMAs of the
  // tile before it: left free, the scheduler sinks them to the end of that
  // tile (less address-register pressure), where the wait right after them
  // exposes the whole memory latency
  for (; kt + 1 < n_kt; kt += 2) {
    issue(kt + 1, B1{});
    __builtin_amdgcn_sched_barrier(0);
    compute(B0{});
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (kt + 2 < n_kt) issue(kt + 2, B0{});
    __builtin_amdgcn_sched_barrier(0);
    compute(B1{});
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  if (kt < n_kt) compute(B0{});
  store_wave_tile(acc, res, y, M, n, m0 + wm, n0 + wn, c16, q4, vec != 0);
}

// Row tail of fewer than 256 rows left by the 256 x 256 kernel, for shapes
// where that tail would otherwise run as a few half-empty 128 x 128
// workgroups through the whole k loop (a second round as long as the first):
// split-K. Workgroup (column tile, row tile, split s) computes a 64 x 64 tile
// over the k tiles [s * KT / S, (s + 1) * KT / S) and writes its fp32 partial
// sums to part[s]; gemm_tail_reduce_kernel then adds the S partials in order
// of s and the residual, and rounds once. The partials live in the first rows
// of y, which the 256 x 256 kernel overwrites afterwards on the same stream,
// so the call allocates nothing. Four waves, each 16 columns (W rows, read
// straight from global memory one k tile ahead) x the 64 rows (X tile staged
// in LDS); operand roles and fragment layout as in the kernels above.
constexpr int kSThreads = 256;
constexpr int kSM = 64, kSN = 64;
constexpr int kSPer = kSM * kGUnits / kSThreads;   // X units per thread per k tile (2)

struct GemmSplitSmem {
  uint16_t x[2][kSM][kGK + kGPad];
};

__global__ __launch_bounds__(kSThreads)
void gemm_bf16_splitk_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
                             float* __restrict__ part, int64_t M, int n, int k, int splits) {
  __shared__ GemmSplitSmem sm;
  const int n0 = blockIdx.x * kSN;
  const int64_t m0 = static_cast<int64_t>(blockIdx.y) * kSM;
  const int s = blockIdx.z;
  const int KT = k / kGK;
  const int kt0 = static_cast<int>(static_cast<int64_t>(s) * KT / splits);
  const int kt1 = static_cast<int>(static_cast<int64_t>(s + 1) * KT / splits);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c16 = lane & 15;
  const int q4 = lane >> 4;
  const int wn = wave * 16;

  u32x4 rx[kSPer];
  auto load_x = [&](int kt) {
#pragma unroll
    for (int i = 0; i < kSPer; ++i) {
      const int u = tid + i * kSThreads;
      const int64_t gr = m0 + u / kGUnits;
      const int kk = kt * kGK + (u % kGUnits) * 8;
      rx[i] = gr < M ? *reinterpret_cast<const u32x4*>(x + gr * k + kk) : u32x4{0, 0, 0, 0};
    }
  };
  auto store_x = [&](int buf) {
#pragma unroll
    for (int i = 0; i < kSPer; ++i) {
      const int u = tid + i * kSThreads;
      *reinterpret_cast<u32x4*>(&sm.x[buf][u / kGUnits][(u % kGUnits) * 8]) = rx[i];
    }
  };
  // rows past n read row n - 1 (finite values whose sums are never stored).
  // The W fragments of the current and of the next k tile are separate named
  // registers (a runtime-indexed pair would become selects that wait for the
  // load just issued).
  const uint16_t* wrow = w + static_cast<int64_t>(min(n0 + wn + c16, n - 1)) * k + q4 * 8;
  auto load_w = [&](int kt, bf16x8 (&f)[2]) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
      f[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(wrow + kt * kGK + ks * 32));
  };
  bf16x8 wcur[2], wnext[2];

  f32x4 acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (kt0 < kt1) {
    load_x(kt0);
    load_w(kt0, wcur);
    store_x(0);
  }
  __syncthreads();
  if (kt0 + 1 < kt1) {
    load_x(kt0 + 1);
    load_w(kt0 + 1, wnext);
  }
  for (int kt = kt0; kt < kt1; ++kt) {
    const int cur = (kt - kt0) & 1;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bf16x8 fx = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(&sm.x[cur][i * 16 + c16][ks * 32 + q4 * 8]));
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wcur[ks], fx, acc[i], 0, 0, 0);
      }
    }
    if (kt + 1 < kt1) {
      store_x(cur ^ 1);
      wcur[0] = wnext[0];
      wcur[1] = wnext[1];
      if (kt + 2 < kt1) {
        load_x(kt + 2);
        load_w(kt + 2, wnext);
      }
    }
    __syncthreads();
  }
  // lane holds rows i*16 + c16, columns q4*4 .. q4*4+3 of its wave's 16
  float* ps = part + static_cast<int64_t>(s) * M * n;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t gr = m0 + i * 16 + c16;
    if (gr >= M) continue;
    const int gc = n0 + wn + q4 * 4;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (gc + r < n) ps[gr * n + gc + r] = acc[i][r];
  }
}

// y[m, c] = bf16(sum over s of part[s][m, c] (+ residual[m, c])), s in order
__global__ __launch_bounds__(256)
void gemm_tail_reduce_kernel(const float* __restrict__ part, const uint16_t* __restrict__ res,
                             uint16_t* __restrict__ y, int64_t count, int splits) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= count) return;
  float v = part[e];
  for (int s = 1; s < splits; ++s) v += part[static_cast<int64_t>(s) * count + e];
  if (res) v += bf16_to_f32(res[e]);
  y[e] = f32_to_bf16(v);
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
  if (M == 0) return RC_OK;
  auto overlaps = [](const void* a, int64_t a_bytes, const void* b, int64_t b_bytes) {
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + static_cast<uintptr_t>(b_bytes) && b0 < a0 + static_cast<uintptr_t>(a_bytes);
  };
  const int64_t y_bytes = M * n * 2;
  if (overlaps(y, y_bytes, x, M * k * 2) || overlaps(y, y_bytes, w, static_cast<int64_t>(n) * k * 2) ||
      (residual && overlaps(y, y_bytes, residual, y_bytes)))
    return fail(RC_ERR_INVALID_ARG, "y must not alias or overlap x, w or residual");
  const uint16_t* xs = static_cast<const uint16_t*>(x);
  const uint16_t* rs = static_cast<const uint16_t*>(residual);
  uint16_t* ys = static_cast<uint16_t*>(y);
  const int vec = n % 4 == 0 && reinterpret_cast<uintptr_t>(y) % 8 == 0 &&
                  reinterpret_cast<uintptr_t>(residual) % 8 == 0;
  if (k % kGK == 0 && M >= kBM && n >= kBN) {
    // whole 256-row tiles on the big kernel; a tail of fewer than 256 rows
    // goes to split-K (below) when the 128 x 128 kernel would run it on few
    // workgroups, else to that kernel (a partial big tile would cost as much
    // as a full one and, with few tiles per CU, a whole extra round)
    const int64_t M_main = (M / kBM) * kBM;
    const int64_t tm = M_main / kBM;
    const int tn = (n + kBN - 1) / kBN;
    if (tm * tn > 0x7fffffff) return fail(RC_ERR_UNSUPPORTED, "grid too large");
    const int64_t M_tail = M - M_main;
    const int KT = k / kGK;
    const int64_t small_tiles = ((M_tail + kGM - 1) / kGM) * ((n + kGN - 1) / kGN);
    const int64_t split_tiles = ((M_tail + kSM - 1) / kSM) * ((n + kSN - 1) / kSN);
    // splits: about 512 workgroups, at least 2 k tiles each, and the partials
    // (splits x M_tail x n fp32) inside the first M_main rows of y (bf16)
    int64_t splits64 = 512 / (split_tiles > 0 ? split_tiles : 1);
    if (splits64 > KT / 2) splits64 = KT / 2;
    if (M_tail > 0 && splits64 > M_main / (2 * M_tail)) splits64 = M_main / (2 * M_tail);
    const int splits = static_cast<int>(splits64);
    if (M_tail > 0 && small_tiles < 128 && splits >= 2 && reinterpret_cast<uintptr_t>(y) % 16 == 0) {
      float* part = reinterpret_cast<float*>(ys);
      hipLaunchKernelGGL(gemm_bf16_splitk_kernel,
                         dim3(static_cast<unsigned>((n + kSN - 1) / kSN), static_cast<unsigned>((M_tail + kSM - 1) / kSM),
                              static_cast<unsigned>(splits)),
                         dim3(kSThreads), 0, stream, xs + M_main * k, static_cast<const uint16_t*>(w), part,
                         M_tail, n, k, splits);
      if (int st = check_launch("rc_gemm_bf16")) return st;
      const int64_t count = M_tail * n;
      hipLaunchKernelGGL(gemm_tail_reduce_kernel, dim3(static_cast<unsigned>((count + 255) / 256)), dim3(256), 0,
                         stream, part, rs ? rs + M_main * n : nullptr, ys + M_main * n, count, splits);
      if (int st = check_launch("rc_gemm_bf16")) return st;
      // the body last: it overwrites the partials
      hipLaunchKernelGGL(gemm_bf16_big_kernel, dim3(static_cast<unsigned>(tm * tn)), dim3(kBThreads), 0,
                         stream, xs, static_cast<const uint16_t*>(w), rs, ys, M_main, n, k,
                         static_cast<int>(tm), tn, vec);
      return check_launch("rc_gemm_bf16");
    }
    hipLaunchKernelGGL(gemm_bf16_big_kernel, dim3(static_cast<unsigned>(tm * tn)), dim3(kBThreads), 0,
                       stream, xs, static_cast<const uint16_t*>(w), rs, ys, M_main, n, k,
                       static_cast<int>(tm), tn, vec);
    if (int st = check_launch("rc_gemm_bf16")) return st;
    if (M_main == M) return RC_OK;
    xs += M_main * k;
    if (rs) rs += M_main * n;
    ys += M_main * n;
    M -= M_main;
  }
  const int64_t tiles_m = (M + kGM - 1) / kGM;
  const int tiles_n = (n + kGN - 1) / kGN;
  const int64_t blocks = tiles_m * tiles_n;
  if (blocks > 0x7fffffff) return fail(RC_ERR_UNSUPPORTED, "grid too large");
  hipLaunchKernelGGL(gemm_bf16_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kGThreads), 0,
                     stream, xs, static_cast<const uint16_t*>(w), rs, ys, M, n, k,
                     static_cast<int>(tiles_m), tiles_n, vec);
  return check_launch("rc_gemm_bf16");
}
