// Heavy-hitter selection and correction (RcLLM, arXiv 2605.07443,
// Sec. III-C.2b with the deviation term of Eq. (3) for M = K, lambda = 1, and
// Sec. III-C.3 step (iii)).
//
//   deviation_kernel  one wave per position: L1 distance between the fresh
//                     and the assembled key row (HBM-bound, 16-byte loads,
//                     wave reduction)
//   topk_kernel       one 1024-thread workgroup per request: range-adaptive
//                     radix select of the k-th largest score key in LDS
//                     (11-bit digits), then a block scan that emits the fresh
//                     and selected positions in ascending order
//   patch_kernel      copies the fresh K/V rows of the selected cached
//                     positions over the assembled rows
#include "rc_common.h"

namespace rc {
namespace {

using u32x4 = uint32_t __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ deviation

constexpr int kDevWaves = 4;
constexpr int kDevTokPerWave = 4;

// d[t] = sum |k_fresh[t] - k_asm[t]| over the row of t (t = b*N + i).
template <int ES>
__global__ __launch_bounds__(64 * kDevWaves) void deviation_kernel(
    const char* __restrict__ k_fresh, const char* __restrict__ k_asm, int64_t rows, int row_units,
    float* __restrict__ scores) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t t0 = (static_cast<int64_t>(blockIdx.x) * kDevWaves + wave) * kDevTokPerWave;
  float acc[kDevTokPerWave];
#pragma unroll
  for (int r = 0; r < kDevTokPerWave; ++r) acc[r] = 0.f;
  for (int u0 = 0; u0 < row_units; u0 += 64) {
    const int u = u0 + lane;
    u32x4 a[kDevTokPerWave], c[kDevTokPerWave];
#pragma unroll
    for (int r = 0; r < kDevTokPerWave; ++r) {
      const int64_t t = t0 + r;
      if (t < rows && u < row_units) {
        a[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(k_fresh + t * row_units * 16) + u);
        c[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(k_asm + t * row_units * 16) + u);
      }
    }
#pragma unroll
    for (int r = 0; r < kDevTokPerWave; ++r)
      if (t0 + r < rows && u < row_units) acc[r] += absdiff_sum<ES>(a[r], c[r]);
  }
#pragma unroll
  for (int r = 0; r < kDevTokPerWave; ++r) {
    const float s = wave_sum(acc[r]);
    if (lane == 0 && t0 + r < rows) scores[t0 + r] = s;
  }
}

// ---------------------------------------------------------------------- top-k

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;
constexpr int kBins = 2048;  // 11-bit digits
constexpr int kDigitBits = 11;
constexpr int kBinsPerThread = kBins / kTopkThreads;

// Total order on fp32: larger key = larger value; +NaN above +inf.
__device__ __forceinline__ uint32_t score_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Inclusive block scan of one int per thread (1024 threads); also returns
// the block total. `warp_tot` is LDS scratch of kTopkWaves ints.
__device__ __forceinline__ int block_inclusive_scan(int x, int* warp_tot, int& total) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) warp_tot[wave] = x;
  __syncthreads();
  int before = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kTopkWaves; ++w) {
    const int v = warp_tot[w];
    before += (w < wave) ? v : 0;
    total += v;
  }
  __syncthreads();
  return x + before;
}

__device__ __forceinline__ int block_sum(int x, int* warp_tot) {
  int total;
  block_inclusive_scan(x, warp_tot, total);
  return total;
}

// One workgroup per request. Candidates are positions outside fresh
// segments; each belongs to one of two classes: class 0 (history, or every
// cached position when item_mask is 0) and class 1 (blocks of the pools set
// in item_mask). Class c keeps its k_c largest keys, key of position i =
// score_key(score[i]), order (key desc, i asc). Fresh positions are always
// taken; the taken positions are written in ascending order. NC: number of
// classes with a budget (1: class 0 only, k1 is 0).
template <int NC>
__global__ __launch_bounds__(kTopkThreads) void topk_kernel(
    const float* __restrict__ scores, const int4* __restrict__ segs, int S, int N,
    uint32_t item_mask, int k0, int k1, int R, int32_t* __restrict__ rows) {
  __shared__ uint32_t s_key[kMaxSelectN];
  __shared__ uint8_t s_cls[kMaxSelectN];  // 0 fresh, 1 + class for candidates; bit 7 = taken
  __shared__ int4 s_segs[kMaxSegments];
  __shared__ int s_hist[kBins];
  __shared__ int s_wt[kTopkWaves];
  __shared__ uint32_t s_bounds[NC][4];

  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  for (int s = tid; s < S; s += kTopkThreads) s_segs[s] = segs[static_cast<size_t>(b) * S + s];
  if (tid < NC) {
    s_bounds[tid][0] = 0xffffffffu;
    s_bounds[tid][1] = 0u;
  }
  __syncthreads();

  uint32_t kmin[2] = {0xffffffffu, 0xffffffffu}, kmax[2] = {0u, 0u};
  int ncand[2] = {0, 0};
  for (int i = tid; i < N; i += kTopkThreads) {
    const int s = find_segment(s_segs, S, i);
    const int pool = s >= 0 ? s_segs[s].z : -1;
    const int cls = pool < 0 ? 0 : 1 + static_cast<int>(pool < 32 && ((item_mask >> pool) & 1u));
    const uint32_t key = score_key(scores[static_cast<size_t>(b) * N + i]);
    s_key[i] = key;
    s_cls[i] = static_cast<uint8_t>(cls);
#pragma unroll
    for (int c = 0; c < NC; ++c)
      if (cls == c + 1) {
        kmin[c] = min(kmin[c], key);
        kmax[c] = max(kmax[c], key);
        ++ncand[c];
      }
  }
  // block reductions of min/max/count per class
#pragma unroll
  for (int c = 0; c < NC; ++c) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      kmin[c] = min(kmin[c], static_cast<uint32_t>(__shfl_xor(static_cast<int>(kmin[c]), off, 64)));
      kmax[c] = max(kmax[c], static_cast<uint32_t>(__shfl_xor(static_cast<int>(kmax[c]), off, 64)));
    }
    if ((tid & 63) == 0) {
      atomicMin(&s_bounds[c][0], kmin[c]);
      atomicMax(&s_bounds[c][1], kmax[c]);
    }
  }
  const int kc_arg[2] = {k0, k1};
  int kk[2] = {0, 0};
  uint32_t T[2] = {0u, 0u};
  int need[2] = {0, 0};
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    if (kc_arg[c] <= 0) continue;  // uniform: kernel arguments
    const int nc = block_sum(ncand[c], s_wt);  // contains barriers
    kk[c] = min(kc_arg[c], nc);
    if (kk[c] == 0) continue;
    // ---- threshold key T_c: the kk-th largest key of class c
    uint32_t lo = s_bounds[c][0], hi = s_bounds[c][1];
    int nd = kk[c];  // how many of the class's keys in [lo, hi] we still take
    const uint8_t want = static_cast<uint8_t>(c + 1);
    while (lo != hi) {
      const uint32_t range = hi - lo;
      const int bits = 32 - __clz(range);
      const int shift = bits > kDigitBits ? bits - kDigitBits : 0;
      for (int j = tid; j < kBins; j += kTopkThreads) s_hist[j] = 0;
      __syncthreads();
      for (int i = tid; i < N; i += kTopkThreads) {
        const uint32_t key = s_key[i];
        if (s_cls[i] == want && key >= lo && key <= hi) atomicAdd(&s_hist[(key - lo) >> shift], 1);
      }
      __syncthreads();
      // suffix sums from the top bin: thread t owns kBinsPerThread adjacent
      // bins, threads ordered from the highest bins down
      const int top = kBins - 1 - kBinsPerThread * tid;
      int cnt[kBinsPerThread];
      int mine = 0;
#pragma unroll
      for (int j = 0; j < kBinsPerThread; ++j) {
        cnt[j] = s_hist[top - j];
        mine += cnt[j];
      }
      int total;
      int run = block_inclusive_scan(mine, s_wt, total) - mine;  // count in bins above `top`
      // the bin where the running count first reaches `nd`
      if (run < nd && run + mine >= nd) {
#pragma unroll
        for (int j = 0; j < kBinsPerThread; ++j) {
          if (run < nd && run + cnt[j] >= nd) {
            s_bounds[c][2] = static_cast<uint32_t>(top - j);
            s_bounds[c][3] = static_cast<uint32_t>(run);
          }
          run += cnt[j];
        }
      }
      __syncthreads();
      const uint32_t bin = s_bounds[c][2];
      nd -= static_cast<int>(s_bounds[c][3]);
      const uint32_t nlo = lo + (bin << shift);
      const uint32_t width_m1 = (shift >= 32) ? 0xffffffffu : ((1u << shift) - 1u);
      const uint32_t nhi = (hi - nlo > width_m1) ? nlo + width_m1 : hi;
      lo = nlo;
      hi = nhi;
      __syncthreads();
    }
    T[c] = lo;
    need[c] = nd;  // candidates of class c with key == T_c to take, lowest positions first
  }

  __syncthreads();  // s_key / s_cls complete even when no class ran a selection

  // ---- emit rows: fresh positions, keys > T_c, and the first need_c ties
  const int per = (N + kTopkThreads - 1) / kTopkThreads;
  const int beg = min(N, tid * per), end = min(N, beg + per);
  int ties = 0;  // class-0 ties in the low 16 bits, class-1 ties in the high 16
  for (int i = beg; i < end; ++i) {
    const int cls = s_cls[i];
    if (cls == 1 && kk[0] > 0 && s_key[i] == T[0]) ties += 1;
    if (NC == 2 && cls == 2 && kk[1] > 0 && s_key[i] == T[1]) ties += 1 << 16;
  }
  int tot;
  const int tb = block_inclusive_scan(ties, s_wt, tot) - ties;
  int tb0 = tb & 0xffff, tb1 = tb >> 16;  // ties of each class before this thread
  int take = 0;
  for (int i = beg; i < end; ++i) {
    const int cls = s_cls[i];
    bool t;
    if (cls == 0) {
      t = true;
    } else if (NC == 1 && cls == 2) {
      t = false;  // class 1 has no budget
    } else {
      const bool one = NC == 2 && cls == 2;
      const int kkc = one ? kk[1] : kk[0];
      const uint32_t Tc = one ? T[1] : T[0];
      const int ndc = one ? need[1] : need[0];
      const uint32_t key = s_key[i];
      if (kkc == 0) {
        t = false;
      } else if (key > Tc) {
        t = true;
      } else if (key == Tc) {
        if (one) {
          t = tb1 < ndc;
          ++tb1;
        } else {
          t = tb0 < ndc;
          ++tb0;
        }
      } else {
        t = false;
      }
    }
    take += t ? 1 : 0;
    s_cls[i] = static_cast<uint8_t>(cls | (t ? 0x80 : 0));
  }
  __syncthreads();
  int out = block_inclusive_scan(take, s_wt, tot) - take;
  for (int i = beg; i < end; ++i) {
    if (s_cls[i] & 0x80) {
      if (out < R) rows[static_cast<size_t>(b) * R + out] = i;
      ++out;
    }
  }
  // pad a short list (inconsistent n_fresh) with the last position
  __syncthreads();
  for (int r = tot + tid; r < R; r += kTopkThreads) rows[static_cast<size_t>(b) * R + r] = N - 1;
}

// ------------------------------------------------------------------ Eq. (3)

// Full importance score, one wave per position (4 per wave, grid.y = request):
//   S_i = (1 - lambda) sum_g mass[b, g, i]
//         + lambda (|K_fresh - K_asm|_1 + |V_fresh - V_asm|_1)   (not for item blocks)
template <int ES>
__global__ __launch_bounds__(64 * kDevWaves) void eq3_score_kernel(
    const int4* __restrict__ segs, int S, int N, int Hkv, uint32_t item_mask, float lambda,
    const float* __restrict__ mass, const char* __restrict__ k_fresh,
    const char* __restrict__ v_fresh, const char* __restrict__ k_asm,
    const char* __restrict__ v_asm, int row_units, float* __restrict__ scores) {
  __shared__ int4 s_segs[kMaxSegments];
  const int b = blockIdx.y;
  for (int s = threadIdx.x; s < S; s += 64 * kDevWaves) s_segs[s] = segs[static_cast<size_t>(b) * S + s];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int i0 = (blockIdx.x * kDevWaves + wave) * kDevTokPerWave;
  float dev[kDevTokPerWave];
  bool div[kDevTokPerWave];
#pragma unroll
  for (int r = 0; r < kDevTokPerWave; ++r) {
    dev[r] = 0.f;
    const int i = i0 + r;
    div[r] = false;
    if (i < N) {
      const int s = find_segment(s_segs, S, i);
      const int pool = s >= 0 ? s_segs[s].z : -1;
      div[r] = !(pool >= 0 && pool < 32 && ((item_mask >> pool) & 1u));
    }
  }
  for (int u0 = 0; u0 < row_units; u0 += 64) {
    const int u = u0 + lane;
    u32x4 a[kDevTokPerWave], c[kDevTokPerWave], e[kDevTokPerWave], f[kDevTokPerWave];
#pragma unroll
    for (int r = 0; r < kDevTokPerWave; ++r) {
      if (div[r] && u < row_units) {
        const size_t off = (static_cast<size_t>(b) * N + i0 + r) * row_units + u;
        a[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(k_fresh) + off);
        c[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(k_asm) + off);
        e[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(v_fresh) + off);
        f[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(v_asm) + off);
      }
    }
#pragma unroll
    for (int r = 0; r < kDevTokPerWave; ++r)
      if (div[r] && u < row_units) dev[r] += absdiff_sum<ES>(a[r], c[r]) + absdiff_sum<ES>(e[r], f[r]);
  }
#pragma unroll
  for (int r = 0; r < kDevTokPerWave; ++r) {
    const int i = i0 + r;
    const float d = wave_sum(dev[r]);
    float m = 0.f;
    if (i < N)
      for (int g = lane; g < Hkv; g += 64) m += mass[(static_cast<size_t>(b) * Hkv + g) * N + i];
    m = wave_sum(m);
    if (lane == 0 && i < N) scores[static_cast<size_t>(b) * N + i] = (1.f - lambda) * m + lambda * d;
  }
}

// ---------------------------------------------------------------------- patch

constexpr int kPatchThreads = 256;

__global__ __launch_bounds__(kPatchThreads) void patch_kernel(
    const int4* __restrict__ segs, int S, int N, const int32_t* __restrict__ rows, int R,
    int rows_per_wg, int row_units, const char* __restrict__ k_fresh,
    const char* __restrict__ v_fresh, char* __restrict__ k_asm, char* __restrict__ v_asm) {
  __shared__ int4 s_segs[kMaxSegments];
  __shared__ int s_pos[256];
  const int b = blockIdx.y;
  const int r0 = blockIdx.x * rows_per_wg;
  const int cnt = min(rows_per_wg, R - r0);
  for (int s = threadIdx.x; s < S; s += kPatchThreads) s_segs[s] = segs[static_cast<size_t>(b) * S + s];
  __syncthreads();
  for (int t = threadIdx.x; t < cnt; t += kPatchThreads) {
    const int i = rows[static_cast<size_t>(b) * R + r0 + t];
    int pos = -1;
    if (i >= 0 && i < N) {
      const int s = find_segment(s_segs, S, i);
      if (s >= 0 && s_segs[s].z >= 0) pos = i;  // cached position: patch it
    }
    s_pos[t] = pos;
  }
  __syncthreads();
  const int items = cnt * row_units;
  for (int base = threadIdx.x; base < items; base += kPatchThreads * 4) {
    u32x4 kv[4], vv[4];
    int tk[4], un[4];
    bool ok[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = base + u * kPatchThreads;
      ok[u] = idx < items;
      tk[u] = ok[u] ? idx / row_units : 0;
      un[u] = idx - tk[u] * row_units;
      ok[u] = ok[u] && s_pos[tk[u]] >= 0;
      if (ok[u]) {
        const size_t off = (static_cast<size_t>(b) * N + s_pos[tk[u]]) * row_units;
        kv[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(k_fresh) + off + un[u]);
        vv[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(v_fresh) + off + un[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (!ok[u]) continue;
      const size_t off = (static_cast<size_t>(b) * N + s_pos[tk[u]]) * row_units;
      reinterpret_cast<u32x4*>(k_asm)[off + un[u]] = kv[u];
      reinterpret_cast<u32x4*>(v_asm)[off + un[u]] = vv[u];
    }
  }
}

}  // namespace
}  // namespace rc

namespace rc {
namespace {

// Shared by both selection entry points. eq3: score by Eq. (3) from `mass`
// with lambda and item_mask (else by the K deviation); k0/k1: budgets of the
// two classes of the top-k.
int select_impl(const rc_shape* shape, const rc_segment* segs, int32_t S, int32_t n_fresh,
                bool eq3, uint32_t item_mask, float lambda, int32_t k0, int32_t k1,
                const float* mass, const void* k_fresh, const void* v_fresh, void* k_asm,
                void* v_asm, const float* scores_in, float* scores_out, int32_t* rows,
                int32_t patch, hipStream_t stream, const char* what) {
  if (int st = check_shape(shape, false)) return st;
  const int N = shape->N, B = shape->B;
  const int ksum = k0 + k1;
  if (!segs) return fail(RC_ERR_INVALID_ARG, "segs must be non-NULL");
  if (S < 1) return fail(RC_ERR_INVALID_ARG, "S=%d must be >= 1", S);
  if (S > kMaxSegments) return fail(RC_ERR_UNSUPPORTED, "S=%d exceeds %d segments", S, kMaxSegments);
  if (N > kMaxSelectN) return fail(RC_ERR_UNSUPPORTED, "N=%d exceeds %d", N, kMaxSelectN);
  if (n_fresh < 0 || n_fresh > N) return fail(RC_ERR_INVALID_ARG, "n_fresh=%d not in [0, N]", n_fresh);
  if (k0 < 0 || k1 < 0 || ksum > N - n_fresh)
    return fail(RC_ERR_INVALID_ARG, "budgets k=%d and %d (sum) not in [0, N - n_fresh = %d]", k0, k1,
                N - n_fresh);
  if (!rows && n_fresh + ksum > 0) return fail(RC_ERR_INVALID_ARG, "rows must be non-NULL");
  if (!scores_in && !scores_out)
    return fail(RC_ERR_INVALID_ARG, "without scores_in, scores_out is required");
  if (!scores_in && (!k_fresh || !k_asm))
    return fail(RC_ERR_INVALID_ARG, "without scores_in, k_fresh and k_asm are required");
  if (eq3 && !scores_in && (!v_fresh || !v_asm || !mass))
    return fail(RC_ERR_INVALID_ARG, "without scores_in, the Eq. (3) score needs v_fresh, v_asm and mass");
  if (eq3 && !scores_in && !(lambda >= 0.f && lambda <= 1.f))
    return fail(RC_ERR_INVALID_ARG, "lambda must be in [0, 1]");
  if (patch && (!k_fresh || !v_fresh || !k_asm || !v_asm))
    return fail(RC_ERR_INVALID_ARG, "patch needs k_fresh, v_fresh, k_asm and v_asm");
  if (B > 65535) return fail(RC_ERR_UNSUPPORTED, "B=%d exceeds 65535", B);
  const int es = elem_size(shape->dtype);
  const int row_units = shape->Hkv * shape->D * es / 16;
  const int4* segs4 = reinterpret_cast<const int4*>(segs);
  const int R = n_fresh + ksum;

  const float* sc = scores_in;
  if (!scores_in) {
    const int per_wg = kDevWaves * kDevTokPerWave;
    if (eq3) {
      dim3 grid(static_cast<unsigned>((N + per_wg - 1) / per_wg), B);
      auto launch = [&](auto kern) {
        hipLaunchKernelGGL(kern, grid, dim3(64 * kDevWaves), 0, stream, segs4, S, N, shape->Hkv,
                           item_mask, lambda, mass, static_cast<const char*>(k_fresh),
                           static_cast<const char*>(v_fresh), static_cast<const char*>(k_asm),
                           static_cast<const char*>(v_asm), row_units, scores_out);
      };
      shape->dtype == RC_BF16 ? launch(eq3_score_kernel<2>) : launch(eq3_score_kernel<4>);
    } else {
      const int64_t nrows = static_cast<int64_t>(B) * N;
      dim3 grid(static_cast<unsigned>((nrows + per_wg - 1) / per_wg));
      if (shape->dtype == RC_BF16)
        hipLaunchKernelGGL(deviation_kernel<2>, grid, dim3(64 * kDevWaves), 0, stream,
                           static_cast<const char*>(k_fresh), static_cast<const char*>(k_asm), nrows,
                           row_units, scores_out);
      else
        hipLaunchKernelGGL(deviation_kernel<4>, grid, dim3(64 * kDevWaves), 0, stream,
                           static_cast<const char*>(k_fresh), static_cast<const char*>(k_asm), nrows,
                           row_units, scores_out);
    }
    if (int st = check_launch(what)) return st;
    sc = scores_out;
  } else if (scores_out && scores_out != scores_in) {
    if (hipMemcpyAsync(scores_out, scores_in, sizeof(float) * B * N, hipMemcpyDeviceToDevice, stream) !=
        hipSuccess)
      return fail(RC_ERR_HIP, "%s: copy of scores_in failed", what);
  }
  if (R > 0) {
    if (k1 > 0)
      hipLaunchKernelGGL(topk_kernel<2>, dim3(B), dim3(kTopkThreads), 0, stream, sc, segs4, S, N,
                         item_mask, k0, k1, R, rows);
    else  // class 1 takes nothing: its candidates are simply not taken
      hipLaunchKernelGGL(topk_kernel<1>, dim3(B), dim3(kTopkThreads), 0, stream, sc, segs4, S, N,
                         item_mask, k0, k1, R, rows);
    if (int st = check_launch(what)) return st;
  }
  if (patch && ksum > 0) {
    const int rows_per_wg = 4;  // many small workgroups: the selected rows are scattered
    dim3 grid((R + rows_per_wg - 1) / rows_per_wg, B);
    hipLaunchKernelGGL(patch_kernel, grid, dim3(kPatchThreads), 0, stream, segs4, S, N, rows, R,
                       rows_per_wg, row_units, static_cast<const char*>(k_fresh),
                       static_cast<const char*>(v_fresh), static_cast<char*>(k_asm),
                       static_cast<char*>(v_asm));
    if (int st = check_launch(what)) return st;
  }
  return RC_OK;
}

}  // namespace
}  // namespace rc

extern "C" int rc_select_tokens(const rc_shape* shape, const rc_segment* segs, int32_t S,
                                int32_t n_fresh, int32_t k, const void* k_fresh,
                                const void* v_fresh, void* k_asm, void* v_asm,
                                const float* scores_in, float* scores_out, int32_t* rows,
                                int32_t patch, hipStream_t stream) {
  rc::clear_error();
  return rc::select_impl(shape, segs, S, n_fresh, false, 0u, 1.f, k, 0, nullptr, k_fresh, v_fresh,
                         k_asm, v_asm, scores_in, scores_out, rows, patch, stream,
                         "rc_select_tokens");
}

extern "C" int rc_select_tokens_eq3(const rc_shape* shape, const rc_segment* segs, int32_t S,
                                    int32_t n_fresh, uint32_t item_pool_mask, float lambda,
                                    int32_t k_hist, int32_t k_item, const float* mass,
                                    const void* k_fresh, const void* v_fresh, void* k_asm,
                                    void* v_asm, const float* scores_in, float* scores_out,
                                    int32_t* rows, int32_t patch, hipStream_t stream) {
  rc::clear_error();
  if (item_pool_mask >> rc::kMaxPools)
    return rc::fail(RC_ERR_INVALID_ARG, "item_pool_mask names pools beyond %d", rc::kMaxPools);
  return rc::select_impl(shape, segs, S, n_fresh, true, item_pool_mask, lambda, k_hist, k_item,
                         mass, k_fresh, v_fresh, k_asm, v_asm, scores_in, scores_out, rows, patch,
                         stream, "rc_select_tokens_eq3");
}
