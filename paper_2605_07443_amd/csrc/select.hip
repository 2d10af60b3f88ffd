// Heavy-hitter selection and correction (RcLLM, arXiv 2605.07443,
// Sec. III-C.2b with the deviation term of Eq. (3) for M = K, lambda = 1, and
// Sec. III-C.3 step (iii)).
//
//   deviation_kernel  one wave per position: L1 distance between the fresh
//                     and the assembled key row (HBM-bound, 16-byte loads,
//                     wave reduction)
//   topk_kernel       keys held in registers: range-adaptive radix select of
//                     the k-th largest score key (11-bit digits, LDS
//                     histograms), then the fresh and selected positions
//                     written in ascending order from per-wave counts; with
//                     the patch, several workgroups per request select the
//                     same rows and each copies the fresh K/V rows of its
//                     share of the selected cached positions over the
//                     assembled ones (one wave per row)
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

constexpr int kTopkMaxPer = 16;  // positions per thread at most
constexpr int kPatchList = 2048;  // list slots of one workgroup's share of the patch
constexpr int kSelectTargetWgs = 256;  // workgroups of a patching launch: one per compute unit
constexpr int kBins = 2048;                           // 11-bit digits
constexpr int kDigitBits = 11;
constexpr int kCoarse = 64;                           // coarse bins of 32 digits
static_assert(kBins == 32 * kCoarse, "top-k bin layout");
static_assert(kMaxSelectN <= 1024 * kTopkMaxPer, "top-k positions per thread");

// Total order on fp32: larger key = larger value; +NaN above +inf.
__device__ __forceinline__ uint32_t score_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Inclusive scan over the lanes of a wave in lane order: shifts within each
// row of 16 lanes (DPP row_shr), then the row totals carried across rows.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x111, 0xf, 0xf, false));
  x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x112, 0xf, 0xf, false));
  x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x114, 0xf, 0xf, false));
  x += static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x118, 0xf, 0xf, false));
  const uint32_t r0 = __builtin_amdgcn_readlane(x, 15);
  const uint32_t r1 = __builtin_amdgcn_readlane(x, 31);
  const uint32_t r2 = __builtin_amdgcn_readlane(x, 47);
  const int row = (threadIdx.x & 63) >> 4;
  return x + (row >= 1 ? r0 : 0u) + (row >= 2 ? r1 : 0u) + (row >= 3 ? r2 : 0u);
}

// Minimum / maximum over the wave, in every lane: quad and row rotations
// (DPP), then the gfx950 row swaps across the four rows.
template <bool MAX>
__device__ __forceinline__ uint32_t wave_extreme(uint32_t x) {
  auto pick = [](uint32_t a, uint32_t b) { return MAX ? max(a, b) : min(a, b); };
  x = pick(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0xb1, 0xf, 0xf, false)));
  x = pick(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x4e, 0xf, 0xf, false)));
  x = pick(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x124, 0xf, 0xf, false)));
  x = pick(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x128, 0xf, 0xf, false)));
  const auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = pick(a[0], a[1]);
  const auto c = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return pick(c[0], c[1]);
}

// Set lanes of `mask` below this lane.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                    __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

// Workgroups (part, b) of request b. Candidates are positions outside fresh
// segments; each belongs to one of two classes: class 0 (history, or every
// cached position when item_mask is 0) and class 1 (blocks of the pools set
// in item_mask). Class c keeps its k_c largest keys, key of position i =
// score_key(score[i]), order (key desc, i asc). Fresh positions are always
// taken; the taken positions are written in ascending order. NC: number of
// classes with a budget (1: class 0 only, k1 is 0).
//
// Thread t of TPB holds positions j * TPB + t (j < NJ, TPB NJ >= N) in
// registers, so that (j, wave, lane) runs in position order; every loop over
// j is unrolled and its memory reads are issued together. The whole request
// runs on one compute unit, where vector-ALU issue is the limit: NJ follows
// N closely so that few slots are padding. (256 threads, one wave per SIMD,
// were slower: latencies are then exposed.) The k-th largest key of a class is
// found by a range-adaptive radix select: each pass histograms the keys in
// [lo, hi] on 11-bit digits (plus a 64-bin coarse histogram), one wave finds
// the boundary digit by two lane scans, and [lo, hi] narrows to it. The
// histograms rotate over three LDS buffers, so that a pass costs two
// barriers. The output is written from per-(j, wave) counts with one
// barrier: each lane's slot is the count of taken positions before it.
// Every part of a request computes the same selection; part 0 writes rows,
// and with PATCH part p copies the rows of the cached positions whose output
// slots are p, p + parts, ... (collected in an LDS list, one wave per row).
// VREF (with PATCH): v_asm is a table of 64-bit value-row addresses, one per
// position; the patch copies the key row and points the position's entry at
// its fresh value row instead of copying that row.
template <int NC, int NJ, int TPB, bool PATCH, bool VREF = false>
__global__ __launch_bounds__(TPB) void topk_kernel(
    const float* __restrict__ scores, const int4* __restrict__ segs, int S, int N,
    uint32_t item_mask, int k0, int k1, int R, int32_t* __restrict__ rows, int row_units,
    const char* __restrict__ k_fresh, const char* __restrict__ v_fresh, char* __restrict__ k_asm,
    char* __restrict__ v_asm) {
  __shared__ int4 s_segs[kMaxSegments];
  __shared__ int s_list[PATCH ? kPatchList : 1];        // this workgroup's share of the patch
  __shared__ uint32_t s_hist[3][kBins];
  __shared__ uint32_t s_coarse[3][kCoarse];
  constexpr int W = TPB / 64;                           // waves
  static_assert(!VREF || PATCH, "value references are redirected by the patch");
  static_assert(W % 4 == 0 && NJ * W <= 256 && NJ <= kTopkMaxPer, "top-k shape");
  __shared__ uint32_t s_cnt[2][NJ * W];                  // per (j, wave): taken | ties << 16; ties of class 1
  __shared__ uint32_t s_bounds[2][3];                   // per class: min key, max key, candidates
  __shared__ uint32_t s_sel[2];                         // boundary digit, keys above it

  const int b = blockIdx.y;
  const int part = blockIdx.x;   // which share of the patch (every part selects)
  const int parts = gridDim.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // scores first: their latency overlaps the segment table's
  float sc[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    sc[j] = scores[static_cast<size_t>(b) * N + min(j * TPB + tid, N - 1)];
  {
    constexpr int SP = kMaxSegments / TPB;
    int4 sv[SP];
#pragma unroll
    for (int q = 0; q < SP; ++q) sv[q] = segs[static_cast<size_t>(b) * S + min(q * TPB + tid, S - 1)];
#pragma unroll
    for (int q = 0; q < SP; ++q)
      if (q * TPB + tid < S) s_segs[q * TPB + tid] = sv[q];
  }
#pragma unroll
  for (int q = 0; q < kBins / TPB; ++q) {
    s_hist[0][q * TPB + tid] = 0u;
    s_hist[1][q * TPB + tid] = 0u;
  }
  if (tid < kCoarse) {
    s_coarse[0][tid] = 0u;
    s_coarse[1][tid] = 0u;
  }
  if constexpr (PATCH) {
    for (int q = tid; q < kPatchList; q += TPB) s_list[q] = -1;
  }
  if (tid < 2) {
    s_bounds[tid][0] = 0xffffffffu;
    s_bounds[tid][1] = 0u;
    s_bounds[tid][2] = 0u;
  }
  __syncthreads();

  // class of each position, 2 bits per j: 0 fresh, 1 + c for a candidate of
  // class c, 3 beyond N. The segment of a position is found by a binary
  // search with a uniform step count, the searches of all j side by side.
  int top = 1;  // smallest power of two >= S
  while (top < S) top <<= 1;
  int seg[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) seg[j] = 0;
  for (int step = top >> 1; step > 0; step >>= 1) {
    int x[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) x[j] = s_segs[min(seg[j] + step, S - 1)].x;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (seg[j] + step < S && x[j] <= j * TPB + tid) seg[j] += step;
  }
  int4 sg[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) sg[j] = s_segs[seg[j]];
  uint32_t key[NJ];
  uint32_t cls = 0u;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int i = j * TPB + tid;
    key[j] = i < N ? score_key(sc[j]) : 0u;
    const bool inside = sg[j].x <= i && i < sg[j].x + sg[j].y;
    const int pool = inside ? sg[j].z : -1;
    const uint32_t c = i >= N     ? 3u
                       : pool < 0 ? 0u
                                  : 1u + static_cast<uint32_t>(pool < 32 && ((item_mask >> pool) & 1u));
    cls |= c << (2 * j);
  }

  // per class: smallest and largest key, number of candidates
  {
    uint32_t kmin[2] = {0xffffffffu, 0xffffffffu}, kmax[2] = {0u, 0u};
    uint32_t ncand[2] = {0u, 0u};
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const bool is = ((cls >> (2 * j)) & 3u) == static_cast<uint32_t>(c + 1);
        if (is) {
          kmin[c] = min(kmin[c], key[j]);
          kmax[c] = max(kmax[c], key[j]);
        }
        ncand[c] += __popcll(__ballot(is));
      }
    }
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      kmin[c] = wave_extreme<false>(kmin[c]);
      kmax[c] = wave_extreme<true>(kmax[c]);
      if (lane == 0) {
        atomicMin(&s_bounds[c][0], kmin[c]);
        atomicMax(&s_bounds[c][1], kmax[c]);
        atomicAdd(&s_bounds[c][2], ncand[c]);
      }
    }
  }
  __syncthreads();

  const int kc_arg[2] = {k0, k1};
  int kk[2] = {0, 0};
  uint32_t T[2] = {0u, 0u};
  int need[2] = {0, 0};
  int pass = 0;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    if (kc_arg[c] <= 0) continue;  // uniform: kernel arguments
    kk[c] = min(kc_arg[c], static_cast<int>(s_bounds[c][2]));
    if (kk[c] == 0) continue;
    uint32_t lo = s_bounds[c][0], hi = s_bounds[c][1];
    int nd = kk[c];  // how many of the class's keys in [lo, hi] are still to take (>= 1)
    const uint32_t want = static_cast<uint32_t>(c + 1);
    while (lo != hi) {
      const uint32_t range = hi - lo;
      const int bits = 32 - __clz(range);
      const int shift = bits > kDigitBits ? bits - kDigitBits : 0;
      uint32_t* hist = s_hist[pass % 3];
      uint32_t* coarse = s_coarse[pass % 3];
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        if (((cls >> (2 * j)) & 3u) == want && key[j] >= lo && key[j] <= hi) {
          const uint32_t d = (key[j] - lo) >> shift;
          atomicAdd(&hist[d], 1u);
          atomicAdd(&coarse[d >> 5], 1u);
        }
      }
      __syncthreads();
      // the buffers of pass + 2 were last read in pass - 1, before the
      // barrier above, and are next written after the barrier below
#pragma unroll
      for (int q = 0; q < kBins / TPB; ++q) s_hist[(pass + 2) % 3][q * TPB + tid] = 0u;
      if (tid < kCoarse) s_coarse[(pass + 2) % 3][tid] = 0u;
      if (wave == 0) {
        // lane l: coarse bin 63 - l, so the lane scan counts from the top
        const uint32_t mc = coarse[kCoarse - 1 - lane];
        const uint32_t ic = wave_incl_scan(mc);
        const int lc = __builtin_ctzll(__ballot(ic >= static_cast<uint32_t>(nd) || lane == 63));
        const uint32_t above_c = __builtin_amdgcn_readlane(ic - mc, lc);
        const int cb = kCoarse - 1 - lc;
        // lanes 0..31: the digits of coarse bin cb, from its top
        const uint32_t mf = lane < 32 ? hist[cb * 32 + 31 - lane] : 0u;
        const uint32_t inf = wave_incl_scan(mf);
        const uint32_t rest = static_cast<uint32_t>(nd) - above_c;
        const int lf = __builtin_ctzll(__ballot(inf >= rest || lane == 31));
        const uint32_t above_f = __builtin_amdgcn_readlane(inf - mf, lf);
        if (lane == 0) {
          s_sel[0] = static_cast<uint32_t>(cb * 32 + 31 - lf);
          s_sel[1] = above_c + above_f;
        }
      }
      __syncthreads();
      const uint32_t bin = s_sel[0];
      nd -= static_cast<int>(s_sel[1]);
      const uint32_t nlo = lo + (bin << shift);
      const uint32_t width_m1 = (1u << shift) - 1u;  // shift <= 21
      hi = (hi - nlo > width_m1) ? nlo + width_m1 : hi;
      lo = nlo;
      ++pass;
    }
    T[c] = lo;
    need[c] = nd;  // candidates of class c with key == T_c to take, lowest positions first
  }

  // ---- emit rows: fresh positions, keys > T_c, and the first need_c ties
  // per j: taken outright (gt), tie at the threshold of class 0 / 1 (e0, e1)
  uint32_t fgt = 0u, fe0 = 0u, fe1 = 0u;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const uint32_t c = (cls >> (2 * j)) & 3u;
    const bool gt = c == 0u || (c == 1u && kk[0] > 0 && key[j] > T[0]) ||
                    (NC == 2 && c == 2u && kk[1] > 0 && key[j] > T[1]);
    const bool e0 = c == 1u && kk[0] > 0 && key[j] == T[0];
    const bool e1 = NC == 2 && c == 2u && kk[1] > 0 && key[j] == T[1];
    fgt |= static_cast<uint32_t>(gt) << j;
    fe0 |= static_cast<uint32_t>(e0) << j;
    fe1 |= static_cast<uint32_t>(e1) << j;
    const uint32_t ng = __popcll(__ballot(gt));
    const uint32_t n0 = __popcll(__ballot(e0));
    const uint32_t n1 = __popcll(__ballot(e1));
    if (lane == 0) {
      s_cnt[0][j * W + wave] = ng | (n0 << 16);
      s_cnt[1][j * W + wave] = n1;
    }
  }
  __syncthreads();
  // exclusive prefix of every (j, wave) entry in position order: lane l sums
  // entries 4l .. 4l + 3 (fields of at most N < 2^16 never carry over)
  constexpr int E = NJ * W;
  uint32_t c0[4], c1[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = 4 * lane + q;
    c0[q] = e < E ? s_cnt[0][e] : 0u;
    c1[q] = e < E ? s_cnt[1][e] : 0u;
  }
  const uint32_t l0 = c0[0] + c0[1] + c0[2] + c0[3];
  const uint32_t l1 = c1[0] + c1[1] + c1[2] + c1[3];
  const uint32_t i0 = wave_incl_scan(l0);
  const uint32_t i1 = wave_incl_scan(l1);
  const int sub = wave & 3;  // this wave's entries sit at offset sub of their lane
  uint32_t p0 = i0 - l0, p1 = i1 - l1;
#pragma unroll
  for (int q = 0; q < 3; ++q)
    if (q < sub) {
      p0 += c0[q];
      p1 += c1[q];
    }
  const uint32_t t0 = __builtin_amdgcn_readlane(i0, 63);
  const uint32_t t1 = __builtin_amdgcn_readlane(i1, 63);
  const int total = static_cast<int>((t0 & 0xffffu) + min(t0 >> 16, static_cast<uint32_t>(need[0])) +
                                     min(t1, static_cast<uint32_t>(need[1])));
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int src = j * (W / 4) + (wave >> 2);
    const uint32_t q0 = __builtin_amdgcn_readlane(p0, src);
    const uint32_t q1 = __builtin_amdgcn_readlane(p1, src);
    const uint32_t gt_before = q0 & 0xffffu, t0_before = q0 >> 16, t1_before = q1;
    const bool gt = (fgt >> j) & 1u, e0 = (fe0 >> j) & 1u, e1 = (fe1 >> j) & 1u;
    const uint32_t r0 = t0_before + lanes_below(__ballot(e0));  // tie rank in class 0
    const uint32_t r1 = t1_before + lanes_below(__ballot(e1));
    const bool take = gt || (e0 && r0 < static_cast<uint32_t>(need[0])) ||
                      (e1 && r1 < static_cast<uint32_t>(need[1]));
    const uint32_t out = gt_before + min(t0_before, static_cast<uint32_t>(need[0])) +
                         min(t1_before, static_cast<uint32_t>(need[1])) + lanes_below(__ballot(take));
    // A list longer than R (more fresh positions than n_fresh) loses its
    // tail; its last entry is then -1 so that the request is recognisable.
    if (part == 0 && take && out < static_cast<uint32_t>(R))
      rows[static_cast<size_t>(b) * R + out] =
          (total > R && out == static_cast<uint32_t>(R - 1)) ? -1 : j * TPB + tid;
    if constexpr (PATCH) {
      // selected cached positions of slots part, part + parts, ... go to this
      // workgroup's list
      const uint32_t c = (cls >> (2 * j)) & 3u;
      if (take && (c == 1u || c == 2u) && out < static_cast<uint32_t>(R) &&
          static_cast<int>(out % parts) == part)
        s_list[out / parts] = j * TPB + tid;
    }
  }
  // a list shorter than R (fewer fresh positions than n_fresh, or a budget
  // above its class's size) is padded with -1
  if (part == 0)
    for (int r = total + tid; r < R; r += TPB) rows[static_cast<size_t>(b) * R + r] = -1;

  if constexpr (PATCH && VREF) {
    // (iii) heavy-hitter update: one wave per listed position copies the
    // fresh K row over the assembled one and redirects the value entry
    __syncthreads();
    const int slots = (R + parts - 1) / parts;
    for (int sl = wave; sl < slots; sl += TPB / 64) {
      const int i = s_list[sl];
      if (i < 0) continue;
      const size_t off = (static_cast<size_t>(b) * N + i) * row_units;
      const u32x4* kf = reinterpret_cast<const u32x4*>(k_fresh) + off;
      u32x4* ka = reinterpret_cast<u32x4*>(k_asm) + off;
      if (lane == 0)
        reinterpret_cast<uint64_t*>(v_asm)[static_cast<size_t>(b) * N + i] =
            reinterpret_cast<uint64_t>(reinterpret_cast<const u32x4*>(v_fresh) + off);
      for (int u0 = 0; u0 < row_units; u0 += 128) {
        const int u1 = u0 + lane, u2 = u0 + 64 + lane;
        u32x4 ka1, ka2;
        if (u1 < row_units) ka1 = __builtin_nontemporal_load(kf + u1);
        if (u2 < row_units) ka2 = __builtin_nontemporal_load(kf + u2);
        if (u1 < row_units) ka[u1] = ka1;
        if (u2 < row_units) ka[u2] = ka2;
      }
    }
  } else if constexpr (PATCH) {
    // (iii) heavy-hitter update: one wave per listed position copies the
    // fresh K and V rows over the assembled ones (16-byte units)
    __syncthreads();
    const int slots = (R + parts - 1) / parts;
    for (int sl = wave; sl < slots; sl += TPB / 64) {
      const int i = s_list[sl];
      if (i < 0) continue;
      const size_t off = (static_cast<size_t>(b) * N + i) * row_units;
      const u32x4* kf = reinterpret_cast<const u32x4*>(k_fresh) + off;
      const u32x4* vf = reinterpret_cast<const u32x4*>(v_fresh) + off;
      u32x4* ka = reinterpret_cast<u32x4*>(k_asm) + off;
      u32x4* va = reinterpret_cast<u32x4*>(v_asm) + off;
      for (int u0 = 0; u0 < row_units; u0 += 128) {
        const int u1 = u0 + lane, u2 = u0 + 64 + lane;
        u32x4 ka1, va1, ka2, va2;
        if (u1 < row_units) {
          ka1 = __builtin_nontemporal_load(kf + u1);
          va1 = __builtin_nontemporal_load(vf + u1);
        }
        if (u2 < row_units) {
          ka2 = __builtin_nontemporal_load(kf + u2);
          va2 = __builtin_nontemporal_load(vf + u2);
        }
        if (u1 < row_units) {
          ka[u1] = ka1;
          va[u1] = va1;
        }
        if (u2 < row_units) {
          ka[u2] = ka2;
          va[u2] = va2;
        }
      }
    }
  }
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
                int32_t patch, hipStream_t stream, const char* what, bool vref = false) {
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
    return fail(RC_ERR_INVALID_ARG, "patch needs k_fresh, v_fresh, k_asm and %s",
                vref ? "v_ref" : "v_asm");
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
    // NC = 1 when class 1 takes nothing (its candidates are simply not
    // taken); NJ = positions per thread (rounded up to an even count past 8).
    // With the patch, several workgroups per request each select (the same
    // rows, deterministically) and copy their share of the selected rows, so
    // that the copy runs on many compute units; only the first writes rows.
    const bool do_patch = patch && ksum > 0;
    int parts = 1;
    if (do_patch) {
      parts = max((kSelectTargetWgs + B - 1) / B, (R + kPatchList - 1) / kPatchList);
      parts = min(parts, 64);
      if ((R + parts - 1) / parts > kPatchList) return fail(RC_ERR_UNSUPPORTED, "R=%d too large", R);
    }
    const char* kf = static_cast<const char*>(k_fresh);
    const char* vf = static_cast<const char*>(v_fresh);
    char* ka = static_cast<char*>(k_asm);
    char* va = static_cast<char*>(v_asm);
    auto launch = [&](auto kern, int tpb) {
      hipLaunchKernelGGL(kern, dim3(parts, B), dim3(tpb), 0, stream, sc, segs4, S, N, item_mask, k0,
                         k1, R, rows, row_units, kf, vf, ka, va);
    };
    auto by_chunks = [&](auto nc, auto pt, auto vr) {
      constexpr int NC = decltype(nc)::value;
      constexpr bool PT = decltype(pt)::value;
      constexpr bool VR = decltype(vr)::value && PT;
      switch ((N + 1023) / 1024) {
        case 1: launch(topk_kernel<NC, 1, 1024, PT, VR>, 1024); break;
        case 2: launch(topk_kernel<NC, 2, 1024, PT, VR>, 1024); break;
        case 3: launch(topk_kernel<NC, 3, 1024, PT, VR>, 1024); break;
        case 4: launch(topk_kernel<NC, 4, 1024, PT, VR>, 1024); break;
        case 5: launch(topk_kernel<NC, 5, 1024, PT, VR>, 1024); break;
        case 6: launch(topk_kernel<NC, 6, 1024, PT, VR>, 1024); break;
        case 7: launch(topk_kernel<NC, 7, 1024, PT, VR>, 1024); break;
        case 8: launch(topk_kernel<NC, 8, 1024, PT, VR>, 1024); break;
        case 9: case 10: launch(topk_kernel<NC, 10, 1024, PT, VR>, 1024); break;
        case 11: case 12: launch(topk_kernel<NC, 12, 1024, PT, VR>, 1024); break;
        default: launch(topk_kernel<NC, 16, 1024, PT, VR>, 1024); break;
      }
    };
    using One = std::integral_constant<int, 1>;
    using Two = std::integral_constant<int, 2>;
    auto by_patch = [&](auto nc) {
      if (!do_patch) by_chunks(nc, std::false_type{}, std::false_type{});
      else if (vref) by_chunks(nc, std::true_type{}, std::true_type{});
      else by_chunks(nc, std::true_type{}, std::false_type{});
    };
    if (k1 > 0) by_patch(Two{});
    else by_patch(One{});
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
  // item tokens are scored (1 - lambda) * mass: at lambda = 1 every item score
  // is 0 and an item budget would take the lowest positions, not a ranking
  if (!scores_in && lambda == 1.f && k_item > 0)
    return rc::fail(RC_ERR_INVALID_ARG, "lambda = 1 leaves item tokens unranked (k_item=%d > 0)", k_item);
  return rc::select_impl(shape, segs, S, n_fresh, true, item_pool_mask, lambda, k_hist, k_item,
                         mass, k_fresh, v_fresh, k_asm, v_asm, scores_in, scores_out, rows, patch,
                         stream, "rc_select_tokens_eq3");
}

extern "C" int rc_select_tokens_vref(const rc_shape* shape, const rc_segment* segs, int32_t S,
                                     int32_t n_fresh, int32_t k, const void* k_fresh,
                                     const void* v_fresh, void* k_asm, uint64_t* v_ref,
                                     const float* scores_in, float* scores_out, int32_t* rows,
                                     hipStream_t stream) {
  rc::clear_error();
  return rc::select_impl(shape, segs, S, n_fresh, false, 0u, 1.f, k, 0, nullptr, k_fresh, v_fresh,
                         k_asm, v_ref, scores_in, scores_out, rows, 1, stream,
                         "rc_select_tokens_vref", true);
}
