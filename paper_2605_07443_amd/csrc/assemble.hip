// Assembly of cached KV blocks with fused RoPE re-alignment, and the
// standalone re-alignment pass (RcLLM, arXiv 2605.07443, Sec. III-C.3 steps
// (i) and (ii); logical-to-physical block mapping of Sec. III-A).
//
// Both are HBM-bound copies. The common case (a request of at most 64
// segments, a key row of a power-of-two number of rotation pairs) runs on
// kv_gather_kernel / rerope_wave_kernel: each wave owns a few positions, finds
// each position's segment with one ballot over the request's segment table
// (one entry per lane, no LDS), issues all of its 16-byte loads and stores
// the rotated rows, without barriers. Other shapes and the token-granular
// gather run on kv_rows_kernel, where a workgroup of 256 threads owns TOK
// consecutive positions (TOK * key row = 8 KiB), resolves them through a
// segment table staged in LDS (or a per-position map) and then streams the
// rows. Source rows and assembled rows go through the caches with ordinary
// loads and stores (pool rows of popular items recur across requests and
// batches, and the attention reads the assembled rows next); the fresh key
// rows read for the score are non-temporal. A key unit pairs element block
// [j, j+E) of a head with [j+D/2, j+D/2+E) so the rotation of the pairs
// (j, j+D/2) happens in registers between the load and the store.
#include "rc_common.h"

namespace rc {
namespace {

using u32x4 = u32x4_t;

constexpr int kThreads = 256;
constexpr int kMaxTok = 64;       // positions per workgroup (8 KiB of the smallest key row, 128 B)
constexpr int kFewSegments = 64;  // segment capacity in LDS of the common instance
constexpr int kKPer = 1;                 // key pairs per thread per pass
constexpr int kVPer = 2;                 // value units per thread per pass
constexpr int kKItems = kKPer * kThreads;   // key pairs per pass
constexpr int kVItems = kVPer * kThreads;   // value units per pass
constexpr int kRowBytesPerWg = kKItems * 32;  // key-row bytes of a workgroup (8 KiB)

// ASSEMBLE: source rows come from the segment table (pool block or fresh
// row), V is copied as well, delta = dst_start for pool rows when tables are
// given. REROPE (in place): source = destination = k, delta from the array.
// SCORE (with ASSEMBLE): also reads the fresh K row of every cached position
// and writes the deviation score sum |K_fresh - K_asm| of the row it just
// produced (0 at fresh positions, whose assembled row is the fresh row).
// WRITE = false (with ASSEMBLE and SCORE): score only -- the aligned key rows
// are formed in registers and compared, nothing is stored and V is not read.
// MAP (with ASSEMBLE): sources come from a per-position map {pool, row,
// delta, -} instead of the segment table (single-token prototypes).
// Every load of a workgroup's 16-byte units is issued before the first use.
// MAXS: segments the LDS table holds (S <= MAXS); a small table keeps the
// workgroup's LDS small, so that more workgroups fit a compute unit.
template <int ES, bool ASSEMBLE, bool SCORE, bool WRITE = true, bool MAP = false,
          int MAXS = kMaxSegments>
__global__ __launch_bounds__(kThreads) void kv_rows_kernel(
    PoolArgs pools, const int4* __restrict__ segs, int S, int N, int tok_per_wg, int row_units,
    int head_units, const char* __restrict__ k_fresh, const char* __restrict__ v_fresh,
    const int32_t* __restrict__ delta_arr, const int4* __restrict__ map,
    const float* __restrict__ cos_t,
    const float* __restrict__ sin_t, int max_pos, int half, char* __restrict__ k_out,
    char* __restrict__ v_out, float* __restrict__ scores) {
  constexpr int E = 16 / ES;  // elements per 16-byte unit
  __shared__ int4 s_segs[(ASSEMBLE && !MAP) ? MAXS : 1];
  __shared__ const char* s_srck[kMaxTok];
  __shared__ const char* s_srcv[kMaxTok];
  __shared__ int s_delta[kMaxTok];
  __shared__ int s_cached[SCORE ? kMaxTok : 1];
  __shared__ float s_part[SCORE ? kKItems : 1];

  const int b = blockIdx.y;
  const size_t row_bytes = static_cast<size_t>(row_units) * 16;
  const int tid = threadIdx.x;

  if constexpr (ASSEMBLE && !MAP) {
    for (int s = tid; s < S; s += kThreads) s_segs[s] = segs[static_cast<size_t>(b) * S + s];
    __syncthreads();
  }
  // token blocks of this request; a bounded grid loops over them
  const int n_blk = (N + tok_per_wg - 1) / tok_per_wg;
  for (int blk = blockIdx.x; blk < n_blk; blk += gridDim.x) {
  const int i0 = blk * tok_per_wg;
  const int tok_cnt = min(tok_per_wg, N - i0);
  for (int t = tid; t < tok_cnt; t += kThreads) {
    const int i = i0 + t;
    const size_t row_off = (static_cast<size_t>(b) * N + i) * row_bytes;
    const char* sk = nullptr;
    const char* sv = nullptr;
    int d = 0, cached = 0;
    if constexpr (ASSEMBLE && MAP) {
      const int4 m = map[static_cast<size_t>(b) * N + i];  // {pool, row, delta, -}
      if (m.x < 0) {
        sk = k_fresh + row_off;
        sv = v_fresh + row_off;
      } else if (m.x < pools.n && m.y >= 0 &&
                 m.y < static_cast<int64_t>(pools.num_blocks[m.x]) * pools.block_len[m.x]) {
        const size_t src = static_cast<size_t>(m.y) * row_bytes;
        sk = pools.k[m.x] + src;
        sv = pools.v[m.x] + src;
        cached = 1;
        if (cos_t != nullptr && m.z < max_pos && -m.z < max_pos) d = m.z;
      }
    } else if constexpr (ASSEMBLE) {
      const int s = find_segment(s_segs, S, i);
      if (s >= 0) {
        const int4 g = s_segs[s];
        if (g.z < 0) {
          sk = k_fresh + row_off;
          sv = v_fresh + row_off;
        } else if (g.z < pools.n && g.w >= 0 && g.w < pools.num_blocks[g.z] && g.x >= 0 &&
                   i - g.x < pools.block_len[g.z]) {
          const size_t src = (static_cast<size_t>(g.w) * pools.block_len[g.z] + (i - g.x)) * row_bytes;
          sk = pools.k[g.z] + src;
          sv = pools.v[g.z] + src;
          cached = 1;
          if (cos_t != nullptr && g.x < max_pos) d = g.x;
        }
      }
    } else {
      const int dd = delta_arr[static_cast<size_t>(b) * N + i];
      if (dd != 0 && dd < max_pos && -dd < max_pos) {
        sk = k_out + row_off;
        d = dd;
      }
    }
    s_srck[t] = sk;
    s_srcv[t] = sv;
    s_delta[t] = d;
    if constexpr (SCORE) s_cached[t] = cached;
  }
  __syncthreads();

  const int pairs_per_row = row_units / 2;
  const int half_units = head_units / 2;
  const int k_items = tok_cnt * pairs_per_row;
  const int v_items = (ASSEMBLE && WRITE) ? tok_cnt * row_units : 0;
  for (int it = 0; it * kKItems < k_items || it * kVItems < v_items; ++it) {
    // ---- issue every load: key pairs (+ fresh key pairs), value units
    u32x4 ua[kKPer], ub[kKPer], fa[kKPer], fb[kKPer], vv[kVPer];
    int ktok[kKPer], kunit[kKPer], vtok[kVPer], vunit[kVPer];
    bool kok[kKPer], fok[kKPer], vok[kVPer];
#pragma unroll
    for (int u = 0; u < kKPer; ++u) {
      const int idx = it * kKItems + u * kThreads + tid;
      kok[u] = idx < k_items;
      ktok[u] = kok[u] ? idx / pairs_per_row : 0;
      const int pr = idx - ktok[u] * pairs_per_row;
      const int head = pr / half_units;
      kunit[u] = head * head_units + (pr - head * half_units);
      kok[u] = kok[u] && s_srck[ktok[u]] != nullptr;
      fok[u] = false;
      if (kok[u]) {
        const u32x4* src = reinterpret_cast<const u32x4*>(s_srck[ktok[u]]);
        if constexpr (ASSEMBLE) {
          ua[u] = src[kunit[u]];
          ub[u] = src[kunit[u] + half_units];
        } else {
          ua[u] = src[kunit[u]];
          ub[u] = src[kunit[u] + half_units];
        }
        if constexpr (SCORE) {
          fok[u] = s_cached[ktok[u]] != 0;
          if (fok[u]) {
            const u32x4* fr = reinterpret_cast<const u32x4*>(
                k_fresh + (static_cast<size_t>(b) * N + i0 + ktok[u]) * row_bytes);
            fa[u] = __builtin_nontemporal_load(fr + kunit[u]);
            fb[u] = __builtin_nontemporal_load(fr + kunit[u] + half_units);
          }
        }
      }
    }
    if constexpr (ASSEMBLE && WRITE) {
#pragma unroll
      for (int u = 0; u < kVPer; ++u) {
        const int idx = it * kVItems + u * kThreads + tid;
        vok[u] = idx < v_items;
        vtok[u] = vok[u] ? idx / row_units : 0;
        vunit[u] = idx - vtok[u] * row_units;
        vok[u] = vok[u] && s_srcv[vtok[u]] != nullptr;
        if (vok[u]) vv[u] = reinterpret_cast<const u32x4*>(s_srcv[vtok[u]])[vunit[u]];
      }
    }

    // ---- keys: rotate, store, deviation partials
#pragma unroll
    for (int u = 0; u < kKPer; ++u) {
      if (kok[u]) {
        const int d = s_delta[ktok[u]];
        if (d != 0) {
          const int a = d < 0 ? -d : d;
          const int j0 = (kunit[u] % head_units) * E;  // element offset in the half
          float c[E], sn[E];
#pragma unroll
          for (int e = 0; e < E; ++e) {
            c[e] = cos_t[static_cast<size_t>(a) * half + j0 + e];
            const float sv = sin_t[static_cast<size_t>(a) * half + j0 + e];
            sn[e] = d < 0 ? -sv : sv;
          }
          rotate_unit<ES>(ua[u], ub[u], c, sn);
        }
        if constexpr (WRITE) {
          u32x4* dst = reinterpret_cast<u32x4*>(k_out + (static_cast<size_t>(b) * N + i0 + ktok[u]) * row_bytes);
          if constexpr (ASSEMBLE) {
            dst[kunit[u]] = ua[u];
            dst[kunit[u] + half_units] = ub[u];
          } else {
            dst[kunit[u]] = ua[u];
            dst[kunit[u] + half_units] = ub[u];
          }
        }
      }
      if constexpr (SCORE) {
        const int idx = u * kThreads + tid;  // scoring runs a single key pass (it == 0)
        if (it == 0 && idx < k_items)
          s_part[idx] = fok[u] ? absdiff_sum<ES>(fa[u], ua[u]) + absdiff_sum<ES>(fb[u], ub[u]) : 0.f;
      }
    }
    if constexpr (ASSEMBLE && WRITE) {
#pragma unroll
      for (int u = 0; u < kVPer; ++u) {
        if (!vok[u]) continue;
        u32x4* dst = reinterpret_cast<u32x4*>(v_out + (static_cast<size_t>(b) * N + i0 + vtok[u]) * row_bytes);
        dst[vunit[u]] = vv[u];
      }
    }
  }

  if constexpr (SCORE) {
    // one wave per position: fixed-order sum of its key-pair partials
    __syncthreads();
    const int lane = tid & 63;
    for (int t = tid >> 6; t < tok_cnt; t += kThreads / 64) {
      float x = 0.f;
      for (int j = lane; j < pairs_per_row; j += 64) x += s_part[t * pairs_per_row + j];
      x = wave_sum(x);
      if (lane == 0) scores[static_cast<size_t>(b) * N + i0 + t] = x;
    }
  }
  __syncthreads();  // the next block reuses the workgroup's LDS
  }
}

// Wave-level gather for requests of at most 64 segments whose key row has a
// power-of-two number of pairs ppr dividing 64 * KP (every workload shape
// here): no LDS and no barrier. Wave w of workgroup x owns the T = 64 KP /
// ppr positions starting at (4 x + w) T of request blockIdx.y. The request's
// segment table is held one entry per lane; a position's segment is the
// lane whose range holds it (one ballot). Lane l carries key pairs
// k * 64 + l (k < KP: position (k * 64 + l) / ppr, pair (k * 64 + l) % ppr)
// and value units k * 64 + l (k < 2 KP) of those T positions; every load is
// issued before the first use. The deviation of a position is the sum of its
// pairs' partials in a fixed order (shuffles within the lanes of one
// position when ppr < 64, then a wave sum), so the score is deterministic.
// VREF (with WRITE): value rows are not copied; v_out is then a table of one
// 64-bit address per position, that of the row the copy would have read (the
// pool row of a cached position, else the fresh row), lane t of the wave
// writing the entry of its position t (T <= 64 with KP = 1).
template <int ES, bool SCORE, bool WRITE, int KP, bool VREF = false>
__global__ __launch_bounds__(kThreads) void kv_gather_kernel(
    PoolArgs pools, const int4* __restrict__ segs, int S, int N, int row_units, int head_units,
    int log2_ppr, const char* __restrict__ k_fresh, const char* __restrict__ v_fresh,
    const float* __restrict__ cos_t, const float* __restrict__ sin_t, int max_pos, int half,
    char* __restrict__ k_out, char* __restrict__ v_out, float* __restrict__ scores) {
  constexpr int E = 16 / ES;     // elements per 16-byte unit
  constexpr int VP = 2 * KP;     // value units per lane
  static_assert(!VREF || (WRITE && KP == 1), "value references need the writing instance, KP = 1");
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ppr = 1 << log2_ppr;
  const int T = (64 * KP) >> log2_ppr;                   // positions of this wave
  const int i0 = (blockIdx.x * (kThreads / 64) + wave) * T;
  if (i0 >= N) return;
  const size_t row_bytes = static_cast<size_t>(row_units) * 16;
  const int half_units = head_units / 2;

  const int4 sg = lane < S ? segs[static_cast<size_t>(b) * S + lane] : int4{0x7fffffff, 0, -1, 0};

  // per-lane slots: the position of each key pair and value unit
  int kt[KP], vt[VP];
#pragma unroll
  for (int k = 0; k < KP; ++k) kt[k] = (k * 64 + lane) >> log2_ppr;
#pragma unroll
  for (int k = 0; k < VP; ++k) vt[k] = (k * 64 + lane) / row_units;
  const char* ksrc[KP] = {};
  const char* vsrc[VP] = {};
  int kd[KP] = {};
  bool kc[KP] = {};
  uint64_t vref_own = 0;  // VREF: address of the value row of position lane
  // resolve the wave's positions one at a time (uniform values)
  for (int t = 0; t < T; ++t) {
    const int i = i0 + t;
    if (i >= N) break;
    const uint64_t m = __ballot(sg.x <= i && i - sg.x < sg.y);
    const char* sk = nullptr;
    const char* sv = nullptr;
    int d = 0;
    bool cached = false;
    if (m != 0) {
      const int sl = __builtin_ctzll(m);
      const int gx = __builtin_amdgcn_readlane(sg.x, sl);
      const int gp = __builtin_amdgcn_readlane(sg.z, sl);
      const int gb = __builtin_amdgcn_readlane(sg.w, sl);
      if (gp < 0) {
        const size_t off = (static_cast<size_t>(b) * N + i) * row_bytes;
        sk = k_fresh + off;
        sv = v_fresh + off;
      } else if (gp < pools.n && gb >= 0 && gb < pools.num_blocks[gp] && gx >= 0 &&
                 i - gx < pools.block_len[gp]) {
        const size_t off = (static_cast<size_t>(gb) * pools.block_len[gp] + (i - gx)) * row_bytes;
        sk = pools.k[gp] + off;
        sv = pools.v[gp] + off;
        cached = true;
        if (cos_t != nullptr && gx < max_pos) d = gx;
      }
    }
#pragma unroll
    for (int k = 0; k < KP; ++k)
      if (kt[k] == t) {
        ksrc[k] = sk;
        kd[k] = d;
        kc[k] = cached;
      }
    if constexpr (VREF) {
      const char* va = sv != nullptr ? sv : v_fresh + (static_cast<size_t>(b) * N + i) * row_bytes;
      if (lane == t) vref_own = reinterpret_cast<uint64_t>(va);
    } else {
#pragma unroll
      for (int k = 0; k < VP; ++k)
        if (vt[k] == t) vsrc[k] = sv;
    }
  }
  if constexpr (VREF) {
    if (lane < T && i0 + lane < N)
      reinterpret_cast<uint64_t*>(v_out)[static_cast<size_t>(b) * N + i0 + lane] = vref_own;
  }

  // ---- issue every load
  u32x4 ua[KP], ub[KP], fa[KP], fb[KP], vv[VP];
  int kunit[KP];
#pragma unroll
  for (int k = 0; k < KP; ++k) {
    const int pr = (k * 64 + lane) & (ppr - 1);
    const int head = pr / half_units;
    kunit[k] = head * head_units + (pr - head * half_units);
    if (ksrc[k] != nullptr) {
      const u32x4* src = reinterpret_cast<const u32x4*>(ksrc[k]);
      ua[k] = src[kunit[k]];
      ub[k] = src[kunit[k] + half_units];
      if (SCORE && kc[k]) {
        const u32x4* fr = reinterpret_cast<const u32x4*>(
            k_fresh + (static_cast<size_t>(b) * N + i0 + kt[k]) * row_bytes);
        fa[k] = __builtin_nontemporal_load(fr + kunit[k]);
        fb[k] = __builtin_nontemporal_load(fr + kunit[k] + half_units);
      }
    }
  }
  if constexpr (WRITE && !VREF) {
#pragma unroll
    for (int k = 0; k < VP; ++k)
      if (vsrc[k] != nullptr) vv[k] = reinterpret_cast<const u32x4*>(vsrc[k])[(k * 64 + lane) % row_units];
  }

  // ---- keys: rotate, store, deviation partials
  float part[KP];
#pragma unroll
  for (int k = 0; k < KP; ++k) {
    part[k] = 0.f;
    if (ksrc[k] == nullptr) continue;
    if (kd[k] != 0) {
      const int j0 = (kunit[k] % head_units) * E;   // element offset in the half
      float c[E], sn[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        c[e] = cos_t[static_cast<size_t>(kd[k]) * half + j0 + e];
        sn[e] = sin_t[static_cast<size_t>(kd[k]) * half + j0 + e];
      }
      rotate_unit<ES>(ua[k], ub[k], c, sn);
    }
    if constexpr (WRITE) {
      u32x4* dst = reinterpret_cast<u32x4*>(k_out + (static_cast<size_t>(b) * N + i0 + kt[k]) * row_bytes);
      dst[kunit[k]] = ua[k];
      dst[kunit[k] + half_units] = ub[k];
    }
    if (SCORE && kc[k]) part[k] = absdiff_sum<ES>(fa[k], ua[k]) + absdiff_sum<ES>(fb[k], ub[k]);
  }
  if constexpr (WRITE && !VREF) {
#pragma unroll
    for (int k = 0; k < VP; ++k) {
      if (vsrc[k] == nullptr) continue;
      u32x4* dst = reinterpret_cast<u32x4*>(v_out + (static_cast<size_t>(b) * N + i0 + vt[k]) * row_bytes);
      dst[(k * 64 + lane) % row_units] = vv[k];
    }
  }

  if constexpr (SCORE) {
    if (ppr >= 64) {
      // position t holds the slots k with (k * 64) >> log2_ppr == t: ppr / 64 of them
      const int per = ppr >> 6;
      for (int t = 0; t < T; ++t) {
        float x = 0.f;
#pragma unroll
        for (int k = 0; k < KP; ++k)
          if (k / per == t) x += part[k];
        x = wave_sum(x);
        if (lane == 0 && i0 + t < N) scores[static_cast<size_t>(b) * N + i0 + t] = x;
      }
    } else {
      // each slot k: positions of ppr consecutive lanes; sum within them
#pragma unroll
      for (int k = 0; k < KP; ++k) {
        float x = part[k];
        for (int off = ppr >> 1; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
        if ((lane & (ppr - 1)) == 0 && i0 + kt[k] < N)
          scores[static_cast<size_t>(b) * N + i0 + kt[k]] = x;
      }
    }
  }
}

// Standalone re-alignment with the wave-level layout of kv_gather_kernel: the
// T positions of wave w of workgroup x are rotated in place, each by its own
// delta (rows with delta 0 or |delta| >= max_pos are not touched).
template <int ES, int KP>
__global__ __launch_bounds__(kThreads) void rerope_wave_kernel(
    int N, int row_units, int head_units, int log2_ppr, const int32_t* __restrict__ delta,
    const float* __restrict__ cos_t, const float* __restrict__ sin_t, int max_pos, int half,
    char* __restrict__ k) {
  constexpr int E = 16 / ES;
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ppr = 1 << log2_ppr;
  const int T = (64 * KP) >> log2_ppr;
  const int i0 = (blockIdx.x * (kThreads / 64) + wave) * T;
  if (i0 >= N) return;
  const size_t row_bytes = static_cast<size_t>(row_units) * 16;
  const int half_units = head_units / 2;
  u32x4 ua[KP], ub[KP];
  int kd[KP], kunit[KP], kt[KP];
#pragma unroll
  for (int q = 0; q < KP; ++q) {
    kt[q] = (q * 64 + lane) >> log2_ppr;
    const int i = i0 + kt[q];
    const int pr = (q * 64 + lane) & (ppr - 1);
    const int head = pr / half_units;
    kunit[q] = head * head_units + (pr - head * half_units);
    const int d = i < N ? delta[static_cast<size_t>(b) * N + i] : 0;
    kd[q] = (d != 0 && d < max_pos && -d < max_pos) ? d : 0;
    if (kd[q] != 0) {
      const u32x4* src = reinterpret_cast<const u32x4*>(k + (static_cast<size_t>(b) * N + i) * row_bytes);
      ua[q] = src[kunit[q]];
      ub[q] = src[kunit[q] + half_units];
    }
  }
#pragma unroll
  for (int q = 0; q < KP; ++q) {
    if (kd[q] == 0) continue;
    const int a = kd[q] < 0 ? -kd[q] : kd[q];
    const int j0 = (kunit[q] % head_units) * E;
    float c[E], sn[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      c[e] = cos_t[static_cast<size_t>(a) * half + j0 + e];
      const float sv = sin_t[static_cast<size_t>(a) * half + j0 + e];
      sn[e] = kd[q] < 0 ? -sv : sv;
    }
    rotate_unit<ES>(ua[q], ub[q], c, sn);
    u32x4* dst = reinterpret_cast<u32x4*>(k + (static_cast<size_t>(b) * N + i0 + kt[q]) * row_bytes);
    dst[kunit[q]] = ua[q];
    dst[kunit[q] + half_units] = ub[q];
  }
}

int tokens_per_wg(int row_bytes) {
  int t = kRowBytesPerWg / row_bytes;
  return t < 1 ? 1 : (t > kMaxTok ? kMaxTok : t);
}

constexpr int kWaveGatherKP = 1;  // key pairs per lane of the wave-level gather

// The wave-level gather serves requests of at most 64 segments whose key row
// has a power-of-two pair count dividing 64 * KP.
bool wave_gather_ok(const rc_shape& s, int S, int row_units) {
  const int ppr = row_units / 2;
  return S <= 64 && ppr >= 1 && (ppr & (ppr - 1)) == 0 && ppr <= 64 * kWaveGatherKP;
}

template <bool ASSEMBLE, bool MAP = false>
int launch_rows(const rc_shape* s, const PoolArgs& pools, const int4* segs, int S,
                const void* k_fresh, const void* v_fresh, const int32_t* delta, const float* cos_t,
                const float* sin_t, int max_pos, void* k_out, void* v_out, float* scores,
                hipStream_t stream, const int4* map = nullptr, int max_wgs = 0,
                bool vref = false) {
  const int es = elem_size(s->dtype);
  const int row_bytes = s->Hkv * s->D * es;
  const int row_units = row_bytes / 16;
  const int head_units = s->D * es / 16;
  const int tok = tokens_per_wg(row_bytes);
  if (scores && tok * (row_units / 2) > kKItems)
    return fail(RC_ERR_UNSUPPORTED, "scoring needs a key row of at most %d bytes", kRowBytesPerWg);
  dim3 grid((s->N + tok - 1) / tok, s->B);
  if (max_wgs > 0) {  // bounded grid: each workgroup loops over token blocks
    const int gx = max(1, max_wgs / s->B);
    grid.x = min(grid.x, static_cast<unsigned>(gx));
  }
  if (grid.y > 65535) return fail(RC_ERR_UNSUPPORTED, "B=%d exceeds 65535", s->B);
  auto args = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, dim3(kThreads), 0, stream, pools, segs, S, s->N, tok, row_units,
                       head_units, static_cast<const char*>(k_fresh),
                       static_cast<const char*>(v_fresh), delta, map, cos_t, sin_t, max_pos, s->D / 2,
                       static_cast<char*>(k_out), static_cast<char*>(v_out), scores);
  };
  if (!ASSEMBLE && wave_gather_ok(*s, 1, row_units)) {
    int log2_ppr = 0;
    while ((1 << log2_ppr) < row_units / 2) ++log2_ppr;
    const int T = (64 * kWaveGatherKP) >> log2_ppr;
    dim3 g2((s->N + (kThreads / 64) * T - 1) / ((kThreads / 64) * T), s->B);
    auto args2 = [&](auto kern) {
      hipLaunchKernelGGL(kern, g2, dim3(kThreads), 0, stream, s->N, row_units, head_units, log2_ppr,
                         delta, cos_t, sin_t, max_pos, s->D / 2, static_cast<char*>(k_out));
    };
    if (s->dtype == RC_BF16) args2(rerope_wave_kernel<2, kWaveGatherKP>);
    else args2(rerope_wave_kernel<4, kWaveGatherKP>);
  } else if (!ASSEMBLE) {
    if (s->dtype == RC_BF16) args(kv_rows_kernel<2, false, false>);
    else args(kv_rows_kernel<4, false, false>);
  } else if (MAP) {
    if (scores) {
      if (s->dtype == RC_BF16) args(kv_rows_kernel<2, true, true, true, true>);
      else args(kv_rows_kernel<4, true, true, true, true>);
    } else {
      if (s->dtype == RC_BF16) args(kv_rows_kernel<2, true, false, true, true>);
      else args(kv_rows_kernel<4, true, false, true, true>);
    }
  } else if (wave_gather_ok(*s, S, row_units)) {
    int log2_ppr = 0;
    while ((1 << log2_ppr) < row_units / 2) ++log2_ppr;
    const int T = (64 * kWaveGatherKP) >> log2_ppr;
    dim3 g2((s->N + (kThreads / 64) * T - 1) / ((kThreads / 64) * T), s->B);
    auto args2 = [&](auto kern) {
      hipLaunchKernelGGL(kern, g2, dim3(kThreads), 0, stream, pools, segs, S, s->N, row_units,
                         head_units, log2_ppr, static_cast<const char*>(k_fresh),
                         static_cast<const char*>(v_fresh), cos_t, sin_t, max_pos, s->D / 2,
                         static_cast<char*>(k_out), static_cast<char*>(v_out), scores);
    };
    constexpr int KP = kWaveGatherKP;
    if (vref && scores) {
      if (s->dtype == RC_BF16) args2(kv_gather_kernel<2, true, true, KP, true>);
      else args2(kv_gather_kernel<4, true, true, KP, true>);
    } else if (vref) {
      if (s->dtype == RC_BF16) args2(kv_gather_kernel<2, false, true, KP, true>);
      else args2(kv_gather_kernel<4, false, true, KP, true>);
    } else if (scores && !k_out) {
      if (s->dtype == RC_BF16) args2(kv_gather_kernel<2, true, false, KP>);
      else args2(kv_gather_kernel<4, true, false, KP>);
    } else if (scores) {
      if (s->dtype == RC_BF16) args2(kv_gather_kernel<2, true, true, KP>);
      else args2(kv_gather_kernel<4, true, true, KP>);
    } else {
      if (s->dtype == RC_BF16) args2(kv_gather_kernel<2, false, true, KP>);
      else args2(kv_gather_kernel<4, false, true, KP>);
    }
  } else {
    auto seg_table = [&](auto few) {
      constexpr int MS = decltype(few)::value ? kFewSegments : kMaxSegments;
      if (scores && !k_out) {
        if (s->dtype == RC_BF16) args(kv_rows_kernel<2, true, true, false, false, MS>);
        else args(kv_rows_kernel<4, true, true, false, false, MS>);
      } else if (scores) {
        if (s->dtype == RC_BF16) args(kv_rows_kernel<2, true, true, true, false, MS>);
        else args(kv_rows_kernel<4, true, true, true, false, MS>);
      } else {
        if (s->dtype == RC_BF16) args(kv_rows_kernel<2, true, false, true, false, MS>);
        else args(kv_rows_kernel<4, true, false, true, false, MS>);
      }
    };
    if (S <= kFewSegments) seg_table(std::true_type{});
    else seg_table(std::false_type{});
  }
  return check_launch(MAP ? "rc_kv_gather_tokens" : vref ? "rc_kv_assemble_vref"
                      : ASSEMBLE ? "rc_kv_assemble" : "rc_rerope");
}

}  // namespace
}  // namespace rc

namespace rc {
namespace {

// Checks and launch shared by rc_kv_assemble and rc_kv_assemble_vref (v_out:
// the assembled value rows, or with vref the table of value-row addresses).
int assemble_entry(const rc_shape* shape, const rc_pool* pools, int32_t n_pools,
                   const rc_segment* segs, int32_t S, const void* k_fresh, const void* v_fresh,
                   const float* rope_cos, const float* rope_sin, int32_t max_pos, void* k_asm,
                   void* v_out, float* scores_out, hipStream_t stream, bool vref) {
  const char* what = vref ? "v_ref" : "v_asm";
  if (int st = check_shape(shape, false)) return st;
  if (n_pools < 1 || n_pools > kMaxPools)
    return fail(n_pools > kMaxPools ? RC_ERR_UNSUPPORTED : RC_ERR_INVALID_ARG,
                "n_pools=%d (1..%d)", n_pools, kMaxPools);
  if (!pools) return fail(RC_ERR_INVALID_ARG, "pools is NULL");
  if (!segs || !k_fresh || !v_fresh)
    return fail(RC_ERR_INVALID_ARG, "segs, k_fresh and v_fresh must be non-NULL");
  if (vref && (!k_asm || !v_out))
    return fail(RC_ERR_INVALID_ARG, "k_asm and v_ref must be non-NULL");
  if ((k_asm == nullptr) != (v_out == nullptr))
    return fail(RC_ERR_INVALID_ARG, "k_asm and %s must both be given or both be NULL", what);
  if (!k_asm && !scores_out)
    return fail(RC_ERR_INVALID_ARG, "without k_asm/v_asm (score only) scores_out is required");
  if (S < 1) return fail(RC_ERR_INVALID_ARG, "S=%d must be >= 1", S);
  if (S > kMaxSegments) return fail(RC_ERR_UNSUPPORTED, "S=%d exceeds %d segments", S, kMaxSegments);
  if ((rope_cos == nullptr) != (rope_sin == nullptr))
    return fail(RC_ERR_INVALID_ARG, "rope_cos and rope_sin must both be given or both be NULL");
  if (rope_cos && max_pos < shape->N)
    return fail(RC_ERR_INVALID_ARG, "max_pos=%d < N=%d", max_pos, shape->N);
  if (k_asm && (k_asm == k_fresh || v_out == v_fresh || k_asm == v_out))
    return fail(RC_ERR_INVALID_ARG, "outputs alias inputs");
  if (vref) {
    const int row_units = shape->Hkv * shape->D * elem_size(shape->dtype) / 16;
    if (!wave_gather_ok(*shape, S, row_units))
      return fail(RC_ERR_UNSUPPORTED,
                  "value references need S <= 64 and a key row of a power-of-two number of "
                  "32-byte pairs, at most 64 (S=%d, row of %d bytes)", S, row_units * 16);
  }
  PoolArgs pa{};
  pa.n = n_pools;
  for (int p = 0; p < n_pools; ++p) {
    if (!pools[p].k || !pools[p].v || pools[p].num_blocks < 1 || pools[p].block_len < 1)
      return fail(RC_ERR_INVALID_ARG, "pool %d: NULL tensor or empty shape", p);
    pa.k[p] = static_cast<const char*>(pools[p].k);
    pa.v[p] = static_cast<const char*>(pools[p].v);
    pa.num_blocks[p] = pools[p].num_blocks;
    pa.block_len[p] = pools[p].block_len;
  }
  return launch_rows<true>(shape, pa, reinterpret_cast<const int4*>(segs), S, k_fresh, v_fresh,
                           nullptr, rope_cos, rope_sin, rope_cos ? max_pos : 0, k_asm, v_out,
                           scores_out, stream, nullptr, 0, vref);
}

}  // namespace
}  // namespace rc

extern "C" int rc_kv_assemble(const rc_shape* shape, const rc_pool* pools, int32_t n_pools,
                              const rc_segment* segs, int32_t S, const void* k_fresh,
                              const void* v_fresh, const float* rope_cos, const float* rope_sin,
                              int32_t max_pos, void* k_asm, void* v_asm, float* scores_out,
                              hipStream_t stream) {
  rc::clear_error();
  return rc::assemble_entry(shape, pools, n_pools, segs, S, k_fresh, v_fresh, rope_cos, rope_sin,
                            max_pos, k_asm, v_asm, scores_out, stream, false);
}

extern "C" int rc_kv_assemble_vref(const rc_shape* shape, const rc_pool* pools, int32_t n_pools,
                                   const rc_segment* segs, int32_t S, const void* k_fresh,
                                   const void* v_fresh, const float* rope_cos,
                                   const float* rope_sin, int32_t max_pos, void* k_asm,
                                   uint64_t* v_ref, float* scores_out, hipStream_t stream) {
  rc::clear_error();
  return rc::assemble_entry(shape, pools, n_pools, segs, S, k_fresh, v_fresh, rope_cos, rope_sin,
                            max_pos, k_asm, v_ref, scores_out, stream, true);
}

extern "C" int rc_rerope(const rc_shape* shape, void* k, const int32_t* delta,
                         const float* rope_cos, const float* rope_sin, int32_t max_pos,
                         hipStream_t stream) {
  using namespace rc;
  clear_error();
  if (int st = check_shape(shape, false)) return st;
  if (!k || !delta || !rope_cos || !rope_sin)
    return fail(RC_ERR_INVALID_ARG, "k, delta, rope_cos and rope_sin must be non-NULL");
  if (max_pos < 1) return fail(RC_ERR_INVALID_ARG, "max_pos=%d must be >= 1", max_pos);
  PoolArgs pa{};
  return launch_rows<false>(shape, pa, nullptr, 0, nullptr, nullptr, delta, rope_cos, rope_sin,
                            max_pos, k, nullptr, nullptr, stream);
}

extern "C" int rc_kv_gather_tokens(const rc_shape* shape, const rc_pool* pools, int32_t n_pools,
                                   const rc_token_src* map, const void* k_fresh,
                                   const void* v_fresh, const float* rope_cos,
                                   const float* rope_sin, int32_t max_pos, void* k_asm,
                                   void* v_asm, float* scores_out, int32_t max_workgroups,
                                   hipStream_t stream) {
  using namespace rc;
  clear_error();
  if (int st = check_shape(shape, false)) return st;
  if (n_pools < 1 || n_pools > kMaxPools)
    return fail(n_pools > kMaxPools ? RC_ERR_UNSUPPORTED : RC_ERR_INVALID_ARG,
                "n_pools=%d (1..%d)", n_pools, kMaxPools);
  if (!pools || !map || !k_fresh || !v_fresh || !k_asm || !v_asm)
    return fail(RC_ERR_INVALID_ARG, "pools, map, k_fresh, v_fresh, k_asm and v_asm must be non-NULL");
  if ((rope_cos == nullptr) != (rope_sin == nullptr))
    return fail(RC_ERR_INVALID_ARG, "rope_cos and rope_sin must both be given or both be NULL");
  if (rope_cos && max_pos < 1) return fail(RC_ERR_INVALID_ARG, "max_pos=%d must be >= 1", max_pos);
  if (k_asm == k_fresh || v_asm == v_fresh || k_asm == v_asm)
    return fail(RC_ERR_INVALID_ARG, "outputs alias inputs");
  if (max_workgroups < 0) return fail(RC_ERR_INVALID_ARG, "max_workgroups=%d must be >= 0", max_workgroups);
  PoolArgs pa{};
  pa.n = n_pools;
  for (int p = 0; p < n_pools; ++p) {
    if (!pools[p].k || !pools[p].v || pools[p].num_blocks < 1 || pools[p].block_len < 1)
      return fail(RC_ERR_INVALID_ARG, "pool %d: NULL tensor or empty shape", p);
    pa.k[p] = static_cast<const char*>(pools[p].k);
    pa.v[p] = static_cast<const char*>(pools[p].v);
    pa.num_blocks[p] = pools[p].num_blocks;
    pa.block_len[p] = pools[p].block_len;
  }
  return launch_rows<true, true>(shape, pa, nullptr, 0, k_fresh, v_fresh, nullptr, rope_cos,
                                 rope_sin, rope_cos ? max_pos : 0, k_asm, v_asm, scores_out, stream,
                                 reinterpret_cast<const int4*>(map), max_workgroups);
}
