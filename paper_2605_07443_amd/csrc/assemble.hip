// Assembly of cached KV blocks with fused RoPE re-alignment, and the
// standalone re-alignment pass (RcLLM, arXiv 2605.07443, Sec. III-C.3 steps
// (i) and (ii); logical-to-physical block mapping of Sec. III-A).
//
// Both are HBM-bound copies. A workgroup of 256 threads owns TOK consecutive
// positions of one request (TOK * key row = 8 KiB): it first
// resolves each position to its source row (binary search of the request's
// segment table staged in LDS), then streams 16-byte units. Source rows and
// the assembled rows go through the caches with ordinary loads and stores
// (pool rows of popular items recur across requests and batches, and the
// attention reads the assembled rows next); the fresh key rows read for the
// score are non-temporal. A key unit pairs
// element block [j, j+E) of a head with [j+D/2, j+D/2+E) so the rotation of
// the pairs (j, j+D/2) happens in registers between the load and the store.
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

int tokens_per_wg(int row_bytes) {
  int t = kRowBytesPerWg / row_bytes;
  return t < 1 ? 1 : (t > kMaxTok ? kMaxTok : t);
}

template <bool ASSEMBLE, bool MAP = false>
int launch_rows(const rc_shape* s, const PoolArgs& pools, const int4* segs, int S,
                const void* k_fresh, const void* v_fresh, const int32_t* delta, const float* cos_t,
                const float* sin_t, int max_pos, void* k_out, void* v_out, float* scores,
                hipStream_t stream, const int4* map = nullptr, int max_wgs = 0) {
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
  if (!ASSEMBLE) {
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
  return check_launch(MAP ? "rc_kv_gather_tokens" : ASSEMBLE ? "rc_kv_assemble" : "rc_rerope");
}

}  // namespace
}  // namespace rc

extern "C" int rc_kv_assemble(const rc_shape* shape, const rc_pool* pools, int32_t n_pools,
                              const rc_segment* segs, int32_t S, const void* k_fresh,
                              const void* v_fresh, const float* rope_cos, const float* rope_sin,
                              int32_t max_pos, void* k_asm, void* v_asm, float* scores_out,
                              hipStream_t stream) {
  using namespace rc;
  clear_error();
  if (int st = check_shape(shape, false)) return st;
  if (n_pools < 1 || n_pools > kMaxPools)
    return fail(n_pools > kMaxPools ? RC_ERR_UNSUPPORTED : RC_ERR_INVALID_ARG,
                "n_pools=%d (1..%d)", n_pools, kMaxPools);
  if (!pools) return fail(RC_ERR_INVALID_ARG, "pools is NULL");
  if (!segs || !k_fresh || !v_fresh)
    return fail(RC_ERR_INVALID_ARG, "segs, k_fresh and v_fresh must be non-NULL");
  if ((k_asm == nullptr) != (v_asm == nullptr))
    return fail(RC_ERR_INVALID_ARG, "k_asm and v_asm must both be given or both be NULL");
  if (!k_asm && !scores_out)
    return fail(RC_ERR_INVALID_ARG, "without k_asm/v_asm (score only) scores_out is required");
  if (S < 1) return fail(RC_ERR_INVALID_ARG, "S=%d must be >= 1", S);
  if (S > kMaxSegments) return fail(RC_ERR_UNSUPPORTED, "S=%d exceeds %d segments", S, kMaxSegments);
  if ((rope_cos == nullptr) != (rope_sin == nullptr))
    return fail(RC_ERR_INVALID_ARG, "rope_cos and rope_sin must both be given or both be NULL");
  if (rope_cos && max_pos < shape->N)
    return fail(RC_ERR_INVALID_ARG, "max_pos=%d < N=%d", max_pos, shape->N);
  if (k_asm && (k_asm == k_fresh || v_asm == v_fresh || k_asm == v_asm))
    return fail(RC_ERR_INVALID_ARG, "outputs alias inputs");
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
                           nullptr, rope_cos, rope_sin, rope_cos ? max_pos : 0, k_asm, v_asm,
                           scores_out, stream);
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
