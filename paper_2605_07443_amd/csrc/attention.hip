// Selective causal attention (RcLLM, arXiv 2605.07443, Sec. III-C.2b: exact
// attention recomputed for the selected rows over the full assembled context;
// Eq. (1) with a causal mask and grouped-query heads) and the Full-Recompute
// baseline (every row; Sec. IV-A).
//
// bf16 path (matrix cores, gfx950 v_mfma_f32_16x16x32_bf16):
//   * A workgroup owns M = 128 query vectors of one (request, KV head): BR
//     consecutive selected rows x the G = Hq/Hkv query heads that share the KV
//     head, so one K/V stream feeds all of them. When BR does not divide the
//     row count, the short tile is the first (lowest positions, fewest keys)
//     rather than the last (the longest).
//   * Each of the 4 waves owns 32 query vectors (consecutive rows, all G heads
//     of each: its rows span the fewest positions, so its causal band is
//     narrow and it skips the tiles past its last row) and computes
//     S^T = K Q^T for a 64-key tile (keys on the MFMA rows, queries on its columns) with Q held
//     in registers and K read from LDS. In the output layout a lane then holds
//     4 consecutive keys of one query column, which is also the B-operand
//     layout of the second product O^T = V^T P^T, so P never leaves registers;
//     V is staged key-major in LDS and read with the gfx950 transposed LDS
//     read (ds_read_b64_tr_b16) straight into the A-operand layout.
//   * Online softmax in the log2 domain with a lazily raised reference max;
//     the running denominators are column sums of the bf16 P^T taken on the
//     matrix cores (ones x P^T), consistent with the P used for O. K/V tiles
//     are double-buffered in LDS (one barrier per tile) with the next tile's
//     global loads in flight during compute. For D = 128 (not paged) the
//     tiles go from HBM straight into LDS and every K/V read of the tile loop
//     is issued as assembly (layouts and ordering at AttnBufDirect).
//   * A tile is computed in halves of 32 keys, so that the probabilities of
//     the second half are formed on the vector ALU beside the matrix
//     products of the first (compute_tile).
//   * Workgroup ids are remapped so that all row tiles of one (request, KV
//     head) run on the same XCD (ids are dealt round-robin over the 8 XCDs),
//     sharing its L2 for the K/V stream. Each XCD starts its longest (latest)
//     tiles first, across all of its groups when the batch's K/V fits the
//     Infinity Cache, else within chunks of groups that fit its L2.
// Paged mode (zero-copy, over the logical-to-physical block mapping of
// Sec. III-A): no assembled copy exists; each key of a tile is resolved
// through the request's segment table while it is staged -- a fresh row, the
// fresh row again when the key is itself a recomputed row (the heavy-hitter
// update of Sec. III-C.3 (iii)), or the pool row, whose key pairs are rotated
// by the segment's dst_start in registers (step (ii)) before they reach LDS.
// The tiles are then bit-identical to those of the assembled path.
// fp32 path: one wave per (request, row, head), fp32 FMA on the vector ALUs.
#include <cmath>
#include <type_traits>

#include "rc_common.h"

namespace rc {
namespace {

constexpr int kAttnThreads = 256;
constexpr int kM = 128;  // query vectors per workgroup
constexpr int kKT = 64;  // keys per KV tile
constexpr int kXcds = 8;
constexpr int kPagedMaxSegments = 64;  // segment table of a request kept in LDS

using u32x2 = uint32_t __attribute__((ext_vector_type(2)));
using u32x4 = uint32_t __attribute__((ext_vector_type(4)));

// Row pads keep the two LDS read patterns conflict-free: 16-byte reads of 16
// consecutive K rows (row stride = 16 mod 256 bytes), and transposed 8-byte
// reads of 8 consecutive V rows per half-wave (row stride = 32 mod 256 bytes).
// Two buffers: the next tile is written while the current one is read.
template <int D>
struct AttnSmem {
  uint16_t k[2][kKT][D + 8];   // K tiles, key-major
  uint16_t v[2][kKT][D + 16];  // V tiles, key-major (read transposed)
};

// D = 128, not paged: tiles land in LDS straight from global memory
// (global_load_lds_dwordx4: each wave instruction writes 1 KB contiguously, 4
// whole rows of 256 bytes, the best-coalesced fetch), so rows cannot be
// padded; the 16-byte chunks of a row are XOR-swizzled instead. K row r keeps
// data chunk c at chunk c ^ (r % 16): a fragment read of 16 consecutive rows
// hits 16 distinct chunks. V row r keeps data chunk c at chunk c ^ 2 (r % 8):
// the transposed reads of one half-wave (8 consecutive rows, two adjacent
// chunks) hit 16 distinct chunks. Every K and V read of the tile loop is
// issued as assembly from a few precomputed per-lane addresses plus constant
// offsets (tile row block, buffer), and the tile loads as assembly too: the
// compiler sees none of them, so it inserts no waits between the loads in
// flight and the reads of the other buffer (after LDS lowering both buffers
// are offsets of one object, and it would drain every load before each
// read); the kernel orders them itself with explicit waits and barriers.
struct AttnBufDirect {
  uint16_t k[kKT * 128];
  uint16_t v[kKT * 128];
};
struct AttnNone {
  int unused;
};

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// gfx950 transposed LDS read (ds_read_b64_tr_b16). Within each group of 16
// lanes, lane s reads 4 consecutive 16-bit elements at its address; lane j
// receives element j%4 of the reads of lanes j/4, j/4+4, j/4+8, j/4+12. With
// lane s pointing at row (r0 + s/4), column (c0 + 4*(s%4)) of a row-major tile,
// lane j receives column c0 + j of rows r0 .. r0+3.
__device__ __forceinline__ u32x2 lds_read_tr4(const uint16_t* p) {
  const v4i16 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_v4i16*)((__attribute__((address_space(3))) char*)(p)));
  return __builtin_bit_cast(u32x2, r);
}

// The same transposed read as inline assembly, at lds_addr + OFF bytes. The
// compiler does not track it: its result is valid only after lds_wait_tied
// has covered it.
template <int OFF>
__device__ __forceinline__ u32x2 lds_read_tr4_async(uint32_t lds_addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset field");
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(lds_addr), "n"(OFF));
  return r;
}

// One global->LDS load (16 bytes per lane, 1 KB per wave) from a wave-uniform
// base plus a 32-bit per-lane byte offset into the LDS bytes at lds_addr
// (wave-uniform). Issued as assembly: the compiler does not track it, so the
// caller waits for it with an explicit vmcnt wait before the data is read.
// M0 (the LDS destination) is restored afterwards: the compiler does not
// expect an assembly statement to change it.
__device__ __forceinline__ void dma16(uint32_t lds_addr, const void* gbase, uint32_t goff) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %2, %3\n\ts_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_addr), "v"(goff), "s"(gbase)
      : "memory");
}

// The same global->LDS load from a per-lane 64-bit address.
__device__ __forceinline__ void dma16_abs(uint32_t lds_addr, const void* gaddr) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %2, off\n\ts_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_addr), "v"(gaddr)
      : "memory");
}

// A 16-byte LDS read at lds_addr + OFF bytes as assembly; valid after
// lds_wait_tied has covered it.
template <int OFF>
__device__ __forceinline__ u32x4 lds_read_b128_async(uint32_t lds_addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset field");
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(lds_addr), "n"(OFF));
  return r;
}

template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// Waits until at most N LDS operations of this wave are outstanding. LDS
// operations complete in issue order, so this covers every read issued more
// than N operations ago. x and y are tied to the wait so that their uses
// cannot be scheduled above it.
template <int N>
__device__ __forceinline__ void lds_wait_tied(u32x2& x, u32x2& y) {
  asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(x), "+v"(y) : "n"(N));
}
template <int N>
__device__ __forceinline__ void lds_wait_tied(u32x4& x) {
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(x) : "n"(N));
}

// Maximum over the four 16-lane rows of a wave for each lane position
// (lanes l, l^16, l^32, l^48), with the gfx950 row-swap permutes on the vector
// ALU instead of LDS-routed shuffles.
__device__ __forceinline__ float max_over_rows(float m) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  m = __builtin_elementwise_maximum(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  return __builtin_elementwise_maximum(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// two fp32 -> packed bf16 (round to nearest even), one v_cvt_pk_bf16_f32
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// Softmax exponents use a running reference max that is only raised when a
// score exceeds it by more than 2^kLazy (log2 units): p <= 2^kLazy stays exact
// in fp32 and bf16, and the O/l rescale is skipped on most tiles.
constexpr float kLazy = 8.f;

// SELECTIVE: query rows come from `rows`; otherwise row r is position r
// (Full-Recompute). Separate instances keep the two modes apart in profiles.
// LSE: also write each row's natural log-sum-exp, from an fp32 sum of the
// unrounded exponentials (the bf16 column sums only normalise O).
// PAGED: k, v are the fresh tensors; other keys come from `pools` through
// `segs` (S <= kPagedMaxSegments), rotated with the cos/sin tables when given.
template <int D, bool SELECTIVE, bool LSE, bool PAGED, bool VREF = false>
__global__ __launch_bounds__(kAttnThreads) __attribute__((amdgpu_waves_per_eu(2)))
void attn_bf16_kernel(const uint16_t* __restrict__ q, const int32_t* __restrict__ rows, int R,
                      int N, int Hq, int Hkv, int G, int BR, int shift, const uint16_t* __restrict__ k,
                      const uint16_t* __restrict__ v, float scale_log2e,
                      uint16_t* __restrict__ out, float* __restrict__ lse, int n_tiles,
                      int n_groups, int gpx, int chunk, PoolArgs pools,
                      const int4* __restrict__ segs, int S, const float* __restrict__ cos_t,
                      const float* __restrict__ sin_t, int max_pos) {
  constexpr int DC = D / 32;          // 32-wide d chunks (S^T reduction)
  constexpr int DB = D / 16;          // 16-wide d blocks (O^T rows)
  constexpr int UPR = D / 8;          // 16-byte units per K/V head row
  constexpr int KU = kKT * UPR / kAttnThreads;   // K (and V) units per thread
  constexpr int KSTEP = kAttnThreads / UPR;      // keys between a thread's units
  constexpr bool DIRECT = (D == 128) && !PAGED;
  static_assert(!VREF || DIRECT, "V rows by reference need the direct D = 128 staging");
  __shared__ std::conditional_t<DIRECT, AttnNone, AttnSmem<D>> sm;
  __shared__ std::conditional_t<DIRECT, AttnBufDirect, AttnNone> sbuf[2];
  __shared__ int s_ext[4];
  __shared__ int4 s_psegs[PAGED ? kPagedMaxSegments : 1];
  __shared__ uint32_t s_sel[PAGED ? kMaxSelectN / 32 : 1];  // recomputed rows of the request

  // ---- work item: XCD-major; the XCD's groups in chunks of `chunk` groups,
  // longest tiles first within a chunk
  const int hw = blockIdx.x;
  const int xcd = hw % kXcds;
  const int slot = hw / kXcds;
  const int per_chunk = chunk * n_tiles;
  const int ci = slot / per_chunk;
  const int in_chunk = slot - ci * per_chunk;
  const int cg = min(chunk, gpx - ci * chunk);   // groups in this chunk
  const int rank = in_chunk / cg;
  const int grp = (ci * chunk + (in_chunk - rank * cg)) * kXcds + xcd;
  if (rank >= n_tiles || grp >= n_groups) return;
  const int tile = n_tiles - 1 - rank;
  const int b = grp / Hkv;
  const int g = grp - b * Hkv;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c16 = lane & 15;
  const int q4 = lane >> 4;

  // ---- the two query vectors (S^T columns) this lane serves
  int pos[2], head[2], row[2];
  bool valid[2], bad[2];
  int pmax = 0, pmin = 0x7fffffff;
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int m = wave * 32 + nb * 16 + c16;
    const int rl = m / G;          // vector m: row m / G, head m % G
    const int hh = m - rl * G;
    const int r = tile * BR + rl - shift;
    valid[nb] = hh < G && r >= 0 && r < R;
    bad[nb] = false;
    int p = 0;
    if (valid[nb]) {
      p = SELECTIVE ? rows[static_cast<size_t>(b) * R + r] : r;
      // a listed position outside [0, N) computes row 0 and stores NaN
      bad[nb] = p < 0 || p >= N;
      p = bad[nb] ? 0 : p;
      pmax = max(pmax, p);
      pmin = min(pmin, p);
    }
    pos[nb] = p;
    head[nb] = g * G + (hh < G ? hh : 0);
    row[nb] = r;
  }
  pmax = wave_max_i(pmax);
  const int wave_pmin = wave_min_i(pmin);
  if (lane == 0) s_ext[wave] = pmax;
  if constexpr (PAGED) {
    for (int s = tid; s < S; s += kAttnThreads) s_psegs[s] = segs[static_cast<size_t>(b) * S + s];
    for (int w = tid; w < (N + 31) / 32; w += kAttnThreads) s_sel[w] = 0u;
    __syncthreads();
    for (int r = tid; r < R; r += kAttnThreads) {
      const int p = rows[static_cast<size_t>(b) * R + r];
      if (p >= 0 && p < N) atomicOr(&s_sel[p >> 5], 1u << (p & 31));
    }
  }
  __syncthreads();
  const int wg_pmax = max(max(s_ext[0], s_ext[1]), max(s_ext[2], s_ext[3]));
  const int n_kv = wg_pmax / kKT + 1;

  // ---- Q fragments (B operand of S^T = K Q^T): 8 consecutive dims per lane
  bf16x8 qf[2][DC];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const uint16_t* qrow = q + ((static_cast<size_t>(b) * N + pos[nb]) * Hq + head[nb]) * D;
#pragma unroll
    for (int dc = 0; dc < DC; ++dc)
      qf[nb][dc] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(qrow + dc * 32 + q4 * 8));
  }

  // ---- K/V staging: thread owns units (key tid/UPR + i*KSTEP, dims (tid%UPR)*8 ..);
  // paged: key pairs (key tid/PPR + i*PSTEP, dims ps*8 .. and ps*8 + D/2 ..)
  const size_t stride = static_cast<size_t>(Hkv) * D;   // elements between keys
  constexpr int PPR = UPR / 2;                           // pair slots per key head row
  constexpr int PSTEP = kAttnThreads / PPR;              // keys between a thread's pairs
  constexpr int PK = kKT / PSTEP;                        // key pairs per thread
  static_assert(2 * PK == KU, "paged staging moves as many units as plain staging");
  const int key0 = PAGED ? tid / PPR : tid / UPR;
  const int col0 = PAGED ? (tid % PPR) * 8 : (tid % UPR) * 8;
  const size_t off0 = (static_cast<size_t>(b) * N + key0) * stride + static_cast<size_t>(g) * D + col0;
  const uint16_t* kp = k + off0;
  const uint16_t* vp = v + off0;
  const size_t tile_step = static_cast<size_t>(kKT) * stride;
  u32x4 kreg[DIRECT ? 1 : KU], vreg[DIRECT ? 1 : KU];
  int pdelta[PAGED ? PK : 1];  // paged: rotation of each staged key (0: none)
  int pseg[PAGED ? PK : 1] = {};  // paged: last segment starting at or before each slot's key
  // DIRECT: wave w fills rows 16w .. 16w+15 of both tiles with 4 + 4 loads;
  // lane l writes chunk l % 16 of row 16w + 4j + l / 16 and so fetches the
  // data chunk that the swizzle stores there. Keys past N repeat key N - 1
  // (finite values; the causal mask removes them).
  // DIRECT, whole tiles: per-lane 32-bit byte offsets of the sources within a
  // tile, so that a tile costs one scalar base and eight loads; LDS
  // destinations derive from the wave index kept in an SGPR
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  uint32_t koff[DIRECT ? 4 : 1], voff[DIRECT ? 4 : 1];
  if constexpr (DIRECT) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = wave * 16 + j * 4 + (lane >> 4);
      koff[j] = static_cast<uint32_t>((row * stride + g * D + (((lane & 15) ^ (row & 15)) * 8)) * 2);
      voff[j] = static_cast<uint32_t>((row * stride + g * D + (((lane & 15) ^ (2 * (row & 7))) * 8)) * 2);
      // VREF: the byte offset of this lane's chunk within its V row
      if constexpr (VREF) voff[j] = static_cast<uint32_t>((g * D + (((lane & 15) ^ (2 * (row & 7))) * 8)) * 2);
    }
  }
  // VREF: v holds the address of every position's V row ([B, N], 8 bytes
  // each; keys past N repeat key N - 1). One load per lane serves a pair of
  // tiles: lane l holds the entry of row 16 wave + l % 16 of tile
  // t + (l / 16) % 2, and the four entries a lane needs for a tile's loads
  // (vent) are taken from those lanes by permutes. The pair (t + 2, t + 3)
  // is read during tile t (t even): one extra vector-memory instruction per
  // two tiles instead of four per tile, each of which measured about 2% of
  // the kernel (the waves wait for the last load of a tile at its end).
  const uint64_t* vref = reinterpret_cast<const uint64_t*>(v);
  uint64_t vent[VREF ? 4 : 1];
  uint64_t vown = 0;
  auto load_vent = [&](int t) {
    if constexpr (VREF) {
      const int key = min((t + ((lane >> 4) & 1)) * kKT + wave * 16 + (lane & 15), N - 1);
      vown = vref[static_cast<size_t>(b) * N + key];
    }
  };
  auto spread_vent = [&](auto half_tag) {
    if constexpr (VREF) {
      constexpr int h = decltype(half_tag)::value;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int src = h * 16 + j * 4 + (lane >> 4);
        const uint32_t lo = __shfl(static_cast<uint32_t>(vown), src, 64);
        const uint32_t hi = __shfl(static_cast<uint32_t>(vown >> 32), src, 64);
        vent[j] = (static_cast<uint64_t>(hi) << 32) | lo;
      }
    }
  };
  auto issue_tile = [&](int t, auto buf_tag) {
    if constexpr (DIRECT) {
      auto& dst = sbuf[decltype(buf_tag)::value];
      if ((t + 1) * kKT <= N) {
        const size_t tile0 = (static_cast<size_t>(b) * N + static_cast<size_t>(t) * kKT) * stride;
        const char* kt = reinterpret_cast<const char*>(k + tile0);
        const char* vt = reinterpret_cast<const char*>(v + tile0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          dma16((uint32_t)(uintptr_t)((__attribute__((address_space(3))) uint16_t*)(&dst.k[(wave_u * 16 + j * 4) * 128])),
                kt, koff[j]);
          const uint32_t vdst = (uint32_t)(uintptr_t)((__attribute__((address_space(3))) uint16_t*)(&dst.v[(wave_u * 16 + j * 4) * 128]));
          if constexpr (VREF) dma16_abs(vdst, reinterpret_cast<const char*>(vent[j]) + voff[j]);
          else dma16(vdst, vt, voff[j]);
        }
        return;
      }
      // the last, partial tile: keys past N repeat key N - 1
      const int ch = lane & 15;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = wave * 16 + j * 4 + (lane >> 4);
        const int key = min(t * kKT + row, N - 1);
        const uint16_t* kr = k + (static_cast<size_t>(b) * N + key) * stride + static_cast<size_t>(g) * D;
        const uint16_t* vr = v + (static_cast<size_t>(b) * N + key) * stride + static_cast<size_t>(g) * D;
        __builtin_amdgcn_global_load_lds(
            (const __attribute__((address_space(1))) void*)(kr + ((ch ^ (row & 15)) * 8)),
            (__attribute__((address_space(3))) void*)(&dst.k[(wave * 16 + j * 4) * 128]), 16, 0, 0);
        if constexpr (VREF)
          dma16_abs((uint32_t)(uintptr_t)((__attribute__((address_space(3))) uint16_t*)(&dst.v[(wave_u * 16 + j * 4) * 128])),
                    reinterpret_cast<const char*>(vent[j]) + voff[j]);
        else
          __builtin_amdgcn_global_load_lds(
              (const __attribute__((address_space(1))) void*)(vr + ((ch ^ (2 * (row & 7))) * 8)),
              (__attribute__((address_space(3))) void*)(&dst.v[(wave * 16 + j * 4) * 128]), 16, 0, 0);
      }
    }
  };
  auto load_tile = [&](int t) {
    if constexpr (!DIRECT) {
    if constexpr (PAGED) {
#pragma unroll
      for (int i = 0; i < PK; ++i) {
        const int j = t * kKT + key0 + i * PSTEP;
        const uint16_t* ks = nullptr;
        const uint16_t* vs = nullptr;
        int d = 0;
        if (j < N) {
          // tiles are staged in increasing order, so a slot's key only moves
          // forward: advance its segment instead of searching for it
          int sg = pseg[i];
          while (sg + 1 < S && s_psegs[sg + 1].x <= j) ++sg;
          pseg[i] = sg;
          const int4 sg0 = s_psegs[sg];
          const int4 sgm = (sg0.x <= j && j < sg0.x + sg0.y) ? sg0 : int4{0, 0, -1, 0};
          const bool fresh = sgm.z < 0 || ((s_sel[j >> 5] >> (j & 31)) & 1u);
          if (fresh) {
            const size_t o = (static_cast<size_t>(b) * N + j) * stride + static_cast<size_t>(g) * D + col0;
            ks = k + o;
            vs = v + o;
          } else if (sgm.z < pools.n && sgm.w >= 0 && sgm.w < pools.num_blocks[sgm.z] &&
                     j - sgm.x < pools.block_len[sgm.z]) {
            const size_t prow = static_cast<size_t>(sgm.w) * pools.block_len[sgm.z] + (j - sgm.x);
            const size_t o = prow * stride + static_cast<size_t>(g) * D + col0;
            ks = reinterpret_cast<const uint16_t*>(pools.k[sgm.z]) + o;
            vs = reinterpret_cast<const uint16_t*>(pools.v[sgm.z]) + o;
            if (cos_t != nullptr && sgm.x < max_pos) d = sgm.x;
          }
        }
        pdelta[i] = d;
        kreg[2 * i] = ks ? *reinterpret_cast<const u32x4*>(ks) : u32x4{0, 0, 0, 0};
        kreg[2 * i + 1] = ks ? *reinterpret_cast<const u32x4*>(ks + D / 2) : u32x4{0, 0, 0, 0};
        vreg[2 * i] = vs ? *reinterpret_cast<const u32x4*>(vs) : u32x4{0, 0, 0, 0};
        vreg[2 * i + 1] = vs ? *reinterpret_cast<const u32x4*>(vs + D / 2) : u32x4{0, 0, 0, 0};
      }
      return;
    }
    const uint16_t* kt = kp + t * tile_step;
    const uint16_t* vt = vp + t * tile_step;
    if ((t + 1) * kKT <= N) {
#pragma unroll
      for (int i = 0; i < KU; ++i) {
        kreg[i] = *reinterpret_cast<const u32x4*>(kt + i * KSTEP * stride);
        vreg[i] = *reinterpret_cast<const u32x4*>(vt + i * KSTEP * stride);
      }
    } else {
#pragma unroll
      for (int i = 0; i < KU; ++i) {
        const bool in = t * kKT + key0 + i * KSTEP < N;
        kreg[i] = in ? *reinterpret_cast<const u32x4*>(kt + i * KSTEP * stride) : u32x4{0, 0, 0, 0};
        vreg[i] = in ? *reinterpret_cast<const u32x4*>(vt + i * KSTEP * stride) : u32x4{0, 0, 0, 0};
      }
    }
      }
};
  auto store_tile = [&](int buf) {
    if constexpr (!DIRECT) {
    if constexpr (PAGED) {
#pragma unroll
      for (int i = 0; i < PK; ++i) {
        const int d = pdelta[i];
        if (d != 0) {  // same fp32 operation order and rounding as the gather
          float c[8], sn[8];
          const float* crow = cos_t + static_cast<size_t>(d) * (D / 2) + col0;
          const float* srow = sin_t + static_cast<size_t>(d) * (D / 2) + col0;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            c[e] = crow[e];
            sn[e] = srow[e];
          }
          rotate_unit<2>(kreg[2 * i], kreg[2 * i + 1], c, sn);
        }
        const int key = key0 + i * PSTEP;
        *reinterpret_cast<u32x4*>(&sm.k[buf][key][col0]) = kreg[2 * i];
        *reinterpret_cast<u32x4*>(&sm.k[buf][key][col0 + D / 2]) = kreg[2 * i + 1];
        *reinterpret_cast<u32x4*>(&sm.v[buf][key][col0]) = vreg[2 * i];
        *reinterpret_cast<u32x4*>(&sm.v[buf][key][col0 + D / 2]) = vreg[2 * i + 1];
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < KU; ++i) {
      *reinterpret_cast<u32x4*>(&sm.k[buf][key0 + i * KSTEP][col0]) = kreg[i];
      *reinterpret_cast<u32x4*>(&sm.v[buf][key0 + i * KSTEP][col0]) = vreg[i];
    }
      }
};

  f32x4 o[DB][2];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) o[db][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[2] = {-INFINITY, -INFINITY};  // reference max of the unscaled scores
  // softmax denominators on the matrix cores: ones(16x32) x P^T gives the
  // column sums of P for every query column (all 4 lanes' entries equal)
  f32x4 l_acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  float l32[2] = {0.f, 0.f};  // LSE: this lane's share of the fp32 row sums
  const bf16x8 ones = __builtin_bit_cast(bf16x8, u32x4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});

  const int tr_row = q4 * 4 + (c16 >> 2);
  const int tr_col = 4 * (c16 & 3);

  // LDS addresses of a K fragment (row, 16-byte data chunk u) and of a
  // transposed V read (row, element col)
  auto kfrag = [&](auto buf_tag, int row, int u) -> const uint16_t* {
    constexpr int BUF = decltype(buf_tag)::value;
    if constexpr (DIRECT) return nullptr;   // DIRECT reads K through kaddr below
    else return &sm.k[BUF][row][u * 8];
  };
  auto vtr = [&](auto buf_tag, int row, int col) -> const uint16_t* {
    constexpr int BUF = decltype(buf_tag)::value;
    if constexpr (DIRECT) return nullptr;   // DIRECT reads V through vaddr below
    else return &sm.v[BUF][row][col];
  };
  // DIRECT: LDS byte address of this lane's 8 bytes in the first V block
  // DIRECT: LDS byte address of this lane's transposed V read of 16-dim block
  // db in rows 4 q4 + c16/4 (+ a multiple of 16 rows, a constant offset)
  uint32_t vaddr[DIRECT ? DB : 1], kaddr[DIRECT ? DC : 1];
  if constexpr (DIRECT) {
    const uint32_t v0 = (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) uint16_t*)(&sbuf[0].v[0]));
    const uint32_t k0 = (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) uint16_t*)(&sbuf[0].k[0]));
    const int x = 4 * (q4 & 1) + (c16 >> 2);   // row % 8 of this lane's rows
    const uint32_t lane_part = (4 * q4 + (c16 >> 2)) * 256 + (c16 & 1) * 8;
#pragma unroll
    for (int db = 0; db < DB; ++db) vaddr[db] = v0 + lane_part + (2 * (db ^ x) + ((c16 >> 1) & 1)) * 16;
    // K fragment (kb, dc): row kb*16 + c16, data chunk dc*4 + q4 at chunk (dc*4 + q4) ^ c16
#pragma unroll
    for (int dc = 0; dc < DC; ++dc) kaddr[dc] = k0 + c16 * 256 + (((dc * 4 + q4) ^ c16) * 16);
  }
  constexpr uint32_t kBufBytes = sizeof(AttnBufDirect);
  using Buf0 = std::integral_constant<int, 0>;
  using Buf1 = std::integral_constant<int, 1>;

  if constexpr (DIRECT) {
    load_vent(0);   // tiles 0 and 1
    spread_vent(Buf0{});
    issue_tile(0, Buf0{});
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  } else {
    load_tile(0);
    store_tile(0);
    __syncthreads();
    if (n_kv > 1) load_tile(1);
  }

  // first tile whose last key passes this wave's earliest row
  const int t_mask = min(n_kv, wave_pmin / kKT);
  const int wave_last = pmax / kKT;   // tiles past it are masked for every row of this wave

  // One KV tile (either staging) in an order that lets the vector ALU work
  // beside the matrix cores. Scores of keys 0..31 first; then the scores of keys 32..63
  // are issued, with the probabilities of keys 0..31 against the current
  // reference max placed between them (the compiler moves those below the
  // rescale decision, whose path recomputes them; forcing them above it
  // needs more than the 256 registers of two waves per SIMD and spills);
  // after the rescale decision (taken on the whole tile), V^T P^T of keys
  // 0..31 runs while the probabilities of keys 32..63 are formed. Without a rescale the reference max is unchanged, so every
  // value equals that of the plain order (all scores, then all
  // probabilities); with one, the probabilities of keys 0..31 are recomputed
  // from the scores, which are kept until the decision.
  auto compute_tile = [&](int t, auto buf_tag, auto mask_tag) __attribute__((always_inline)) {
    constexpr int cur = decltype(buf_tag)::value;
    constexpr bool MASKED = decltype(mask_tag)::value;
    f32x4 s[4][2];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) s[kb][0] = s[kb][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    // K fragments in the order (dc, kb) within each half of the keys:
    // fragment gi of half h is key block 2h + gi % 2, d chunk gi / 2
    constexpr int KG = DC * 4;
    constexpr int KAHEAD = 5;
    u32x4 kf[KG];
    auto rdk = [&](auto G) {
      constexpr int gi = decltype(G)::value;
      constexpr int h = gi / (KG / 2), r = gi % (KG / 2);
      constexpr int kb = 2 * h + r % 2, dc = r / 2;
      kf[gi] = lds_read_b128_async<cur * kBufBytes + kb * 4096>(kaddr[dc]);
    };
    auto mm = [&](auto G) {
      constexpr int gi = decltype(G)::value;
      constexpr int later = (KG - 1 - gi) < KAHEAD ? (KG - 1 - gi) : KAHEAD;
      lds_wait_tied<later>(kf[gi]);
      constexpr int h = gi / (KG / 2), r = gi % (KG / 2);
      constexpr int kb = 2 * h + r % 2, dc = r / 2;
      const bf16x8 a = __builtin_bit_cast(bf16x8, kf[gi]);
      s[kb][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[0][dc], s[kb][0], 0, 0, 0);
      s[kb][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[1][dc], s[kb][1], 0, 0, 0);
      if constexpr (gi + KAHEAD + 1 < KG) rdk(std::integral_constant<int, gi + KAHEAD + 1>{});
    };
    auto mask_half = [&](int h) __attribute__((always_inline)) {
      if constexpr (MASKED) {
        const int j0 = t * kKT;
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (j0 + (2 * h + kk) * 16 + q4 * 4 + i > pos[nb]) s[2 * h + kk][nb][i] = -INFINITY;
      }
    };
    // per column: maximum of a half, probabilities of a half (packed) and
    // their fp32 sums by key block
    auto half_max = [&](int h, int nb) __attribute__((always_inline)) -> float {
      return __builtin_elementwise_maximum(
          __builtin_elementwise_maximum(
              __builtin_elementwise_maximum(s[2 * h][nb][0], s[2 * h][nb][1]),
              __builtin_elementwise_maximum(s[2 * h][nb][2], s[2 * h][nb][3])),
          __builtin_elementwise_maximum(
              __builtin_elementwise_maximum(s[2 * h + 1][nb][0], s[2 * h + 1][nb][1]),
              __builtin_elementwise_maximum(s[2 * h + 1][nb][2], s[2 * h + 1][nb][3])));
    };
    bf16x8 pb[2][2];
    float ls[4][2];  // LSE: fp32 sum of each key block's probabilities
    auto probs = [&](int h, int nb, float mc) __attribute__((always_inline)) {
      float p[2][4];
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          p[kk][i] = __builtin_amdgcn_exp2f(fmaf(s[2 * h + kk][nb][i], scale_log2e, -mc));
      if constexpr (LSE) {
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) ls[2 * h + kk][nb] = (p[kk][0] + p[kk][1]) + (p[kk][2] + p[kk][3]);
      }
      const u32x4 w = {pack_bf16x2(p[0][0], p[0][1]), pack_bf16x2(p[0][2], p[0][3]),
                       pack_bf16x2(p[1][0], p[1][1]), pack_bf16x2(p[1][2], p[1][3])};
      pb[h][nb] = __builtin_bit_cast(bf16x8, w);
    };

    // without DIRECT: K fragments through ordinary LDS reads (padded layout)
    auto mmp = [&](auto G) {
      constexpr int gi = decltype(G)::value;
      constexpr int h = gi / (KG / 2), r = gi % (KG / 2);
      constexpr int kb = 2 * h + r % 2, dc = r / 2;
      const bf16x8 a = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(kfrag(buf_tag, kb * 16 + c16, dc * 4 + q4)));
      s[kb][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[0][dc], s[kb][0], 0, 0, 0);
      s[kb][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[1][dc], s[kb][1], 0, 0, 0);
    };
    __builtin_amdgcn_s_setprio(1);
    if constexpr (DIRECT) {
      static_for<0, KAHEAD + 1>(rdk);
      static_for<0, KG / 2>(mm);
      // scores of keys 32..63 on the matrix cores; keys 0..31 on the vector ALU
      static_for<KG / 2, KG>(mm);
    } else {
      static_for<0, KG / 2>(mmp);
      static_for<KG / 2, KG>(mmp);
    }
    mask_half(0);
    float m0[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      m0[nb] = half_max(0, nb);
      probs(0, nb, m_run[nb] * scale_log2e);
    }
    // issue order: the first half's products, then each product of the
    // second half followed by vector work of the first half
    __builtin_amdgcn_sched_group_barrier(0x008, KG, 0);
    static_for<0, KG>([&](auto) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
    });
    __builtin_amdgcn_s_setprio(0);
    mask_half(1);
    float mx[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) mx[nb] = max_over_rows(__builtin_elementwise_maximum(m0[nb], half_max(1, nb)));
    // a query sees key 0 in the first tile, so the reference max is finite after it
    if (__ballot(mx[0] * scale_log2e - m_run[0] * scale_log2e > kLazy ||
                 mx[1] * scale_log2e - m_run[1] * scale_log2e > kLazy) != 0) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const float m_new = fmaxf(m_run[nb], mx[nb]);
        const float alpha = __builtin_amdgcn_exp2f((m_run[nb] - m_new) * scale_log2e);
        l_acc[nb] *= alpha;
        if constexpr (LSE) l32[nb] *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db][nb] *= alpha;
        m_run[nb] = m_new;
        probs(0, nb, m_new * scale_log2e);
      }
    }

    // ---- O^T += V^T P^T: keys 0..31 while the vector ALU forms keys 32..63
    __builtin_amdgcn_s_setprio(1);
    constexpr int NG = 2 * DB;
    constexpr int AHEAD = 4;
    u32x2 lo[NG], hi[NG];
    auto rd = [&](auto G) {
      constexpr int gi = decltype(G)::value;
      constexpr int kc = gi / DB, db = gi % DB;
      lo[gi] = lds_read_tr4_async<cur * kBufBytes + kc * 8192>(vaddr[db]);
      hi[gi] = lds_read_tr4_async<cur * kBufBytes + kc * 8192 + 4096>(vaddr[db]);
    };
    auto pv = [&](auto G) {
      constexpr int gi = decltype(G)::value;
      constexpr int later = (NG - 1 - gi) < AHEAD ? (NG - 1 - gi) : AHEAD;
      lds_wait_tied<2 * later>(lo[gi], hi[gi]);
      constexpr int kc = gi / DB, db = gi % DB;
      const bf16x8 a = __builtin_bit_cast(bf16x8, u32x4{lo[gi][0], lo[gi][1], hi[gi][0], hi[gi][1]});
      o[db][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[kc][0], o[db][0], 0, 0, 0);
      o[db][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[kc][1], o[db][1], 0, 0, 0);
      if constexpr (gi + AHEAD + 1 < NG) rd(std::integral_constant<int, gi + AHEAD + 1>{});
    };
    // without DIRECT: transposed reads of the padded V tile
    auto pvp = [&](auto G) {
      constexpr int gi = decltype(G)::value;
      constexpr int kc = gi / DB, db = gi % DB;
      const u32x2 l2 = lds_read_tr4(vtr(buf_tag, kc * 32 + tr_row, db * 16 + tr_col));
      const u32x2 h2 = lds_read_tr4(vtr(buf_tag, kc * 32 + 16 + tr_row, db * 16 + tr_col));
      const bf16x8 a = __builtin_bit_cast(bf16x8, u32x4{l2[0], l2[1], h2[0], h2[1]});
      o[db][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[kc][0], o[db][0], 0, 0, 0);
      o[db][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[kc][1], o[db][1], 0, 0, 0);
    };
    if constexpr (DIRECT) {
      static_for<0, AHEAD + 1>(rd);
      static_for<0, DB>(pv);
    } else {
      static_for<0, DB>(pvp);
    }
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) probs(1, nb, m_run[nb] * scale_log2e);
    if constexpr (LSE) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        l32[nb] = (((l32[nb] + ls[0][nb]) + ls[1][nb]) + ls[2][nb]) + ls[3][nb];
    }
    if constexpr (DIRECT) static_for<DB, NG>(pv);
    else static_for<DB, NG>(pvp);
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      l_acc[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb[kc][0], l_acc[0], 0, 0, 0);
      l_acc[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb[kc][1], l_acc[1], 0, 0, 0);
    }
    __builtin_amdgcn_s_setprio(0);
  };

  // One KV tile: S^T = K Q^T, (masked) online softmax, O^T += V^T P^T, then
  // stage the next tile. The causal mask is applied only on tiles reaching past
  // some row of this wave (a uniform branch).
  auto do_tile = [&](int t, auto buf_tag) {
    const bool MASK = t >= t_mask;                  // uniform: tiles past this wave's first row
    constexpr int cur = decltype(buf_tag)::value;   // == t & 1
    using Next = std::integral_constant<int, cur ^ 1>;
    // DIRECT: the next tile flows into the other buffer during this one
    if constexpr (DIRECT) {
      if (t + 1 < n_kv) {
        spread_vent(Next{});          // tile t + 1: half (t + 1) % 2 of the pair
        issue_tile(t + 1, Next{});
        // even t: the pair (t + 2, t + 3), after its last use above
        if (cur == 0 && t + 2 < n_kv) load_vent(t + 2);
      }
    }

    // a wave skips the tiles past all of its rows (their weights are zero)
    if (t <= wave_last) {
      if (MASK) compute_tile(t, buf_tag, std::true_type{});
      else compute_tile(t, buf_tag, std::false_type{});
    }

    // ---- stage the next tile into the other buffer, prefetch the one after
    if constexpr (DIRECT) {
      __builtin_amdgcn_s_waitcnt(0);   // this wave's loads of tile t + 1 have landed
    } else if (t + 1 < n_kv) {
      store_tile(cur ^ 1);
      if (t + 2 < n_kv) load_tile(t + 2);
    }
    __syncthreads();
  };

  int t = 0;
  for (; t + 1 < n_kv; t += 2) {
    do_tile(t, Buf0{});
    do_tile(t + 1, Buf1{});
  }
  if (t < n_kv) do_tile(t, Buf0{});

  // ---- log-sum-exp: the 4 lanes of a query column hold disjoint keys
  if constexpr (LSE) {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      float l = l32[nb];
      l += __shfl_xor(l, 16, 64);
      l += __shfl_xor(l, 32, 64);
      if (valid[nb] && q4 == 0)
        lse[(static_cast<size_t>(b) * R + row[nb]) * Hq + head[nb]] =
            bad[nb] ? __builtin_nanf("") : (m_run[nb] * scale_log2e + __log2f(l)) * 0.69314718055994531f;
    }
  }

  // ---- normalise and store: lane holds dims db*16 + q4*4 .. +3 of its query
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const float inv = 1.f / l_acc[nb][0];
    if (!valid[nb]) continue;
    uint16_t* orow = out + ((static_cast<size_t>(b) * R + row[nb]) * Hq + head[nb]) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const u32x2 w = bad[nb] ? u32x2{0x7fc07fc0u, 0x7fc07fc0u}
                              : u32x2{pack_bf16x2(o[db][nb][0] * inv, o[db][nb][1] * inv),
                                      pack_bf16x2(o[db][nb][2] * inv, o[db][nb][3] * inv)};
      *reinterpret_cast<u32x2*>(orow + db * 16 + q4 * 4) = w;
    }
  }
}

// fp32: one wave per (request, row, q-head). Lanes own keys while scoring
// (64 keys per step) and dims while accumulating P V.
template <int D>
__global__ __launch_bounds__(256) void attn_f32_kernel(const float* __restrict__ q,
                                                       const int32_t* __restrict__ rows, int R,
                                                       int N, int Hq, int Hkv,
                                                       const float* __restrict__ k,
                                                       const float* __restrict__ v, float scale,
                                                       float* __restrict__ out,
                                                       float* __restrict__ lse, int64_t total) {
  constexpr int PER = D / 64;
  __shared__ float s_q[4][D];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t w = static_cast<int64_t>(blockIdx.x) * 4 + wave;
  const bool active = w < total;
  const int64_t wi = active ? w : 0;
  const int h = static_cast<int>(wi % Hq);
  const int64_t br = wi / Hq;
  const int r = static_cast<int>(br % R);
  const int b = static_cast<int>(br / R);
  int p = rows ? rows[static_cast<size_t>(b) * R + r] : r;
  const bool bad = p < 0 || p >= N;   // computes row 0, stores NaN
  p = bad ? 0 : p;
  const int g = h / (Hq / Hkv);
  const float* qrow = q + ((static_cast<size_t>(b) * N + p) * Hq + h) * D;
  for (int d = lane; d < D; d += 64) s_q[wave][d] = qrow[d];
  __syncthreads();
  if (!active) return;
  const size_t kv_stride = static_cast<size_t>(Hkv) * D;
  const float* kb = k + static_cast<size_t>(b) * N * kv_stride + static_cast<size_t>(g) * D;
  const float* vb = v + static_cast<size_t>(b) * N * kv_stride + static_cast<size_t>(g) * D;
  float m = -INFINITY, l = 0.f, acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  for (int c = 0; c <= p; c += 64) {
    const int j = c + lane;
    float sc = -INFINITY;
    if (j <= p) {
      const float* kr = kb + j * kv_stride;
      float dot = 0.f;
#pragma unroll 8
      for (int d = 0; d < D; ++d) dot = fmaf(s_q[wave][d], kr[d], dot);
      sc = dot * scale;
    }
    const float cm = wave_max(sc);
    const float m_new = fmaxf(m, cm);
    const float alpha = expf(m - m_new);
    const float pj = j <= p ? expf(sc - m_new) : 0.f;
    l = l * alpha + wave_sum(pj);
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] *= alpha;
    const int cnt = min(64, p - c + 1);
    for (int jj = 0; jj < cnt; ++jj) {
      const float pw = __shfl(pj, jj, 64);
      const float* vr = vb + (c + jj) * kv_stride;
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] = fmaf(pw, vr[lane * PER + e], acc[e]);
    }
    m = m_new;
  }
  float* orow = out + ((static_cast<size_t>(b) * R + r) * Hq + h) * D;
  const float nan = __builtin_nanf("");
#pragma unroll
  for (int e = 0; e < PER; ++e) orow[lane * PER + e] = bad ? nan : acc[e] / l;
  if (lse && lane == 0) lse[(static_cast<size_t>(b) * R + r) * Hq + h] = bad ? nan : m + logf(l);
}

}  // namespace
}  // namespace rc

namespace rc {
namespace {

struct Paged {
  PoolArgs pools;
  const int4* segs;
  int S;
  const float* cos_t;
  const float* sin_t;
  int max_pos;
};

// paged == nullptr: k, v are the assembled tensors; else the fresh tensors.
int attention_impl(const rc_shape* shape, const void* q, const int32_t* rows, int32_t R,
                   const void* k, const void* v, float scale, void* out, float* lse,
                   const Paged* paged, hipStream_t stream, const char* what, bool vref = false) {
  if (int st = check_shape(shape, true)) return st;
  if (R < 0) return fail(RC_ERR_INVALID_ARG, "R=%d must be >= 0", R);
  if (!q || !k || !v || (!out && R > 0))
    return fail(RC_ERR_INVALID_ARG, "q, k, v and out must be non-NULL");
  if (!rows && R != shape->N)
    return fail(RC_ERR_INVALID_ARG, "full-prefill mode (rows NULL) needs R == N (R=%d, N=%d)", R, shape->N);
  if (!(scale > 0.f) || !std::isfinite(scale))
    return fail(RC_ERR_INVALID_ARG, "scale must be finite and > 0");
  if (R == 0) return RC_OK;
  const int B = shape->B, N = shape->N, Hq = shape->Hq, Hkv = shape->Hkv, D = shape->D;
  const int G = Hq / Hkv;
  if (shape->dtype == RC_BF16) {
    if (kM % G != 0) return fail(RC_ERR_UNSUPPORTED, "group size Hq/Hkv=%d must divide %d", G, kM);
    const int BR = kM / G;
    const int n_tiles = (R + BR - 1) / BR;
    const int n_groups = B * Hkv;
    const int gpx = (n_groups + kXcds - 1) / kXcds;   // groups per XCD
    // When the batch's K/V fits the 256 MB Infinity Cache, every group of an
    // XCD is scheduled longest-tile-first together (load balance); otherwise
    // groups go in chunks whose K/V fits one XCD's 4 MB L2 (reuse).
    const double group_bytes = 2.0 * N * D * elem_size(shape->dtype);
    const double batch_bytes = group_bytes * n_groups;
    int chunk = gpx;
    if (batch_bytes > 192.0 * (1 << 20)) chunk = max(1, static_cast<int>((4.0 * (1 << 20)) / group_bytes));
    chunk = min(chunk, gpx);
    const int64_t blocks = static_cast<int64_t>(kXcds) * gpx * n_tiles;
    if (blocks > 0x7fffffff) return fail(RC_ERR_UNSUPPORTED, "grid too large");
    const float scale_log2e = static_cast<float>(static_cast<double>(scale) * 1.4426950408889634);
    dim3 grid(static_cast<unsigned>(blocks));
    const Paged none{};
    const Paged& pg = paged ? *paged : none;
    auto launch = [&](auto kern) {
      hipLaunchKernelGGL(kern, grid, dim3(kAttnThreads), 0, stream,
                         static_cast<const uint16_t*>(q), rows, R, N, Hq, Hkv, G, BR, n_tiles * BR - R,
                         static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v),
                         scale_log2e, static_cast<uint16_t*>(out), lse, n_tiles, n_groups, gpx,
                         chunk, pg.pools, pg.segs, pg.S, pg.cos_t, pg.sin_t, pg.max_pos);
    };
    if (vref) {
      rows ? launch(attn_bf16_kernel<128, true, false, false, true>)
           : launch(attn_bf16_kernel<128, false, false, false, true>);
    } else if (paged) {
      if (D == 128) launch(attn_bf16_kernel<128, true, false, true>);
      else launch(attn_bf16_kernel<64, true, false, true>);
    } else if (lse) {
      if (D == 128)
        rows ? launch(attn_bf16_kernel<128, true, true, false>) : launch(attn_bf16_kernel<128, false, true, false>);
      else
        rows ? launch(attn_bf16_kernel<64, true, true, false>) : launch(attn_bf16_kernel<64, false, true, false>);
    } else {
      if (D == 128)
        rows ? launch(attn_bf16_kernel<128, true, false, false>) : launch(attn_bf16_kernel<128, false, false, false>);
      else
        rows ? launch(attn_bf16_kernel<64, true, false, false>) : launch(attn_bf16_kernel<64, false, false, false>);
    }
  } else {
    if (paged) return fail(RC_ERR_UNSUPPORTED, "paged attention is implemented for bf16");
    const int64_t total = static_cast<int64_t>(B) * R * Hq;
    const int64_t blocks = (total + 3) / 4;
    if (blocks > 0x7fffffff) return fail(RC_ERR_UNSUPPORTED, "grid too large");
    dim3 grid(static_cast<unsigned>(blocks));
    if (D == 128)
      hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(256), 0, stream,
                         static_cast<const float*>(q), rows, R, N, Hq, Hkv,
                         static_cast<const float*>(k), static_cast<const float*>(v), scale,
                         static_cast<float*>(out), lse, total);
    else
      hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(256), 0, stream,
                         static_cast<const float*>(q), rows, R, N, Hq, Hkv,
                         static_cast<const float*>(k), static_cast<const float*>(v), scale,
                         static_cast<float*>(out), lse, total);
  }
  return check_launch(what);
}

}  // namespace
}  // namespace rc

extern "C" int rc_selective_attention(const rc_shape* shape, const void* q, const int32_t* rows,
                                      int32_t R, const void* k, const void* v, float scale,
                                      void* out, hipStream_t stream) {
  rc::clear_error();
  return rc::attention_impl(shape, q, rows, R, k, v, scale, out, nullptr, nullptr, stream,
                            "rc_selective_attention");
}

extern "C" int rc_selective_attention_lse(const rc_shape* shape, const void* q,
                                          const int32_t* rows, int32_t R, const void* k,
                                          const void* v, float scale, void* out, float* lse,
                                          hipStream_t stream) {
  rc::clear_error();
  if (!lse && R > 0) return rc::fail(RC_ERR_INVALID_ARG, "lse must be non-NULL");
  return rc::attention_impl(shape, q, rows, R, k, v, scale, out, lse, nullptr, stream,
                            "rc_selective_attention_lse");
}

extern "C" int rc_selective_attention_vref(const rc_shape* shape, const void* q,
                                           const int32_t* rows, int32_t R, const void* k,
                                           const uint64_t* v_ref, float scale, void* out,
                                           hipStream_t stream) {
  rc::clear_error();
  if (shape && (shape->dtype != RC_BF16 || shape->D != 128))
    return rc::fail(RC_ERR_UNSUPPORTED, "V rows by reference: bf16 with D = 128 only");
  return rc::attention_impl(shape, q, rows, R, k, v_ref, scale, out, nullptr, nullptr, stream,
                            "rc_selective_attention_vref", true);
}

extern "C" int rc_paged_attention(const rc_shape* shape, const void* q, const int32_t* rows,
                                  int32_t R, const rc_pool* pools, int32_t n_pools,
                                  const rc_segment* segs, int32_t S, const void* k_fresh,
                                  const void* v_fresh, const float* rope_cos,
                                  const float* rope_sin, int32_t max_pos, float scale, void* out,
                                  hipStream_t stream) {
  using namespace rc;
  clear_error();
  if (int st = check_shape(shape, true)) return st;
  if (!rows && R > 0) return fail(RC_ERR_INVALID_ARG, "rows must be non-NULL");
  if (n_pools < 1 || n_pools > kMaxPools)
    return fail(n_pools > kMaxPools ? RC_ERR_UNSUPPORTED : RC_ERR_INVALID_ARG,
                "n_pools=%d (1..%d)", n_pools, kMaxPools);
  if (!pools || !segs || !k_fresh || !v_fresh)
    return fail(RC_ERR_INVALID_ARG, "pools, segs, k_fresh and v_fresh must be non-NULL");
  if (S < 1) return fail(RC_ERR_INVALID_ARG, "S=%d must be >= 1", S);
  if (S > kPagedMaxSegments)
    return fail(RC_ERR_UNSUPPORTED, "S=%d exceeds %d segments", S, kPagedMaxSegments);
  if (shape->N > kMaxSelectN) return fail(RC_ERR_UNSUPPORTED, "N=%d exceeds %d", shape->N, kMaxSelectN);
  if ((rope_cos == nullptr) != (rope_sin == nullptr))
    return fail(RC_ERR_INVALID_ARG, "rope_cos and rope_sin must both be given or both be NULL");
  if (rope_cos && max_pos < shape->N)
    return fail(RC_ERR_INVALID_ARG, "max_pos=%d < N=%d", max_pos, shape->N);
  if (shape->dtype != RC_BF16) return fail(RC_ERR_UNSUPPORTED, "paged attention is implemented for bf16");
  Paged pg{};
  pg.pools.n = n_pools;
  for (int p = 0; p < n_pools; ++p) {
    if (!pools[p].k || !pools[p].v || pools[p].num_blocks < 1 || pools[p].block_len < 1)
      return fail(RC_ERR_INVALID_ARG, "pool %d: NULL tensor or empty shape", p);
    pg.pools.k[p] = static_cast<const char*>(pools[p].k);
    pg.pools.v[p] = static_cast<const char*>(pools[p].v);
    pg.pools.num_blocks[p] = pools[p].num_blocks;
    pg.pools.block_len[p] = pools[p].block_len;
  }
  pg.segs = reinterpret_cast<const int4*>(segs);
  pg.S = S;
  pg.cos_t = rope_cos;
  pg.sin_t = rope_sin;
  pg.max_pos = rope_cos ? max_pos : 0;
  return attention_impl(shape, q, rows, R, k_fresh, v_fresh, scale, out, nullptr, &pg, stream,
                        "rc_paged_attention");
}
