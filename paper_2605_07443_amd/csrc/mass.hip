// Attention-mass term of the importance score, Eq. (3) (RcLLM, arXiv
// 2605.07443, Sec. III-C.2b): the first layer is computed in full, and token
// j's term is the L1 norm of the attention weights it receives there,
//   mass[b, g, j] = sum over q-heads h of KV group g, sum over rows p >= j of
//                   exp(scale * q[b,p,h] . k[b,j,g] - lse[b,p,h]),
// with lse the natural log-sum-exp of row p (written by the full attention
// pass). sum_g mass[b, g, j] is ||A_j||_1.
//
// bf16 path (matrix cores, v_mfma_f32_16x16x32_bf16), key-stationary:
//   * A workgroup owns 256 keys of one (request, KV group); each of its 4
//     waves keeps the K fragments of 64 keys in registers (A operand of
//     S^T = K Q^T) for the whole kernel.
//   * The group's query vectors (G heads x positions, from the block's first
//     position on) stream through LDS in double-buffered tiles of 128 with
//     their lse. Every wave multiplies its keys with every tile, turns the
//     scores into weights and adds them to per-lane key sums.
//   * A tile's 8 blocks of 16 query vectors are software-pipelined: the
//     scores of block nb + 1 are issued on the matrix cores while the vector
//     ALU turns block nb into weights (interleaved one product to three
//     vector instructions), with two score sets in registers.
//   * Each key's sum is finished inside one wave (16-lane shuffles), so no
//     atomics are needed and the result is deterministic.
//   * Workgroups of one group run on one XCD (ids are dealt round-robin over
//     the 8 XCDs), longest (earliest) key blocks first.
// fp32 path: one thread per key, fp32 FMA on the vector ALUs.
#include <cmath>
#include <type_traits>

#include "rc_common.h"

namespace rc {
namespace {

constexpr int kMassThreads = 256;
constexpr int kMassKeys = 256;  // keys per workgroup, 64 per wave
constexpr int kQV = 128;        // query vectors per staged tile
constexpr int kMassXcds = 8;

using u32x4 = uint32_t __attribute__((ext_vector_type(4)));

template <int I, int M, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < M) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, M>(f);
  }
}

// Q tile rows padded to 16 mod 256 bytes: the B-operand reads (16 bytes from
// 16 consecutive rows per quarter-wave) are then conflict-free. Declared
// 16-byte aligned so that those reads and the staging stores are single
// 16-byte LDS instructions (with the 4-byte alignment of the members alone
// each is split into two 8-byte halves).
template <int D>
struct alignas(16) MassSmem {
  uint16_t q[2][kQV][D + 8];
  float lse2[2][kQV];  // lse * log2(e); +inf for padding vectors (weight 0)
};

template <int D>
__global__ __launch_bounds__(kMassThreads) __attribute__((amdgpu_waves_per_eu(2)))
void mass_bf16_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                      const float* __restrict__ lse, int N, int Hq, int Hkv, int G,
                      int g_shift, float scale_log2e, float* __restrict__ mass, int n_kblk,
                      int n_groups, int gpx) {
  constexpr int DC = D / 32;                       // 32-wide d chunks
  constexpr int UPR = D / 8;                       // 16-byte units per query row
  constexpr int QU = kQV * UPR / kMassThreads;     // staged units per thread
  constexpr int QSTEP = kMassThreads / UPR;        // rows between a thread's units
  constexpr int NB = kQV / 16;                     // 16-vector blocks per tile
  __shared__ MassSmem<D> sm;

  // ---- work item: XCD-major, longest key blocks first
  const int hw = blockIdx.x;
  const int xcd = hw % kMassXcds;
  const int slot = hw / kMassXcds;
  const int kblk = slot / gpx;
  const int grp = (slot - kblk * gpx) * kMassXcds + xcd;
  if (kblk >= n_kblk || grp >= n_groups) return;
  const int b = grp / Hkv;
  const int g = grp - b * Hkv;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c16 = lane & 15;
  const int q4 = lane >> 4;
  const int QP = kQV / G;                 // positions per tile
  const int p_begin = kblk * kMassKeys;   // first row that sees a key of the block
  const int j0 = p_begin + wave * 64;     // this wave's first key
  const int n_qt = (N - p_begin + QP - 1) / QP;

  // ---- K fragments (A operand): lane holds key j0 + kb*16 + c16, dims dc*32 + q4*8 ..
  const size_t kstride = static_cast<size_t>(Hkv) * D;
  bf16x8 kf[4][DC];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    const int j = j0 + kb * 16 + c16;
    const uint16_t* krow = k + (static_cast<size_t>(b) * N + min(j, N - 1)) * kstride +
                           static_cast<size_t>(g) * D;
#pragma unroll
    for (int dc = 0; dc < DC; ++dc) {
      const u32x4 w = j < N ? *reinterpret_cast<const u32x4*>(krow + dc * 32 + q4 * 8)
                            : u32x4{0, 0, 0, 0};
      kf[kb][dc] = __builtin_bit_cast(bf16x8, w);
    }
  }

  // ---- query staging: vector m = (position p0 + m / G, head g*G + m % G)
  const size_t qstride = static_cast<size_t>(Hq) * D;
  u32x4 qreg[QU];
  float lreg = INFINITY;
  auto load_tile = [&](int t) {
    const int p0 = p_begin + t * QP;
#pragma unroll
    for (int i = 0; i < QU; ++i) {
      const int m = tid / UPR + i * QSTEP;
      const int col = (tid % UPR) * 8;
      const int p = p0 + m / G;
      const int h = g * G + m % G;
      qreg[i] = p < N ? *reinterpret_cast<const u32x4*>(q + (static_cast<size_t>(b) * N + p) * qstride +
                                                          static_cast<size_t>(h) * D + col)
                      : u32x4{0, 0, 0, 0};
    }
    if (tid < kQV) {
      const int p = p0 + tid / G;
      const int h = g * G + tid % G;
      lreg = p < N ? lse[(static_cast<size_t>(b) * N + p) * Hq + h] * 1.4426950408889634f
                   : INFINITY;
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < QU; ++i) {
      const int m = tid / UPR + i * QSTEP;
      const int col = (tid % UPR) * 8;
      *reinterpret_cast<u32x4*>(&sm.q[buf][m][col]) = qreg[i];
    }
    if (tid < kQV) sm.lse2[buf][tid] = lreg;
  };

  float acc[4][4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[kb][i] = 0.f;

  if (n_qt > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();
  if (n_qt > 1) load_tile(1);

  auto do_tile = [&](int t, auto mask_tag) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const int cur = t & 1;
    const int p0 = p_begin + t * QP;
    __builtin_amdgcn_s_setprio(1);
    // scores of block nb + 1 on the matrix cores while the vector ALU turns
    // block nb into weights (two score sets in flight)
    f32x4 sa[4], sb[4];
    auto scores = [&](f32x4 (&sc)[4], int nb) __attribute__((always_inline)) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) sc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        const bf16x8 bq = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(&sm.q[cur][nb * 16 + c16][dc * 32 + q4 * 8]));
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
          sc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kb][dc], bq, sc[kb], 0, 0, 0);
      }
    };
    auto weights = [&](f32x4 (&sc)[4], int nb) __attribute__((always_inline)) {
      const float l2 = sm.lse2[cur][nb * 16 + c16];
      const int pq = p0 + ((nb * 16 + c16) >> g_shift);  // position of this column's vector
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float w = __builtin_amdgcn_exp2f(fmaf(sc[kb][i], scale_log2e, -l2));
          if constexpr (MASK) w = (j0 + kb * 16 + q4 * 4 + i <= pq) ? w : 0.f;
          acc[kb][i] += w;
        }
    };
    auto interleave = [&]() __attribute__((always_inline)) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2 * DC, 0);
      static_for<0, 4 * DC>([&](auto) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
      });
    };
    scores(sa, 0);
#pragma unroll 1
    for (int nb = 0; nb < NB - 2; nb += 2) {
      scores(sb, nb + 1);
      weights(sa, nb);
      interleave();
      scores(sa, nb + 2);
      weights(sb, nb + 1);
      interleave();
    }
    scores(sb, NB - 1);
    weights(sa, NB - 2);
    interleave();
    weights(sb, NB - 1);
    __builtin_amdgcn_s_setprio(0);
    if (t + 1 < n_qt) {
      store_tile(cur ^ 1);
      if (t + 2 < n_qt) load_tile(t + 2);
    }
    __syncthreads();
  };

  // tiles wholly before this wave's keys add nothing; tiles that start at or
  // after its last key need no mask
  const int t_first = min(n_qt, (wave * 64) / QP);
  const int t_free = min(n_qt, (wave * 64 + 63 + QP - 1) / QP);
  int t = 0;
  for (; t < t_first; ++t) {  // keep the barrier rhythm of the other waves
    if (t + 1 < n_qt) {
      store_tile((t & 1) ^ 1);
      if (t + 2 < n_qt) load_tile(t + 2);
    }
    __syncthreads();
  }
  for (; t < t_free; ++t) do_tile(t, std::true_type{});
  for (; t < n_qt; ++t) do_tile(t, std::false_type{});

  // ---- finish each key's sum across the 16 query columns and store
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v = acc[kb][i];
      v += __shfl_xor(v, 1, 64);
      v += __shfl_xor(v, 2, 64);
      v += __shfl_xor(v, 4, 64);
      v += __shfl_xor(v, 8, 64);
      acc[kb][i] = v;
    }
  if (c16 == 0) {
    float* mrow = mass + (static_cast<size_t>(b) * Hkv + g) * N;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = j0 + kb * 16 + q4 * 4 + i;
        if (j < N) mrow[j] = acc[kb][i];
      }
  }
}

// fp32: one thread per (request, group, key), rows p >= j of the group's heads.
template <int D>
__global__ __launch_bounds__(256) void mass_f32_kernel(const float* __restrict__ q,
                                                       const float* __restrict__ k,
                                                       const float* __restrict__ lse, int N,
                                                       int Hq, int Hkv, float scale,
                                                       float* __restrict__ mass) {
  const int G = Hq / Hkv;
  const int g = blockIdx.y % Hkv;
  const int b = blockIdx.y / Hkv;
  const int j = blockIdx.x * 256 + threadIdx.x;
  const int jj = min(j, N - 1);
  float kr[D];
  const float* krow = k + ((static_cast<size_t>(b) * N + jj) * Hkv + g) * D;
#pragma unroll
  for (int d = 0; d < D; ++d) kr[d] = krow[d];
  float acc = 0.f;
  const int p_first = blockIdx.x * 256;  // uniform start; rows before j are masked
  for (int p = p_first; p < N; ++p) {
    for (int hh = 0; hh < G; ++hh) {
      const int h = g * G + hh;
      const float* qrow = q + ((static_cast<size_t>(b) * N + p) * Hq + h) * D;
      float dot = 0.f;
#pragma unroll
      for (int d = 0; d < D; ++d) dot = fmaf(qrow[d], kr[d], dot);
      const float w = expf(dot * scale - lse[(static_cast<size_t>(b) * N + p) * Hq + h]);
      acc += (j <= p) ? w : 0.f;
    }
  }
  if (j < N) mass[(static_cast<size_t>(b) * Hkv + g) * N + j] = acc;
}

}  // namespace
}  // namespace rc

extern "C" int rc_attention_mass(const rc_shape* shape, const void* q, const void* k,
                                 const float* lse, float scale, float* mass,
                                 hipStream_t stream) {
  using namespace rc;
  clear_error();
  if (int st = check_shape(shape, true)) return st;
  if (!q || !k || !lse || !mass) return fail(RC_ERR_INVALID_ARG, "q, k, lse and mass must be non-NULL");
  if (!(scale > 0.f) || !std::isfinite(scale))
    return fail(RC_ERR_INVALID_ARG, "scale must be finite and > 0");
  const int B = shape->B, N = shape->N, Hq = shape->Hq, Hkv = shape->Hkv, D = shape->D;
  const int G = Hq / Hkv;
  if (shape->dtype == RC_BF16) {
    if (kQV % G != 0) return fail(RC_ERR_UNSUPPORTED, "group size Hq/Hkv=%d must divide %d", G, kQV);
    const int n_kblk = (N + kMassKeys - 1) / kMassKeys;
    const int n_groups = B * Hkv;
    const int gpx = (n_groups + kMassXcds - 1) / kMassXcds;
    int g_shift = 0;  // G divides 128, so it is a power of two
    while ((1 << g_shift) < G) ++g_shift;
    const int64_t blocks = static_cast<int64_t>(kMassXcds) * gpx * n_kblk;
    if (blocks > 0x7fffffff) return fail(RC_ERR_UNSUPPORTED, "grid too large");
    const float scale_log2e = static_cast<float>(static_cast<double>(scale) * 1.4426950408889634);
    dim3 grid(static_cast<unsigned>(blocks));
    if (D == 128)
      hipLaunchKernelGGL(mass_bf16_kernel<128>, grid, dim3(kMassThreads), 0, stream,
                         static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), lse, N,
                         Hq, Hkv, G, g_shift, scale_log2e, mass, n_kblk, n_groups, gpx);
    else
      hipLaunchKernelGGL(mass_bf16_kernel<64>, grid, dim3(kMassThreads), 0, stream,
                         static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), lse, N,
                         Hq, Hkv, G, g_shift, scale_log2e, mass, n_kblk, n_groups, gpx);
  } else {
    if (static_cast<int64_t>(B) * Hkv > 65535) return fail(RC_ERR_UNSUPPORTED, "B*Hkv exceeds 65535");
    dim3 grid((N + 255) / 256, B * Hkv);
    if (D == 128)
      hipLaunchKernelGGL(mass_f32_kernel<128>, grid, dim3(256), 0, stream,
                         static_cast<const float*>(q), static_cast<const float*>(k), lse, N, Hq,
                         Hkv, scale, mass);
    else
      hipLaunchKernelGGL(mass_f32_kernel<64>, grid, dim3(256), 0, stream,
                         static_cast<const float*>(q), static_cast<const float*>(k), lse, N, Hq,
                         Hkv, scale, mass);
  }
  return check_launch("rc_attention_mass");
}
