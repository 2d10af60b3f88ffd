/*
 * rcllm.h -- C ABI of the MI355X (gfx950) selective-prefill library for one
 * transformer attention layer, after RcLLM (arXiv 2605.07443).
 *
 * The paper reuses precomputed KV blocks of user histories and candidate
 * items at arbitrary, non-prefix positions of a recommendation prompt and
 * repairs the reuse by recomputing only a few "heavy hitter" tokens
 * (Sec. III-C.2 and III-C.3). One layer of that prefill is four calls:
 *
 *   rc_kv_assemble          (i)  assembly: gather K/V rows of pool blocks
 *                                through a segment table, with
 *                           (ii) alignment: RoPE re-rotation of cached keys
 *                                fused into the gather
 *   rc_rerope               (ii) alignment as a standalone in-place pass
 *   rc_select_tokens        Eq. (3) deviation score (K only, lambda = 1),
 *                           deterministic top-k of cached tokens, and
 *                           (iii) correction: heavy hitters get fresh K/V
 *   rc_selective_attention  Eq. (1) causal GQA attention for the selected
 *                           query rows over the whole assembled context,
 *                           or for every row (Full-Recompute, Sec. IV-A)
 *
 * Selection by the full score of Eq. (3) (the first layer computed in full):
 *
 *   rc_selective_attention_lse  the same attention, also writing each row's
 *                               log-sum-exp
 *   rc_attention_mass           attention weight each token receives in the
 *                               full first layer (the ||A_i||_1 term)
 *   rc_select_tokens_eq3        Eq. (3) score with lambda, K and V divergence
 *                               (dropped for item blocks), separate history
 *                               and item budgets, and the correction (iii)
 *
 * Several layers (the first computed in full, later ones recomputing only the
 * selected rows, Sec. III-C.2b), with random-weight decoder layers:
 *
 *   rc_gemm_bf16                Y = X W^T (+ residual) projections
 *   rc_rmsnorm                  RMSNorm of rows
 *   rc_qkv_rope                 split a QKV projection, rotate q and k to
 *                               their positions, write q/k/v at those
 *                               positions (the heavy-hitter update of a
 *                               cached layer)
 *   rc_silu_mul                 SwiGLU activation
 *   rc_gather_rows              rows of a [B, N, width] tensor by position
 *
 * Token-granular history (single-token prototypes) and host-resident pools:
 *
 *   rc_kv_gather_tokens         gather + alignment through a per-position
 *                               source map instead of segments; pool rows may
 *                               live in pinned host memory (read over PCIe
 *                               by the kernel, zero-copy)
 *
 * The same chain with the value rows taken by reference (only the key rows,
 * which the alignment rotates, are copied; Sec. III-C.2a):
 *
 *   rc_kv_assemble_vref         assembly + alignment of K, and a table of
 *                               value-row addresses (pool or fresh row)
 *   rc_select_tokens_vref       top-k and correction (iii): fresh K rows
 *                               copied, value entries redirected
 *   rc_selective_attention_vref the attention, reading V through the table
 *
 * Zero-copy variant and the local window:
 *
 *   rc_paged_attention          selective attention that reads K/V through
 *                               the segment table (no assembled copy),
 *                               aligning pool keys and taking fresh rows for
 *                               the recomputed positions while it stages them
 *   rc_segments_with_window     (host) the last W positions of every request
 *                               become fresh (recomputed) segments
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pointers are DEVICE pointers unless marked (host). The caller owns every
 *   buffer; the library never allocates, frees or keeps a pointer after the
 *   call returns. Buffers must stay valid until `stream` has run the work.
 * - Every compute call only enqueues kernels on `stream` (no host
 *   synchronisation). A NULL stream is the default stream.
 * - Layouts are row-major and token-major:
 *     pool K/V        [num_blocks, block_len, Hkv, D]
 *     fresh/assembled [B, N, Hkv, D]
 *     Q               [B, N, Hq, D]
 *     out             [B, R, Hq, D]
 *     segments        [B, S] of rc_segment
 *     RoPE tables     [max_pos, D/2] fp32 (cos and sin of pos * base^(-2j/D))
 * - Storage dtype is fp32 or bf16 (rc_dtype) for every K/V/Q/out tensor of a
 *   call; arithmetic is fp32 (attention accumulates in fp32; bf16 products on
 *   the matrix cores).
 * - Return value: RC_OK, or a negative rc_status. On failure nothing was
 *   enqueued and rc_last_error() holds a description.
 * - Supported: D in {64, 128}; Hq % Hkv == 0; for bf16 attention the group
 *   size Hq/Hkv must divide 128; N <= 16384 for rc_select_tokens; S <= 1024
 *   segments per request; at most 8 pools.
 * - Device-side contents (segment tables, block ids, row lists, deltas) cannot
 *   be checked without a synchronisation. Kernels bound-check them and skip
 *   what is out of range (the affected outputs are then unspecified) instead
 *   of reading or writing out of bounds.
 */
#ifndef RCLLM_H
#define RCLLM_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RC_OK = 0,
  RC_ERR_INVALID_ARG = -1, /* NULL pointer, inconsistent sizes, bad value */
  RC_ERR_UNSUPPORTED = -2, /* valid request outside the supported shapes */
  RC_ERR_HIP = -3          /* a HIP launch failed; see rc_last_error() */
} rc_status;

typedef enum { RC_F32 = 0, RC_BF16 = 1 } rc_dtype;

/* Problem shape of one call (host struct). */
typedef struct {
  int32_t B;     /* requests in the batch */
  int32_t N;     /* prompt length (tokens) of every request */
  int32_t Hq;    /* query heads */
  int32_t Hkv;   /* KV heads; q-head h uses KV head h / (Hq / Hkv) */
  int32_t D;     /* head dimension */
  int32_t dtype; /* rc_dtype */
} rc_shape;

/* One precomputed KV pool (host struct, device pointers): the offline item or
 * history KV store of Sec. III-B. Block b, token t, head h, dim d lives at
 * ((b * block_len + t) * Hkv + h) * D + d. Keys are stored rotated to their
 * block-local positions 0 .. block_len-1. */
typedef struct {
  const void* k;
  const void* v;
  int32_t num_blocks;
  int32_t block_len;
} rc_pool;

/* One segment of a request's prompt (the logical-to-physical block mapping of
 * Sec. III-A): positions [dst_start, dst_start + len) come from block `block`
 * of pool `pool`, token offsets 0 .. len-1, or, when pool < 0, are fresh
 * (instruction tokens and cache misses, always recomputed, Sec. III-C.2a).
 * A request's segments must tile [0, N) in increasing dst_start order. */
typedef struct {
  int32_t dst_start;
  int32_t len;
  int32_t pool;
  int32_t block;
} rc_segment;

/* Source of one position for the token-granular gather: history prototypes
 * are single tokens (Sec. III-B), so each cached position names its own pool
 * row. pool < 0: fresh. Otherwise row indexes the pool's rows
 * (num_blocks * block_len of them, [row, Hkv, D] contiguous) and the key is
 * rotated by delta (the position it is placed at minus the position it was
 * stored at; |delta| < max_pos). pad is ignored. */
typedef struct {
  int32_t pool;
  int32_t row;
  int32_t delta;
  int32_t pad;
} rc_token_src;

/* RoPE tables (host). Writes cos/sin of pos * base^(-2j/D) for pos in
 * [0, max_pos), j in [0, D/2), evaluated in fp64 and rounded once to fp32,
 * into host arrays cos_out/sin_out of max_pos * D/2 floats each. The caller
 * uploads them. Rotary encoding as cited for the alignment step
 * (Sec. III-C.3 (ii)); the pair (j, j + D/2) of each head is rotated
 * ("rotate-half" convention). Errors: INVALID_ARG for NULL outputs,
 * max_pos < 1, odd or non-positive D, base <= 0. */
int rc_rope_table(int32_t max_pos, int32_t D, double base, float* cos_out, float* sin_out);

/* Assembly and fused alignment (Sec. III-C.3 (i) and (ii); zero-copy block
 * retrieval of Sec. III-C.2a served from an HBM-resident pool).
 * For request b and position i in segment s = segs[b*S + s]:
 *   fresh segment: K_asm[b,i] = K_fresh[b,i], V_asm[b,i] = V_fresh[b,i]
 *   pool segment:  K_asm[b,i] = R(dst_start) pool.k[block][i - dst_start]
 *                  V_asm[b,i] = pool.v[block][i - dst_start]
 * where R(delta) rotates every head's pairs (j, j+D/2) by delta * theta_j:
 *   x' = x*c - y*s, y' = x*s + y*c in fp32 (no fused multiply-add), c and s
 *   from row delta of the tables, then rounded to the storage dtype (RNE).
 * Blocks are stored at block-local positions from 0, so the rotation that
 * moves a cached row to its absolute position is delta = dst_start.
 * rope_cos/rope_sin NULL: plain gather, no rotation (then max_pos is
 * ignored); otherwise both must be given with max_pos >= N.
 * pools: host array of n_pools rc_pool (1..8). segs: device [B, S].
 * k_fresh/v_fresh: device [B, N, Hkv, D]; rows of fresh segments are copied.
 * k_asm/v_asm: device [B, N, Hkv, D] outputs (must not alias inputs); both
 * NULL with scores_out given: score only (nothing is assembled or stored).
 * scores_out: NULL, or device [B, N] fp32: the same pass then also reads the
 * fresh K row of every cached position and writes the deviation score of
 * Eq. (3) (M = K, lambda = 1) of the row it produced, exactly as
 * rc_select_tokens step 1 defines it (fp32 accumulation; 0 at fresh
 * positions), so that rc_select_tokens can take it as scores_in. Scoring
 * needs a key row (Hkv * D * element size) of at most 8192 bytes.
 * Errors: INVALID_ARG for NULL pointers, bad shape, bad pool, S < 1 or
 * max_pos < N with tables given; UNSUPPORTED for D, dtype, S > 1024, or a
 * key row above 8192 bytes with scores_out. */
int rc_kv_assemble(const rc_shape* shape, const rc_pool* pools, int32_t n_pools,
                   const rc_segment* segs, int32_t S, const void* k_fresh, const void* v_fresh,
                   const float* rope_cos, const float* rope_sin, int32_t max_pos, void* k_asm,
                   void* v_asm, float* scores_out, hipStream_t stream);

/* rc_kv_assemble with the value rows taken by reference (Sec. III-C.3 (i)
 * and (ii); the zero-copy retrieval of Sec. III-C.2a applied to V, which the
 * alignment leaves unchanged): K_asm and scores_out exactly as rc_kv_assemble
 * writes them, and instead of V_asm
 *   v_ref[b*N + i] = byte address of the V row [Hkv, D] that rc_kv_assemble
 *                    would copy to V_asm[b,i]: pool.v[block][i - dst_start]
 *                    for a pool segment, V_fresh[b,i] for a fresh one, and
 *                    V_fresh[b,i] for a position no valid segment covers.
 * v_ref: device [B, N] uint64, must not alias an input; the table refers to
 * the pools and to v_fresh, which must stay allocated and unchanged while it
 * is used. k_asm and v_ref are required (no score-only form).
 * Errors: those of rc_kv_assemble; UNSUPPORTED for S > 64 or a key row
 * (Hkv * D * element size) that is not 32 bytes times a power of two, or is
 * larger than 2 KiB. */
int rc_kv_assemble_vref(const rc_shape* shape, const rc_pool* pools, int32_t n_pools,
                        const rc_segment* segs, int32_t S, const void* k_fresh,
                        const void* v_fresh, const float* rope_cos, const float* rope_sin,
                        int32_t max_pos, void* k_asm, uint64_t* v_ref, float* scores_out,
                        hipStream_t stream);

/* Standalone alignment (Sec. III-C.3 (ii)), in place: K[b,i] <- R(delta[b,i])
 * K[b,i] with the same fp32 operation order as rc_kv_assemble; a negative
 * delta uses cos(|delta|) and -sin(|delta|); rows with delta == 0 are not
 * touched. k: device [B, N, Hkv, D]; delta: device [B, N] int32 with
 * |delta| < max_pos (rows outside are skipped); tables device
 * [max_pos, D/2]. Hq in the shape is unused (may be any value >= 1).
 * Errors: INVALID_ARG for NULL pointers, bad shape, max_pos < 1;
 * UNSUPPORTED for D or dtype. */
int rc_rerope(const rc_shape* shape, void* k, const int32_t* delta, const float* rope_cos,
              const float* rope_sin, int32_t max_pos, hipStream_t stream);

/* Heavy-hitter selection and correction (Sec. III-C.2b, Eq. (3) with M = K
 * and lambda = 1; Sec. III-C.3 (iii)).
 * 1. Score: unless scores_in is given, d[b,i] = sum over h < Hkv, j < D of
 *    |K_fresh[b,i,h,j] - K_asm[b,i,h,j]|, accumulated in fp32, for every
 *    position (0 at fresh positions, whose assembled rows are fresh), written
 *    to scores_out [B, N] (required when scores_in is NULL; optional else).
 * 2. Select: the k cached positions (not in a fresh segment) with the largest
 *    score -- NaN above +inf above every finite value, ties to the lower
 *    position -- together with the n_fresh fresh positions, in ascending
 *    order: rows [B, n_fresh + k] int32. Bit-exact for given scores.
 * 3. Patch (patch != 0): K_asm/V_asm rows of the k selected cached positions
 *    are overwritten with K_fresh/V_fresh rows.
 * n_fresh is the number of fresh positions of every request. It is an
 * argument because the segment table lives on the device and the row count
 * R = n_fresh + k must be known on the host to size `rows` without a
 * synchronisation. A request whose table disagrees with it is marked in its
 * row list instead of being reported here (the library cannot read the table
 * without a synchronisation): fewer fresh positions leave the unfilled tail
 * of its list at -1, more fresh positions drop the tail and set the last
 * entry to -1. rc_selective_attention turns a -1 row into NaN outputs.
 * Requires 0 <= k <= N - n_fresh; rows may be NULL when n_fresh + k == 0.
 * Hq in the shape is unused.
 * Errors: INVALID_ARG for NULL pointers, bad shape, k or n_fresh out of
 * range; UNSUPPORTED for D, dtype, N > 16384, S > 1024. */
int rc_select_tokens(const rc_shape* shape, const rc_segment* segs, int32_t S, int32_t n_fresh,
                     int32_t k, const void* k_fresh, const void* v_fresh, void* k_asm,
                     void* v_asm, const float* scores_in, float* scores_out, int32_t* rows,
                     int32_t patch, hipStream_t stream);

/* rc_select_tokens with patch = 1 over a value-reference table (Sec.
 * III-C.3 (iii)): scores, rows and K_asm exactly as rc_select_tokens writes
 * them, and for every selected cached position i of request b
 *   v_ref[b*N + i] = byte address of V_fresh[b,i]
 * instead of a copy of that row (other entries are left as they are).
 * v_ref: device [B, N] uint64 from rc_kv_assemble_vref.
 * Errors: those of rc_select_tokens with patch = 1. */
int rc_select_tokens_vref(const rc_shape* shape, const rc_segment* segs, int32_t S,
                          int32_t n_fresh, int32_t k, const void* k_fresh, const void* v_fresh,
                          void* k_asm, uint64_t* v_ref, const float* scores_in,
                          float* scores_out, int32_t* rows, hipStream_t stream);

/* Selective attention (Eq. (1); Sec. III-C.2b: exact attention recomputed for
 * the selected rows over the full assembled context).
 * For r < R, p = rows[b*R + r] (or p = r when rows is NULL: Full-Recompute
 * over all N rows, then R must equal N), q-head h, KV head g = h/(Hq/Hkv):
 *   out[b,r,h] = sum_{j<=p} softmax_j(scale * Q[b,p,h] . K[b,j,g]) V[b,j,g]
 * fp32 accumulation and online softmax; bf16 inputs use the matrix cores.
 * q: [B, N, Hq, D]; rows: [B, R] int32, ascending within a request (any
 * order is correct, ascending is fastest); k, v: [B, N, Hkv, D];
 * out: [B, R, Hq, D]. A listed row outside [0, N) (for instance the -1
 * that rc_select_tokens writes for a request whose segment table disagrees
 * with n_fresh) makes its output row NaN; no memory outside the tensors is
 * read.
 * Errors: INVALID_ARG for NULL pointers, bad shape, R < 0, R != N without
 * rows, non-finite or non-positive scale; UNSUPPORTED for D, dtype, or a
 * bf16 group size that does not divide 128. R == 0 enqueues nothing (out may
 * then be NULL). */
int rc_selective_attention(const rc_shape* shape, const void* q, const int32_t* rows, int32_t R,
                           const void* k, const void* v, float scale, void* out,
                           hipStream_t stream);

/* Attention as rc_selective_attention that also writes, for every row r and
 * q-head h, the natural log-sum-exp of the row's scaled causal scores,
 *   lse[b,r,h] = ln sum_{j<=p} exp(scale * Q[b,p,h] . K[b,j,g]),
 * into lse: device [B, R, Hq] fp32 (fp32 sums of the unrounded exponentials).
 * With rows NULL (every row of the first layer, Sec. III-C.2b) this is the
 * input rc_attention_mass takes. A row outside [0, N) makes its lse entries
 * NaN, like its outputs. Errors: those of rc_selective_attention, and
 * INVALID_ARG for a NULL lse with R > 0. */
int rc_selective_attention_lse(const rc_shape* shape, const void* q, const int32_t* rows,
                               int32_t R, const void* k, const void* v, float scale, void* out,
                               float* lse, hipStream_t stream);

/* Attention as rc_selective_attention with the value rows taken by
 * reference (Eq. (1); the gather of Sec. III-C.3 (i) then need not copy V):
 * v_ref: device [B, N] of byte addresses, entry b*N + j the address of the
 * V row [Hkv, D] that position j of request b uses (as written by
 * rc_kv_assemble_vref and redirected by rc_select_tokens_vref). Outputs are
 * bit-identical to rc_selective_attention over the V tensor those rows
 * form. Every entry must address a readable V row: entries are not checked.
 * bf16 with D = 128 only. Errors: those of rc_selective_attention;
 * UNSUPPORTED for another dtype or D. */
int rc_selective_attention_vref(const rc_shape* shape, const void* q, const int32_t* rows,
                                int32_t R, const void* k, const uint64_t* v_ref, float scale,
                                void* out, hipStream_t stream);

/* Attention-mass term of Eq. (3) (Sec. III-C.2b: the first layer is computed
 * in full and a token's importance includes the attention weight it
 * receives). For KV group g and position j of request b:
 *   mass[b,g,j] = sum over q-heads h with h / (Hq/Hkv) == g, rows p in [j, N) of
 *                 exp(scale * Q[b,p,h] . K[b,j,g] - lse[b,p,h])
 * i.e. the softmax weights of key j summed over the group's rows and heads;
 * sum_g mass[b,g,j] is ||A_j||_1. q: [B, N, Hq, D]; k: [B, N, Hkv, D] (the
 * fresh first-layer keys); lse: [B, N, Hq] from rc_selective_attention_lse
 * with rows NULL and the same scale; mass: device [B, Hkv, N] fp32 output,
 * every entry written. Deterministic (no atomics); fp32 accumulation, bf16
 * products on the matrix cores.
 * Errors: INVALID_ARG for NULL pointers, bad shape, non-finite or
 * non-positive scale; UNSUPPORTED for D, dtype, or a bf16 group size that
 * does not divide 128. */
int rc_attention_mass(const rc_shape* shape, const void* q, const void* k, const float* lse,
                      float scale, float* mass, hipStream_t stream);

/* Heavy-hitter selection by the full score of Eq. (3), with separate budgets
 * for history and item tokens (recompute ratios r_rev and r_item, Sec. IV-A),
 * and correction (Sec. III-C.3 (iii)).
 * 1. Score: unless scores_in is given, for every position i of request b
 *      S[b,i] = (1 - lambda) sum_g mass[b,g,i] + lambda div[b,i]
 *    with div the L1 distance between the fresh and assembled rows of K plus
 *    that of V (Hkv * D entries each, fp32 accumulation), except for
 *    positions in blocks of a pool whose bit is set in item_pool_mask: their
 *    cached block is a lexical match and div is dropped (Sec. III-C.2b).
 *    Written to scores_out [B, N] (required when scores_in is NULL).
 *    mass: [B, Hkv, N] from rc_attention_mass; lambda in [0, 1].
 * 2. Select: among cached positions of pools outside item_pool_mask
 *    (history) the k_hist largest scores, among those of pools in it (items)
 *    the k_item largest -- NaN above +inf above every finite value, ties to
 *    the lower position -- together with the n_fresh fresh positions, in
 *    ascending order: rows [B, n_fresh + k_hist + k_item] int32. Bit-exact
 *    for given scores. A budget above its class's count in some request
 *    takes the whole class and leaves the unfilled tail of that request's
 *    row list at -1 (n_fresh disagreeing with the table is marked as in
 *    rc_select_tokens).
 * 3. Patch (patch != 0): K_asm/V_asm rows of the selected cached positions
 *    get the K_fresh/V_fresh rows.
 * k_fresh/v_fresh/k_asm/v_asm: [B, N, Hkv, D]. Hq in the shape is unused.
 * Errors: INVALID_ARG for NULL pointers, bad shape, budgets or n_fresh out
 * of range, lambda outside [0, 1], lambda = 1 with k_item > 0 (item tokens
 * have no divergence term, so every item score would be 0 and the item
 * budget would take the lowest positions instead of a ranking), mask bits
 * beyond pool 7; UNSUPPORTED for D, dtype, N > 16384, S > 1024. */
int rc_select_tokens_eq3(const rc_shape* shape, const rc_segment* segs, int32_t S,
                         int32_t n_fresh, uint32_t item_pool_mask, float lambda, int32_t k_hist,
                         int32_t k_item, const float* mass, const void* k_fresh,
                         const void* v_fresh, void* k_asm, void* v_asm, const float* scores_in,
                         float* scores_out, int32_t* rows, int32_t patch, hipStream_t stream);

/* Token-granular assembly (Sec. III-B history prototypes are single tokens;
 * Sec. III-C.3 (i) and (ii)). For request b and position i, m = map[b*N + i]:
 *   m.pool < 0:  K_asm[b,i] = K_fresh[b,i], V_asm[b,i] = V_fresh[b,i]
 *   otherwise:   K_asm[b,i] = R(m.delta) pool.k[row m.row], V_asm[b,i] = pool.v[row m.row]
 * with R and its fp32 operation order as in rc_kv_assemble (negative deltas
 * rotate by cos(|d|), -sin(|d|)); rope tables NULL: no rotation. Pool rows
 * may be in device memory or in pinned host memory (hipHostMalloc), which
 * the kernel reads directly over PCIe; run such a gather on its own stream
 * to overlap the transfer with compute that does not need the pool (the
 * first layer in full, Sec. III-C.3). scores_out (optional, [B, N] fp32):
 * the K deviation of Eq. (3) as in rc_kv_assemble. map: device [B, N]
 * rc_token_src. Entries naming a missing pool or a row out of range leave
 * the position's output unspecified (not read out of bounds).
 * max_workgroups: 0 = one workgroup per block of positions (fastest alone);
 * > 0 = at most about that many workgroups (at least one per request), each
 * looping over position blocks -- for a gather from host memory beside
 * compute, so that it occupies few compute units while it waits on PCIe.
 * Errors: INVALID_ARG for NULL pointers, bad shape or pools, aliasing
 * outputs, one table without the other, max_workgroups < 0; UNSUPPORTED for
 * D, dtype, a key row above 8192 bytes with scores_out. */
int rc_kv_gather_tokens(const rc_shape* shape, const rc_pool* pools, int32_t n_pools,
                        const rc_token_src* map, const void* k_fresh, const void* v_fresh,
                        const float* rope_cos, const float* rope_sin, int32_t max_pos,
                        void* k_asm, void* v_asm, float* scores_out, int32_t max_workgroups,
                        hipStream_t stream);

/* Zero-copy selective attention (the logical-to-physical block mapping of
 * Sec. III-A applied inside attention; Sec. III-C.2b, III-C.3 (i)-(iii) and
 * Eq. (1) without an assembled K/V copy). Computes exactly what
 *   rc_kv_assemble (with the tables) -> patch of every listed row ->
 *   rc_selective_attention
 * computes, bit for bit, but each key row is fetched while its tile is
 * staged: position j of request b reads the fresh K/V row if j lies in a
 * fresh segment or is itself listed in rows (a recomputed heavy hitter),
 * else the pool row pool.k/v[block][j - dst_start], whose key is rotated by
 * dst_start in fp32 (the gather's operation order) when tables are given.
 * rows: [B, R] int32 (required); q: [B, N, Hq, D]; k_fresh, v_fresh:
 * [B, N, Hkv, D]; pools/segs as for rc_kv_assemble; out: [B, R, Hq, D].
 * Scores for the selection can be taken without an assembled copy by
 * rc_kv_assemble with k_asm = v_asm = NULL.
 * Errors: those of rc_selective_attention; INVALID_ARG for NULL
 * pools/segs/fresh tensors, bad pools, max_pos < N with tables;
 * UNSUPPORTED for fp32 storage, S > 64 segments, N > 16384. */
int rc_paged_attention(const rc_shape* shape, const void* q, const int32_t* rows, int32_t R,
                       const rc_pool* pools, int32_t n_pools, const rc_segment* segs, int32_t S,
                       const void* k_fresh, const void* v_fresh, const float* rope_cos,
                       const float* rope_sin, int32_t max_pos, float scale, void* out,
                       hipStream_t stream);

/* Local sliding window (host; Sec. III-C.2b recomputes the heavy hitters and
 * the local sliding window). Rewrites the segment tables segs_in [B, S]
 * (host) so that positions [N - W, N) of every request are fresh: segments
 * starting before N - W are kept (the one crossing it is cut there), then the
 * window follows as fresh segments, split into single-token pieces plus one
 * remainder where needed so that every request has the same count S_out
 * (<= S + 1). segs_out: host array of at least B * S_cap entries, written as
 * [B, S_out]. W = 0 copies the tables. Errors: INVALID_ARG for NULL
 * pointers, tables that do not tile [0, N) in order, W outside [0, N), a
 * window shorter than the pieces it needs, S_cap < S_out. */
int rc_segments_with_window(const rc_segment* segs_in, int32_t B, int32_t S, int32_t N,
                            int32_t W, rc_segment* segs_out, int32_t S_cap, int32_t* S_out);

/* Projection of a decoder layer on the matrix cores:
 *   y[m, j] = sum_i x[m, i] w[j, i] (+ residual[m, j]),  m < M, j < n, i < k
 * x: [M, k], w: [n, k], residual (optional) and y: [M, n]; all bf16 row-major
 * device tensors; fp32 accumulation, one rounding to bf16 (after adding the
 * residual in fp32). Deterministic. y must not overlap x, w or residual: a
 * short row tail (fewer than 256 rows after whole 256-row tiles) may be
 * computed by split-K with its fp32 partial sums kept in the first rows of y
 * until those rows are written, so the call allocates nothing.
 * Errors: INVALID_ARG for NULL pointers, M < 0, n < 1, k not a positive
 * multiple of 8, y overlapping x, w or residual. */
int rc_gemm_bf16(int64_t M, int32_t n, int32_t k, const void* x, const void* w,
                 const void* residual, void* y, hipStream_t stream);

/* RMSNorm of M rows of width H (bf16 device tensors x, y [M, H], gamma [H]):
 *   y = x / sqrt(mean(x^2) + eps) * gamma   (fp32 statistics, RNE to bf16).
 * Errors: INVALID_ARG for NULL pointers, H not a positive multiple of 8,
 * eps negative or not finite; UNSUPPORTED for H > 8192. */
int rc_rmsnorm(int32_t M, int32_t H, const void* x, const void* gamma, float eps, void* y,
               hipStream_t stream);

/* Split projected rows into q, k, v and place them at their positions
 * (Sec. III-C.2b: a later layer recomputes the selected rows; their fresh
 * K/V replace the cached rows, Sec. III-C.3 (iii)). Row m = b*R + r of qkv
 * ([B*R, (Hq + 2 Hkv) D] bf16: q heads, then k heads, then v heads) belongs
 * to position p = rows[b*R + r] (p = r when rows is NULL, then R = N); q and
 * k heads are rotated by p with the tables (rotate-half pairs, the fp32
 * operation order of rc_kv_assemble; no tables: no rotation) and written to
 * q_out [B, N, Hq, D], k_out / v_out [B, N, Hkv, D] at position p. Positions
 * outside [0, N) are skipped. bf16 only.
 * Errors: INVALID_ARG for NULL pointers, bad shape, rows NULL with R != N,
 * one table without the other, max_pos < N; UNSUPPORTED for fp32, D. */
int rc_qkv_rope(const rc_shape* shape, const void* qkv, const int32_t* rows, int32_t R,
                const float* rope_cos, const float* rope_sin, int32_t max_pos, void* q_out,
                void* k_out, void* v_out, hipStream_t stream);

/* SwiGLU activation: out[m, i] = silu(gu[m, i]) * gu[m, I + i] for m < M,
 * i < I (gate_up: [M, 2I], out: [M, I], bf16; fp32 math). Errors:
 * INVALID_ARG for NULL pointers, M < 0, I not a positive multiple of 8. */
int rc_silu_mul(int64_t M, int32_t I, const void* gate_up, void* out, hipStream_t stream);

/* dst[b, r] = src[b, rows[b*R + r]] for rows of row_bytes bytes (a multiple
 * of 16): src [B, Nsrc, row], dst [B, R, row]. Positions outside [0, Nsrc)
 * leave their destination row untouched. Errors: INVALID_ARG for NULL
 * pointers or bad sizes. */
int rc_gather_rows(int32_t B, int32_t Nsrc, int32_t R, int32_t row_bytes, const void* src,
                   const int32_t* rows, void* dst, hipStream_t stream);

/* Static description of a status code. */
const char* rc_status_string(int status);

/* Description of the last failure on the calling thread ("" if none). */
const char* rc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RCLLM_H */
