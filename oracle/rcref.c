/*
 * rcref.c -- CPU oracle for the selective prefill of one attention layer in
 * RcLLM (arXiv 2605.07443): assembly of cached KV blocks, RoPE re-alignment,
 * heavy-hitter selection by K deviation, and causal attention recomputed only
 * for the selected query rows.
 *
 * TEST INFRASTRUCTURE ONLY. The test suite, the smoke check and the
 * benchmark's CPU-baseline leg are the only code that loads this library. The
 * GPU path never links, calls or falls back to it, and it includes no header
 * and shares no helper, table generator or constant with the GPU path.
 *
 * Style: plain loops in the order the paper states the steps, fp64
 * accumulation, no tiling, no fusion, no reordering beyond what each
 * definition states. OpenMP only splits independent outer iterations.
 * Build with -ffp-contract=off (no fused multiply-add) and without
 * -ffast-math: the RoPE step fixes its fp32 operation order so that it has one
 * exact answer.
 *
 * Storage dtypes: 0 = fp32, 1 = bf16 (stored as uint16 bit patterns).
 * Rounding to storage is round-to-nearest-even.
 *
 * Layouts (row-major, token-major):
 *   pool K/V     [num_blocks, block_len, Hkv, D]
 *   fresh / asm  [B, N, Hkv, D]
 *   Q            [B, N, Hq, D]
 *   out          [B, R, Hq, D]
 *   segments     [B, S, 4] int32 = {dst_start, len, pool, block}, pool = -1
 *                marks a fresh (always recomputed) segment
 *   rope tables  [max_pos, D/2] fp32
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* threads the OpenMP loops below use */
int rcref_num_threads(void) { return omp_get_max_threads(); }

/* ------------------------------------------------------------------ */
/* storage helpers                                                      */
/* ------------------------------------------------------------------ */

static float bf16_bits_to_f32(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

static uint16_t f32_to_bf16_bits(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) /* NaN: keep it a quiet NaN */
    return (uint16_t)((u >> 16) | 0x0040u);
  u += 0x7fffu + ((u >> 16) & 1u); /* round to nearest, ties to even */
  return (uint16_t)(u >> 16);
}

/* element e of a tensor of storage dtype `dt`, as an exact fp32 value */
static float load_el(const void* p, int dt, size_t e) {
  if (dt == 0) return ((const float*)p)[e];
  return bf16_bits_to_f32(((const uint16_t*)p)[e]);
}

static void store_el(void* p, int dt, size_t e, float v) {
  if (dt == 0)
    ((float*)p)[e] = v;
  else
    ((uint16_t*)p)[e] = f32_to_bf16_bits(v);
}

static size_t el_size(int dt) { return dt == 0 ? 4 : 2; }

/* ------------------------------------------------------------------ */
/* RoPE tables                                                          */
/* ------------------------------------------------------------------ */

/* Rotary position embedding (RoFormer, cited for the alignment step of the
 * end-to-end prefill pipeline, Sec. III-C.3). Pair (j, j + D/2) of a head is
 * rotated by the angle pos * base^(-2j/D). Angles and their cosine and sine
 * are evaluated in fp64 and rounded once to fp32. */
void rcref_rope_table(int max_pos, int D, double base, float* cos_tab, float* sin_tab) {
  int half = D / 2;
  for (int p = 0; p < max_pos; ++p) {
    for (int j = 0; j < half; ++j) {
      double inv_freq = pow(base, -2.0 * (double)j / (double)D);
      double theta = (double)p * inv_freq;
      cos_tab[(size_t)p * half + j] = (float)cos(theta);
      sin_tab[(size_t)p * half + j] = (float)sin(theta);
    }
  }
}

/* ------------------------------------------------------------------ */
/* Segment table                                                        */
/* ------------------------------------------------------------------ */

/* A prompt is Instruction + History + Items (Sec. II-A and Sec. IV-A); the
 * KV manager serves each part differently (Sec. III-C.2a): instruction tokens
 * and cache misses are computed fresh, history and item tokens come from
 * cached blocks. Segment s of request b covers [dst_start, dst_start + len). */
typedef struct {
  int32_t dst_start, len, pool, block;
} rcref_seg;

/* number of fresh positions of request b */
static int fresh_count(const rcref_seg* segs, int S, int b) {
  int F = 0;
  for (int s = 0; s < S; ++s)
    if (segs[(size_t)b * S + s].pool < 0) F += segs[(size_t)b * S + s].len;
  return F;
}

/* is position i of request b inside a fresh segment? */
static int is_fresh(const rcref_seg* segs, int S, int b, int i) {
  for (int s = 0; s < S; ++s) {
    const rcref_seg* g = &segs[(size_t)b * S + s];
    if (i >= g->dst_start && i < g->dst_start + g->len) return g->pool < 0;
  }
  return 1; /* not covered: treated as fresh (validated away by callers) */
}

/* ------------------------------------------------------------------ */
/* Step (i) Assembly and step (ii) Alignment                            */
/* ------------------------------------------------------------------ */

/* Rotate one head's key in place by position delta `delta` (may be negative:
 * a rotation by -d uses cos(d) and -sin(d)). The fp32 operation order is
 *   x' = fl(fl(x*c) - fl(y*s)),  y' = fl(fl(x*s) + fl(y*c))
 * followed by rounding to the storage dtype. */
static void rotate_head(void* k, int dt, size_t base_el, int D, int delta,
                        const float* cos_tab, const float* sin_tab) {
  int half = D / 2;
  int a = delta < 0 ? -delta : delta;
  for (int j = 0; j < half; ++j) {
    float c = cos_tab[(size_t)a * half + j];
    float s = sin_tab[(size_t)a * half + j];
    if (delta < 0) s = -s;
    float x = load_el(k, dt, base_el + j);
    float y = load_el(k, dt, base_el + j + half);
    float xc = x * c, ys = y * s, xs = x * s, yc = y * c;
    float nx = xc - ys;
    float ny = xs + yc;
    store_el(k, dt, base_el + j, nx);
    store_el(k, dt, base_el + j + half, ny);
  }
}

/* Assembly (Sec. III-C.3 step i; logical-to-physical block mapping of
 * Sec. III-A): position i of request b takes its K and V row from the pool
 * block its segment names, at block offset i - dst_start, or from the fresh
 * tensors for a fresh segment. With rope tables given, cached K rows are then
 * re-aligned (Sec. III-C.3 step ii): blocks are stored at block-local
 * positions starting at 0, so the row moves by delta = dst_start. */
void rcref_assemble(int B, int N, int Hkv, int D, int dt,
                    const void* const* pool_k, const void* const* pool_v,
                    const int32_t* pool_num_blocks, const int32_t* pool_block_len, int n_pools,
                    const int32_t* segs_raw, int S,
                    const void* k_fresh, const void* v_fresh,
                    const float* cos_tab, const float* sin_tab,
                    void* k_asm, void* v_asm) {
  const rcref_seg* segs = (const rcref_seg*)segs_raw;
  size_t row = (size_t)Hkv * D;
  size_t es = el_size(dt);
  (void)pool_num_blocks;
  (void)n_pools;
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b) {
    for (int s = 0; s < S; ++s) {
      const rcref_seg* g = &segs[(size_t)b * S + s];
      for (int t = 0; t < g->len; ++t) {
        int i = g->dst_start + t;
        size_t dst = ((size_t)b * N + i) * row;
        const char *src_k, *src_v;
        if (g->pool < 0) {
          src_k = (const char*)k_fresh + dst * es;
          src_v = (const char*)v_fresh + dst * es;
        } else {
          size_t src = ((size_t)g->block * pool_block_len[g->pool] + t) * row;
          src_k = (const char*)pool_k[g->pool] + src * es;
          src_v = (const char*)pool_v[g->pool] + src * es;
        }
        memcpy((char*)k_asm + dst * es, src_k, row * es);
        memcpy((char*)v_asm + dst * es, src_v, row * es);
        if (g->pool >= 0 && cos_tab && sin_tab) {
          for (int h = 0; h < Hkv; ++h)
            rotate_head(k_asm, dt, dst + (size_t)h * D, D, g->dst_start, cos_tab, sin_tab);
        }
      }
    }
  }
}

/* Token-granular assembly (Sec. III-B: history prototypes are single tokens;
 * Sec. III-C.3 steps i, ii). map[b, i] = {pool, row, delta, unused}: pool < 0
 * takes the fresh rows; otherwise the K and V rows are row `row` of the pool
 * (its rows counted across blocks), and the key is rotated by delta when
 * tables are given. */
void rcref_gather_tokens(int B, int N, int Hkv, int D, int dt,
                         const void* const* pool_k, const void* const* pool_v,
                         const int32_t* map, const void* k_fresh, const void* v_fresh,
                         const float* cos_tab, const float* sin_tab, void* k_asm, void* v_asm) {
  size_t row = (size_t)Hkv * D;
  size_t es = el_size(dt);
#pragma omp parallel for schedule(static)
  for (long bi = 0; bi < (long)B * N; ++bi) {
    const int32_t* m = map + (size_t)bi * 4;
    size_t dst = (size_t)bi * row;
    const char *src_k, *src_v;
    if (m[0] < 0) {
      src_k = (const char*)k_fresh + dst * es;
      src_v = (const char*)v_fresh + dst * es;
    } else {
      src_k = (const char*)pool_k[m[0]] + (size_t)m[1] * row * es;
      src_v = (const char*)pool_v[m[0]] + (size_t)m[1] * row * es;
    }
    memcpy((char*)k_asm + dst * es, src_k, row * es);
    memcpy((char*)v_asm + dst * es, src_v, row * es);
    if (m[0] >= 0 && m[2] != 0 && cos_tab && sin_tab)
      for (int h = 0; h < Hkv; ++h)
        rotate_head(k_asm, dt, dst + (size_t)h * D, D, m[2], cos_tab, sin_tab);
  }
}

/* Standalone alignment: rotate K[b, i] by delta[b, i]; delta 0 leaves the row
 * untouched (Sec. III-C.3 step ii). */
void rcref_rerope(int B, int N, int Hkv, int D, int dt, void* k, const int32_t* delta,
                  const float* cos_tab, const float* sin_tab) {
  size_t row = (size_t)Hkv * D;
#pragma omp parallel for schedule(static)
  for (long bi = 0; bi < (long)B * N; ++bi) {
    int d = delta[bi];
    if (d == 0) continue;
    for (int h = 0; h < Hkv; ++h)
      rotate_head(k, dt, (size_t)bi * row + (size_t)h * D, D, d, cos_tab, sin_tab);
  }
}

/* ------------------------------------------------------------------ */
/* Heavy-hitter selection (Sec. III-C.2b, Eq. (3))                      */
/* ------------------------------------------------------------------ */

/* Deviation term of the importance score, Eq. (3), restricted to M = K and
 * lambda = 1: d_i = sum over heads and dims of |K_new - K_cached| for token i
 * (an L1 norm over the token's Hkv*D key entries of this layer). Defined for
 * every position; at a fresh position the assembled row is the fresh row, so
 * d_i = 0 there. Accumulated in fp64, stored as fp32. */
void rcref_deviation(int B, int N, int Hkv, int D, int dt,
                     const void* k_fresh, const void* k_asm, float* scores) {
  size_t row = (size_t)Hkv * D;
#pragma omp parallel for schedule(static)
  for (long bi = 0; bi < (long)B * N; ++bi) {
    double acc = 0.0;
    for (size_t e = 0; e < row; ++e) {
      double a = (double)load_el(k_fresh, dt, (size_t)bi * row + e);
      double c = (double)load_el(k_asm, dt, (size_t)bi * row + e);
      acc += fabs(a - c);
    }
    scores[bi] = (float)acc;
  }
}

/* Total order on fp32 scores: larger key = larger score; +NaN ranks above
 * +inf, -NaN below -inf. */
static uint32_t score_key(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

typedef struct {
  uint32_t key;
  int32_t idx;
} cand_t;

/* heavier first; among equal scores the lower position first */
static int cand_cmp(const void* pa, const void* pb) {
  const cand_t* a = (const cand_t*)pa;
  const cand_t* b = (const cand_t*)pb;
  if (a->key != b->key) return a->key > b->key ? -1 : 1;
  return a->idx < b->idx ? -1 : (a->idx > b->idx ? 1 : 0);
}

/* Heavy hitters (Sec. III-C.2b): the k cached (non-fresh) positions with the
 * largest score, ties to the lower position. The recomputed query rows are the
 * fresh positions (always recomputed, Sec. III-C.2a) together with these k,
 * written in ascending order: rows[b, 0 .. F+k). Returns 0, or -1 if k
 * exceeds the number of cached positions of some request or the requests do
 * not share one fresh count F. */
int rcref_topk(int B, int N, const int32_t* segs_raw, int S, int k,
               const float* scores, int32_t* rows) {
  const rcref_seg* segs = (const rcref_seg*)segs_raw;
  int F = fresh_count(segs, S, 0);
  int R = F + k;
  int status = 0;
  for (int b = 1; b < B; ++b) /* every request must recompute the same count */
    if (fresh_count(segs, S, b) != F) return -1;
  cand_t* cand = (cand_t*)malloc(sizeof(cand_t) * (size_t)(N > 0 ? N : 1));
  unsigned char* take = (unsigned char*)malloc((size_t)(N > 0 ? N : 1));
  for (int b = 0; b < B; ++b) {
    int n = 0;
    for (int i = 0; i < N; ++i) {
      if (is_fresh(segs, S, b, i)) continue;
      cand[n].key = score_key(scores[(size_t)b * N + i]);
      cand[n].idx = i;
      ++n;
    }
    if (k > n) {
      status = -1;
      break;
    }
    qsort(cand, (size_t)n, sizeof(cand_t), cand_cmp);
    memset(take, 0, (size_t)N);
    for (int i = 0; i < N; ++i)
      if (is_fresh(segs, S, b, i)) take[i] = 1;
    for (int c = 0; c < k; ++c) take[cand[c].idx] = 1;
    int r = 0;
    for (int i = 0; i < N; ++i)
      if (take[i]) rows[(size_t)b * R + r++] = i;
  }
  free(cand);
  free(take);
  return status;
}

/* Heavy-hitter update (Sec. III-C.3 step iii): every selected cached position
 * gets its freshly computed K and V row. Fresh positions already hold fresh
 * rows after assembly. */
void rcref_patch(int B, int N, int Hkv, int D, int dt, const int32_t* segs_raw, int S,
                 const int32_t* rows, int R,
                 const void* k_fresh, const void* v_fresh, void* k_asm, void* v_asm) {
  const rcref_seg* segs = (const rcref_seg*)segs_raw;
  size_t row = (size_t)Hkv * D;
  size_t es = el_size(dt);
  for (int b = 0; b < B; ++b) {
    for (int r = 0; r < R; ++r) {
      int i = rows[(size_t)b * R + r];
      if (is_fresh(segs, S, b, i)) continue;
      size_t off = ((size_t)b * N + i) * row * es;
      memcpy((char*)k_asm + off, (const char*)k_fresh + off, row * es);
      memcpy((char*)v_asm + off, (const char*)v_fresh + off, row * es);
    }
  }
}

/* ------------------------------------------------------------------ */
/* Attention (Eq. (1)) for the recomputed rows                          */
/* ------------------------------------------------------------------ */

/* Causal scaled dot-product attention, Eq. (1), evaluated only for the query
 * rows listed in `rows` (Sec. III-C.2b: exact attention for the heavy hitters
 * over the full assembled context). Row p of q-head h attends keys 0..p of KV
 * head g = h / (Hq / Hkv) (grouped-query attention). rows == NULL means every
 * position 0..N-1 (the Full-Recompute baseline of Sec. IV-A). Scores, softmax
 * and the weighted sum are in fp64; the result is rounded once to the storage
 * dtype (via fp32). */
void rcref_attention(int B, int N, int Hq, int Hkv, int D, int dt,
                     const void* q, const int32_t* rows, int R,
                     const void* k, const void* v, double scale, void* out) {
  int group = Hq / Hkv;
  int nrows = rows ? R : N;
#pragma omp parallel
  {
    double* z = (double*)malloc(sizeof(double) * (size_t)N);
    double* acc = (double*)malloc(sizeof(double) * (size_t)D);
#pragma omp for collapse(2) schedule(dynamic, 4)
    for (int b = 0; b < B; ++b) {
      for (int r = 0; r < nrows; ++r) {
        int p = rows ? rows[(size_t)b * R + r] : r;
        for (int h = 0; h < Hq; ++h) {
          int g = h / group;
          size_t qoff = (((size_t)b * N + p) * Hq + h) * D;
          double m = -INFINITY;
          for (int j = 0; j <= p; ++j) {
            size_t koff = (((size_t)b * N + j) * Hkv + g) * D;
            double dot = 0.0;
            for (int d = 0; d < D; ++d)
              dot += (double)load_el(q, dt, qoff + d) * (double)load_el(k, dt, koff + d);
            z[j] = dot * scale;
            if (z[j] > m) m = z[j];
          }
          double denom = 0.0;
          for (int d = 0; d < D; ++d) acc[d] = 0.0;
          for (int j = 0; j <= p; ++j) {
            double w = exp(z[j] - m);
            denom += w;
            size_t voff = (((size_t)b * N + j) * Hkv + g) * D;
            for (int d = 0; d < D; ++d) acc[d] += w * (double)load_el(v, dt, voff + d);
          }
          size_t ooff = (((size_t)b * nrows + r) * Hq + h) * D;
          for (int d = 0; d < D; ++d) store_el(out, dt, ooff + d, (float)(acc[d] / denom));
        }
      }
    }
    free(z);
    free(acc);
  }
}

/* ------------------------------------------------------------------ */
/* The full importance score of Eq. (3)                                 */
/* ------------------------------------------------------------------ */

/* Natural log-sum-exp of each row of the first layer's scaled causal scores:
 * lse[b, p, h] = ln sum_{j <= p} exp(scale * q[b,p,h] . k[b,j,g]), g the KV
 * head of q-head h. The first layer is computed in full (Sec. III-C.2b), so
 * every position p = 0 .. N-1 is a row. fp64 throughout. */
void rcref_attention_lse(int B, int N, int Hq, int Hkv, int D, int dt,
                         const void* q, const void* k, double scale, double* lse) {
  int group = Hq / Hkv;
#pragma omp parallel
  {
    double* z = (double*)malloc(sizeof(double) * (size_t)N);
#pragma omp for collapse(2) schedule(dynamic, 4)
    for (int b = 0; b < B; ++b) {
      for (int p = 0; p < N; ++p) {
        for (int h = 0; h < Hq; ++h) {
          int g = h / group;
          size_t qoff = (((size_t)b * N + p) * Hq + h) * D;
          double m = -INFINITY;
          for (int j = 0; j <= p; ++j) {
            size_t koff = (((size_t)b * N + j) * Hkv + g) * D;
            double dot = 0.0;
            for (int d = 0; d < D; ++d)
              dot += (double)load_el(q, dt, qoff + d) * (double)load_el(k, dt, koff + d);
            z[j] = dot * scale;
            if (z[j] > m) m = z[j];
          }
          double sum = 0.0;
          for (int j = 0; j <= p; ++j) sum += exp(z[j] - m);
          lse[((size_t)b * N + p) * Hq + h] = m + log(sum);
        }
      }
    }
    free(z);
  }
}

/* Attention-mass term of Eq. (3). A_j collects the attention weights token j
 * receives in the first layer, computed in full: weight A[h, p, j] is entry j
 * of the softmax of row p of q-head h over keys 0..p (Eq. (1)), so token j is
 * weighted by every row p >= j of every q-head. Its L1 norm is the sum of
 * those weights (all are >= 0). The mass is returned per KV group g (the
 * q-heads h with h / (Hq/Hkv) = g): mass[b, g, j] = sum_{h in g} sum_{p >= j}
 * A[h, p, j], and ||A_j||_1 = sum_g mass[b, g, j]. fp64 throughout. */
void rcref_attention_mass(int B, int N, int Hq, int Hkv, int D, int dt,
                          const void* q, const void* k, double scale, double* mass) {
  int group = Hq / Hkv;
#pragma omp parallel
  {
    double* z = (double*)malloc(sizeof(double) * (size_t)N);
#pragma omp for collapse(2) schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
      for (int g = 0; g < Hkv; ++g) {
        double* col = mass + ((size_t)b * Hkv + g) * N;
        for (int j = 0; j < N; ++j) col[j] = 0.0;
        for (int h = g * group; h < (g + 1) * group; ++h) {
          for (int p = 0; p < N; ++p) {
            size_t qoff = (((size_t)b * N + p) * Hq + h) * D;
            double m = -INFINITY;
            for (int j = 0; j <= p; ++j) {
              size_t koff = (((size_t)b * N + j) * Hkv + g) * D;
              double dot = 0.0;
              for (int d = 0; d < D; ++d)
                dot += (double)load_el(q, dt, qoff + d) * (double)load_el(k, dt, koff + d);
              z[j] = dot * scale;
              if (z[j] > m) m = z[j];
            }
            double denom = 0.0;
            for (int j = 0; j <= p; ++j) denom += exp(z[j] - m);
            for (int j = 0; j <= p; ++j) col[j] += exp(z[j] - m) / denom;
          }
        }
      }
    }
    free(z);
  }
}

/* pool of the segment holding position i of request b (-1: fresh) */
static int pool_of(const rcref_seg* segs, int S, int b, int i) {
  for (int s = 0; s < S; ++s) {
    const rcref_seg* g = &segs[(size_t)b * S + s];
    if (i >= g->dst_start && i < g->dst_start + g->len) return g->pool;
  }
  return -1;
}

/* Importance score of Eq. (3) for every position i:
 *   S_i = (1 - lambda) ||A_i||_1 + lambda (||K_new,i - K_cached,i||_1 + ||V_new,i - V_cached,i||_1)
 * with ||A_i||_1 = sum_g mass[b, g, i] (mass as fp32, the form the GPU path
 * hands over) and the divergence norms over the token's Hkv*D entries of this
 * layer (new = fresh rows, cached = assembled rows after alignment). For a
 * token of an item block (its pool's bit set in item_pool_mask) the cached
 * block is a lexical match and the divergence term is dropped, leaving the
 * attention term alone (Sec. III-C.2b). At fresh positions the assembled rows
 * are the fresh rows, so the divergence is 0 there. fp64, stored as fp32. */
void rcref_score_eq3(int B, int N, int Hkv, int D, int dt, const int32_t* segs_raw, int S,
                     uint32_t item_pool_mask, double lambda, const float* mass,
                     const void* k_fresh, const void* v_fresh, const void* k_asm,
                     const void* v_asm, float* scores) {
  const rcref_seg* segs = (const rcref_seg*)segs_raw;
  size_t row = (size_t)Hkv * D;
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b) {
    for (int i = 0; i < N; ++i) {
      double attn = 0.0;
      for (int g = 0; g < Hkv; ++g) attn += (double)mass[((size_t)b * Hkv + g) * N + i];
      int pool = pool_of(segs, S, b, i);
      int item = pool >= 0 && ((item_pool_mask >> pool) & 1u);
      double div = 0.0;
      if (!item) {
        size_t base = ((size_t)b * N + i) * row;
        for (size_t e = 0; e < row; ++e)
          div += fabs((double)load_el(k_fresh, dt, base + e) - (double)load_el(k_asm, dt, base + e));
        for (size_t e = 0; e < row; ++e)
          div += fabs((double)load_el(v_fresh, dt, base + e) - (double)load_el(v_asm, dt, base + e));
      }
      scores[(size_t)b * N + i] = (float)((1.0 - lambda) * attn + lambda * div);
    }
  }
}

/* Heavy hitters with separate budgets for the two cached components (the
 * recompute ratios r_rev for history and r_item for items, Sec. IV-A): the
 * k_hist largest scores among cached positions of history pools and the
 * k_item largest among cached positions of item pools (bit set in
 * item_pool_mask), ties to the lower position in each. Rows are the fresh
 * positions and both selections in ascending order: rows[b, 0 .. F + k_hist +
 * k_item). Returns 0, or -1 if a budget exceeds its component's cached
 * positions in some request or the requests do not share one fresh count. */
int rcref_topk_split(int B, int N, const int32_t* segs_raw, int S, uint32_t item_pool_mask,
                     int k_hist, int k_item, const float* scores, int32_t* rows) {
  const rcref_seg* segs = (const rcref_seg*)segs_raw;
  int F = fresh_count(segs, S, 0);
  int R = F + k_hist + k_item;
  int status = 0;
  for (int b = 1; b < B; ++b)
    if (fresh_count(segs, S, b) != F) return -1;
  cand_t* cand = (cand_t*)malloc(sizeof(cand_t) * (size_t)(N > 0 ? N : 1));
  unsigned char* take = (unsigned char*)malloc((size_t)(N > 0 ? N : 1));
  for (int b = 0; b < B && status == 0; ++b) {
    memset(take, 0, (size_t)N);
    for (int i = 0; i < N; ++i)
      if (pool_of(segs, S, b, i) < 0) take[i] = 1;
    for (int comp = 0; comp < 2; ++comp) {
      int budget = comp == 0 ? k_hist : k_item;
      int n = 0;
      for (int i = 0; i < N; ++i) {
        int pool = pool_of(segs, S, b, i);
        if (pool < 0) continue;
        int item = (item_pool_mask >> pool) & 1u;
        if (item != comp) continue;
        cand[n].key = score_key(scores[(size_t)b * N + i]);
        cand[n].idx = i;
        ++n;
      }
      if (budget > n) {
        status = -1;
        break;
      }
      qsort(cand, (size_t)n, sizeof(cand_t), cand_cmp);
      for (int c = 0; c < budget; ++c) take[cand[c].idx] = 1;
    }
    if (status != 0) break;
    int r = 0;
    for (int i = 0; i < N; ++i)
      if (take[i]) rows[(size_t)b * R + r++] = i;
  }
  free(cand);
  free(take);
  return status;
}

/* ------------------------------------------------------------------ */
/* The whole pipeline                                                   */
/* ------------------------------------------------------------------ */

/* End-to-end selective prefill of one layer (Sec. III-C.3): (i) assemble,
 * (ii) align, score (Eq. (3) deviation term), select k heavy hitters, (iii)
 * patch them with fresh KV, then attention for the fresh and selected rows
 * over the assembled context. Every intermediate is returned. Returns 0, or -1
 * if k exceeds the cached positions of a request. */
int rcref_selective_prefill(int B, int N, int Hq, int Hkv, int D, int dt,
                            const void* const* pool_k, const void* const* pool_v,
                            const int32_t* pool_num_blocks, const int32_t* pool_block_len,
                            int n_pools, const int32_t* segs, int S, int k,
                            const void* q, const void* k_fresh, const void* v_fresh,
                            const float* cos_tab, const float* sin_tab, double scale,
                            void* k_asm, void* v_asm, float* scores, int32_t* rows,
                            void* out) {
  int F = fresh_count((const rcref_seg*)segs, S, 0);
  int R = F + k;
  rcref_assemble(B, N, Hkv, D, dt, pool_k, pool_v, pool_num_blocks, pool_block_len, n_pools,
                 segs, S, k_fresh, v_fresh, cos_tab, sin_tab, k_asm, v_asm);
  rcref_deviation(B, N, Hkv, D, dt, k_fresh, k_asm, scores);
  if (rcref_topk(B, N, segs, S, k, scores, rows) != 0) return -1;
  rcref_patch(B, N, Hkv, D, dt, segs, S, rows, R, k_fresh, v_fresh, k_asm, v_asm);
  rcref_attention(B, N, Hq, Hkv, D, dt, q, rows, R, k_asm, v_asm, scale, out);
  return 0;
}

/* Selection with the full score of Eq. (3) (Sec. III-C.2b): the first layer
 * is computed in full on the fresh K/V, which gives the attention mass of every
 * token; the cached blocks are assembled and aligned (steps i, ii); every
 * position is scored by Eq. (3); the history and item components each select
 * their own budget; the selected cached positions get fresh K/V (step iii).
 * mass [B, Hkv, N] and scores [B, N] are returned as fp32, rows [B, F +
 * k_hist + k_item]. Returns 0, or -1 if a budget exceeds its component. */
int rcref_eq3_select(int B, int N, int Hq, int Hkv, int D, int dt,
                     const void* const* pool_k, const void* const* pool_v,
                     const int32_t* pool_num_blocks, const int32_t* pool_block_len, int n_pools,
                     const int32_t* segs, int S, uint32_t item_pool_mask, double lambda,
                     int k_hist, int k_item, const void* q, const void* k_fresh,
                     const void* v_fresh, const float* cos_tab, const float* sin_tab,
                     double scale, void* k_asm, void* v_asm, float* mass, float* scores,
                     int32_t* rows) {
  int F = fresh_count((const rcref_seg*)segs, S, 0);
  int R = F + k_hist + k_item;
  size_t nm = (size_t)B * Hkv * N;
  double* m64 = (double*)malloc(sizeof(double) * (nm > 0 ? nm : 1));
  rcref_attention_mass(B, N, Hq, Hkv, D, dt, q, k_fresh, scale, m64);
  for (size_t e = 0; e < nm; ++e) mass[e] = (float)m64[e];
  free(m64);
  rcref_assemble(B, N, Hkv, D, dt, pool_k, pool_v, pool_num_blocks, pool_block_len, n_pools,
                 segs, S, k_fresh, v_fresh, cos_tab, sin_tab, k_asm, v_asm);
  rcref_score_eq3(B, N, Hkv, D, dt, segs, S, item_pool_mask, lambda, mass, k_fresh, v_fresh,
                  k_asm, v_asm, scores);
  if (rcref_topk_split(B, N, segs, S, item_pool_mask, k_hist, k_item, scores, rows) != 0)
    return -1;
  rcref_patch(B, N, Hkv, D, dt, segs, S, rows, R, k_fresh, v_fresh, k_asm, v_asm);
  return 0;
}
