/*
 * Reference oracle for uncertainty-gated block-sparse causal prefill.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow CPU statement of
 * what the GPU path computes.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark load it.  It shares no source with the
 * HIP library and must never be called by it.
 *
 * Arithmetic: every dot product, every softmax and every mean is taken in
 * IEEE double, in the obvious sequential order.  The only fp32 steps are the
 * ones the method's outputs are defined in: the tile score stored as fp32,
 * the cutoff margin sigma (fp32 subtract / divide), and the head mean of
 * sigma (fp32 sum in head order).  bf16 tensors are passed as raw uint16 bit
 * patterns and widened exactly.
 *
 * Paper sections followed (Appendix A, "step-by-step derivation"):
 *   A.1            block-pooled keys (K-mean), plus the Quest K-min/K-max pair
 *                  of Eq. (quest-score)
 *   A.2, A.3       per-row block scores and the per-tile max-pool,
 *                  Eq. (tile-score)
 *   A.4, A.5, A.6  forcing sink and self block, sorted top-(rho k) prefix and
 *                  the normalised cutoff margin, Eq. (sigma-def)
 *   A.7, A.8       head mean and per-layer empirical quantile, Eq. (trigger)
 *   A.9            padded expansion with sentinel N_B
 *   A.10           exact softmax attention over the kept blocks, Eq. (Attn)
 *   App. D         per-row score roughness for the noise-scale estimate
 *                  (empirical recipe, step 3)
 *
 * Readings where the paper is silent (each one also stated in the design
 * notes of the repository):
 *   - no 1/sqrt(d) in either block score (a positive scale changes neither
 *     the order nor sigma);
 *   - candidates are the causally visible, non-forced blocks 1..t-1;
 *   - sigma is taken over the non-forced list with m = k - |F| kept, and a
 *     tile with at most m candidates is "saturated" (sigma = -1, outside the
 *     quantile population, never triggered);
 *   - ties rank the lower block index first; -0 and +0 are equal;
 *   - the quantile threshold is the ceil(q n)-th smallest head-mean sigma
 *     over the population and every tile at or below it triggers;
 *   - GQA: query head h reads kv head h / (H / H_kv).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_BLOCK 64 /* BLOCK_M = BLOCK_N = 64 tokens */

enum { ORC_KMEAN = 0, ORC_QUEST = 1 };

/* ------------------------------------------------------------------ */
/* bf16 helpers                                                        */
/* ------------------------------------------------------------------ */

static double bf16_val(uint16_t bits) {
  uint32_t w = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &w, sizeof f);
  return (double)f;
}

/* Round a double to the nearest bf16, ties to even, by scaling it onto the
 * bf16 grid of its binade and calling nearbyint() (round-half-even in the
 * default rounding mode).  Zero is returned as +0. */
static uint16_t bf16_round(double x) {
  if (x == 0.0) return 0;
  double ax = fabs(x);
  int e;
  frexp(ax, &e);                 /* ax in [2^(e-1), 2^e) */
  int qexp = e - 8;              /* 8 significant bits */
  if (qexp < -133) qexp = -133;  /* bf16 subnormal spacing */
  double quantum = ldexp(1.0, qexp);
  double r = nearbyint(ax / quantum) * quantum;
  float f = (float)r;            /* exact: r has <= 8 significant bits */
  if (x < 0) f = -f;
  uint32_t w;
  memcpy(&w, &f, sizeof w);
  return (uint16_t)(w >> 16);
}

static float canon_zero(float x) { return x == 0.0f ? 0.0f : x; }

/* ------------------------------------------------------------------ */
/* a tiny thread pool: run fn(i, ctx) for i in [0, n)                   */
/* ------------------------------------------------------------------ */

typedef void (*orc_item_fn)(long i, void* ctx);
typedef struct {
  orc_item_fn fn;
  void* ctx;
  long n;
  long next;
  pthread_mutex_t mu;
} orc_pool;

static void* orc_worker(void* arg) {
  orc_pool* p = (orc_pool*)arg;
  for (;;) {
    pthread_mutex_lock(&p->mu);
    long i = p->next++;
    pthread_mutex_unlock(&p->mu);
    if (i >= p->n) break;
    p->fn(i, p->ctx);
  }
  return NULL;
}

static void orc_parallel(long n, int nthreads, orc_item_fn fn, void* ctx) {
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if (nthreads == 1 || n <= 1) {
    for (long i = 0; i < n; ++i) fn(i, ctx);
    return;
  }
  orc_pool p;
  p.fn = fn;
  p.ctx = ctx;
  p.n = n;
  p.next = 0;
  pthread_mutex_init(&p.mu, NULL);
  pthread_t th[256];
  int started = 0;
  for (int k = 0; k < nthreads; ++k)
    if (pthread_create(&th[k], NULL, orc_worker, &p) == 0) started++;
  if (started == 0) orc_worker(&p);
  for (int k = 0; k < started; ++k) pthread_join(th[k], NULL);
  pthread_mutex_destroy(&p.mu);
}

/* ------------------------------------------------------------------ */
/* A.1: block metadata                                                 */
/* ------------------------------------------------------------------ */
/* K    [B, Hkv, N, d] bf16
 * meta K-mean: [B, Hkv, N_B, d]     bf16, mean of the block's 64 keys
 *      Quest : [B, Hkv, N_B, 2, d]  bf16, (element-wise min, element-wise max)
 */
typedef struct {
  int backbone, d, N;
  const uint16_t* K;
  uint16_t* meta;
} meta_ctx;

static void meta_item(long bh_blk, void* vctx) {
  meta_ctx* c = (meta_ctx*)vctx;
  int NB = c->N / ORC_BLOCK, d = c->d;
  long bh = bh_blk / NB;
  int blk = (int)(bh_blk % NB);
  const uint16_t* kb = c->K + ((size_t)bh * c->N + (size_t)blk * ORC_BLOCK) * d;
  if (c->backbone == ORC_KMEAN) {
    uint16_t* out = c->meta + ((size_t)bh * NB + blk) * d;
    for (int e = 0; e < d; ++e) {
      double s = 0.0;
      for (int j = 0; j < ORC_BLOCK; ++j) s += bf16_val(kb[(size_t)j * d + e]);
      out[e] = bf16_round(s / ORC_BLOCK);
    }
  } else {
    uint16_t* omin = c->meta + ((size_t)bh * NB + blk) * 2 * d;
    uint16_t* omax = omin + d;
    for (int e = 0; e < d; ++e) {
      double lo = bf16_val(kb[e]), hi = lo;
      for (int j = 1; j < ORC_BLOCK; ++j) {
        double v = bf16_val(kb[(size_t)j * d + e]);
        if (v < lo) lo = v;
        if (v > hi) hi = v;
      }
      omin[e] = bf16_round(lo); /* exact: lo is a bf16 value */
      omax[e] = bf16_round(hi);
    }
  }
}

int orc_block_meta(int backbone, int B, int Hkv, int N, int d,
                   const uint16_t* K, uint16_t* meta, int nthreads) {
  if (N % ORC_BLOCK || (backbone != ORC_KMEAN && backbone != ORC_QUEST)) return -1;
  meta_ctx c = {backbone, d, N, K, meta};
  orc_parallel((long)B * Hkv * (N / ORC_BLOCK), nthreads, meta_item, &c);
  return 0;
}

/* ------------------------------------------------------------------ */
/* A.2 + A.3: tile scores                                              */
/* ------------------------------------------------------------------ */
/* For each requested unit (b, h, t): out[u, b'] = fp32(max over the 64 rows
 * r of tile t of s[r, b']) for candidate blocks b' in C(t) = {1..t-1}, and
 * -inf elsewhere.  K-mean: s = q . kbar.  Quest: s = sum_d max(q_d kmax_d,
 * q_d kmin_d), the literal Eq. (quest-score).  No 1/sqrt(d). */
typedef struct {
  int backbone, H, Hkv, N, d;
  const uint16_t* Q;
  const uint16_t* meta;
  const int32_t* units; /* 3 ints per unit */
  float* out;
} score_ctx;

static void score_item(long u, void* vctx) {
  score_ctx* c = (score_ctx*)vctx;
  int NB = c->N / ORC_BLOCK, d = c->d, G = c->H / c->Hkv;
  int b = c->units[3 * u], h = c->units[3 * u + 1], t = c->units[3 * u + 2];
  int kvh = h / G;
  float* out = c->out + (size_t)u * NB;
  for (int blk = 0; blk < NB; ++blk) out[blk] = -INFINITY;
  double* q = (double*)malloc(sizeof(double) * (size_t)ORC_BLOCK * d);
  const uint16_t* qb = c->Q + (((size_t)b * c->H + h) * c->N + (size_t)t * ORC_BLOCK) * d;
  for (long x = 0; x < (long)ORC_BLOCK * d; ++x) q[x] = bf16_val(qb[x]);
  int width = (c->backbone == ORC_KMEAN) ? 1 : 2;
  for (int blk = 1; blk <= t - 1; ++blk) {
    const uint16_t* m = c->meta + (((size_t)b * c->Hkv + kvh) * NB + blk) * width * d;
    double best = -INFINITY;
    for (int r = 0; r < ORC_BLOCK; ++r) {
      const double* qr = q + (size_t)r * d;
      double s = 0.0;
      if (c->backbone == ORC_KMEAN) {
        for (int e = 0; e < d; ++e) s += qr[e] * bf16_val(m[e]);
      } else {
        for (int e = 0; e < d; ++e) {
          double a = qr[e] * bf16_val(m[d + e]); /* q_d * kmax_d */
          double z = qr[e] * bf16_val(m[e]);     /* q_d * kmin_d */
          s += (a > z) ? a : z;
        }
      }
      if (s > best) best = s;
    }
    out[blk] = (float)best;
  }
  free(q);
}

int orc_tile_scores(int backbone, int B, int H, int Hkv, int N, int d,
                    const uint16_t* Q, const uint16_t* meta, long n_units,
                    const int32_t* units, float* out, int nthreads) {
  if (N % ORC_BLOCK || H % Hkv) return -1;
  (void)B;
  score_ctx c = {backbone, H, Hkv, N, d, Q, meta, units, out};
  orc_parallel(n_units, nthreads, score_item, &c);
  return 0;
}

/* ------------------------------------------------------------------ */
/* A.4 - A.6: forcing, sorted top-(2k) prefix, sigma                    */
/* ------------------------------------------------------------------ */
typedef struct {
  float s;
  int32_t blk;
} cand_t;

static int cand_cmp(const void* pa, const void* pb) {
  const cand_t* a = (const cand_t*)pa;
  const cand_t* b = (const cand_t*)pb;
  if (a->s > b->s) return -1;
  if (a->s < b->s) return 1;
  return (a->blk < b->blk) ? -1 : (a->blk > b->blk);
}

/* One row: tile t, scores row[0..N_B) (only C(t) = 1..t-1 is read).
 * idx_out gets W = rho k entries: F(t) = [0] (t = 0) or [0, t], then the
 * candidates by (score desc, block asc), truncated to W and padded with N_B
 * (Section 3 step 5: the sorted prefix is cut at rho k).
 * sigma_out: (c[m-1] - c[m]) / (c[0] - c[m]) over the sorted candidates with
 * m = k - |F|, fp32; 0 if the denominator is 0; -1 if |C| <= m. */
static void select_row(int t, int NB, int k, int W, const float* row, int32_t* idx_out,
                       float* sigma_out) {
  int nf = (t == 0) ? 1 : 2;
  int nc = (t >= 1) ? t - 1 : 0;
  int m = k - nf;
  cand_t* c = (cand_t*)malloc(sizeof(cand_t) * (size_t)(nc > 0 ? nc : 1));
  for (int i = 0; i < nc; ++i) {
    c[i].s = canon_zero(row[1 + i]);
    c[i].blk = 1 + i;
  }
  qsort(c, (size_t)nc, sizeof(cand_t), cand_cmp);
  int pos = 0;
  idx_out[pos++] = 0;
  if (t >= 1) idx_out[pos++] = t;
  for (int i = 0; i < nc && pos < W; ++i) idx_out[pos++] = c[i].blk;
  while (pos < W) idx_out[pos++] = NB;
  if (nc <= m) {
    *sigma_out = -1.0f;
  } else {
    float num = c[m - 1].s - c[m].s;
    float den = c[0].s - c[m].s;
    *sigma_out = (den == 0.0f) ? 0.0f : num / den;
  }
  free(c);
}

int orc_select(int NB, int k, int rho, long n_rows, const int32_t* t_of_row,
               const float* tile_score, int32_t* idx_sorted, float* sigma) {
  if (k < 3 || rho < 1) return -1;
  int W = rho * k;
  for (long r = 0; r < n_rows; ++r)
    select_row(t_of_row[r], NB, k, W, tile_score + (size_t)r * NB,
               idx_sorted + (size_t)r * W, sigma + r);
  return 0;
}

/* ------------------------------------------------------------------ */
/* A.7 - A.9: head mean, per-layer quantile, padded expansion           */
/* ------------------------------------------------------------------ */
static int cmp_float_asc(const void* pa, const void* pb) {
  float a = *(const float*)pa, b = *(const float*)pb;
  return (a < b) ? -1 : (a > b);
}

/* Population of tile t: more non-forced candidates than kept slots. */
static int in_population(int t, int k) {
  int nf = (t == 0) ? 1 : 2;
  int nc = (t >= 1) ? t - 1 : 0;
  return nc > k - nf;
}

/* sigma [B, H, T], idx_sorted [B, H, T, W] -> kv_idx [B, H, T, W] with
 * W = rho k (a triggered tile keeps all W slots, the others the first k),
 * sigma_bar [B, T] (-1 outside the population), tau [B] (-1 when nothing
 * triggers), trigger [B, T]. */
int orc_route(int B, int H, int T, int k, int rho, double q, const float* sigma,
              const int32_t* idx_sorted, int32_t* kv_idx, float* sigma_bar,
              float* tau, uint8_t* trigger) {
  if (q < 0.0 || q > 1.0 || k < 3 || rho < 1) return -1;
  int W = rho * k, NB = T;
  float* pop = (float*)malloc(sizeof(float) * (size_t)(T > 0 ? T : 1));
  for (int b = 0; b < B; ++b) {
    int n = 0;
    for (int t = 0; t < T; ++t) {
      float sb = -1.0f;
      if (in_population(t, k)) {
        float s = 0.0f;
        for (int h = 0; h < H; ++h) s += sigma[((size_t)b * H + h) * T + t];
        sb = s / (float)H;
        pop[n++] = sb;
      }
      sigma_bar[(size_t)b * T + t] = sb;
    }
    long n_trig = (long)ceil(q * (double)n);
    float thr = -1.0f;
    if (n_trig > 0) {
      qsort(pop, (size_t)n, sizeof(float), cmp_float_asc);
      thr = pop[n_trig - 1];
    }
    tau[b] = thr;
    for (int t = 0; t < T; ++t) {
      int trig = (n_trig > 0) && in_population(t, k) &&
                 sigma_bar[(size_t)b * T + t] <= thr;
      trigger[(size_t)b * T + t] = (uint8_t)trig;
      for (int h = 0; h < H; ++h) {
        size_t row = (((size_t)b * H + h) * T + t) * W;
        for (int s = 0; s < W; ++s)
          kv_idx[row + s] = (trig || s < k) ? idx_sorted[row + s] : NB;
      }
    }
  }
  free(pop);
  return 0;
}

/* ------------------------------------------------------------------ */
/* A.10 / Eq. (Attn): exact softmax attention over the kept blocks       */
/* ------------------------------------------------------------------ */
/* For unit (b, h, t) and its kv_idx row (W entries; entries outside
 * [0, N_B) are sentinels and are ignored), each row i of tile t attends to
 * J_i = { j <= i : block(j) is listed }.  dense != 0 ignores kv_idx and
 * uses J_i = { j <= i }.  O is [n_units, 64, d] in double; a row with an
 * empty J_i is 0. */
typedef struct {
  int H, Hkv, N, d, W, dense;
  double scale;
  const uint16_t *Q, *K, *V;
  const int32_t* kv_idx;
  const int32_t* units;
  double* O;
} attn_ctx;

static void attn_item(long u, void* vctx) {
  attn_ctx* c = (attn_ctx*)vctx;
  int NB = c->N / ORC_BLOCK, d = c->d, G = c->H / c->Hkv;
  int b = c->units[3 * u], h = c->units[3 * u + 1], t = c->units[3 * u + 2];
  int kvh = h / G;
  char* keep = (char*)calloc((size_t)NB, 1);
  if (c->dense) {
    for (int blk = 0; blk < NB; ++blk) keep[blk] = 1;
  } else {
    const int32_t* row = c->kv_idx + (size_t)u * c->W;
    for (int s = 0; s < c->W; ++s)
      if (row[s] >= 0 && row[s] < NB) keep[row[s]] = 1;
  }
  const uint16_t* Kh = c->K + ((size_t)b * c->Hkv + kvh) * c->N * d;
  const uint16_t* Vh = c->V + ((size_t)b * c->Hkv + kvh) * c->N * d;
  const uint16_t* Qh = c->Q + ((size_t)b * c->H + h) * c->N * d;
  int n_max = (t + 1) * ORC_BLOCK;
  double* logit = (double*)malloc(sizeof(double) * (size_t)n_max);
  double* acc = (double*)malloc(sizeof(double) * (size_t)d);
  double* qv = (double*)malloc(sizeof(double) * (size_t)d);
  for (int r = 0; r < ORC_BLOCK; ++r) {
    int i = t * ORC_BLOCK + r;
    double* o = c->O + ((size_t)u * ORC_BLOCK + r) * d;
    for (int e = 0; e < d; ++e) qv[e] = bf16_val(Qh[(size_t)i * d + e]);
    double mx = -INFINITY;
    int any = 0;
    for (int j = 0; j <= i; ++j) {
      if (!keep[j / ORC_BLOCK]) continue;
      double s = 0.0;
      for (int e = 0; e < d; ++e) s += qv[e] * bf16_val(Kh[(size_t)j * d + e]);
      s *= c->scale;
      logit[j] = s;
      if (s > mx) mx = s;
      any = 1;
    }
    for (int e = 0; e < d; ++e) acc[e] = 0.0;
    if (!any) {
      for (int e = 0; e < d; ++e) o[e] = 0.0;
      continue;
    }
    double den = 0.0;
    for (int j = 0; j <= i; ++j) {
      if (!keep[j / ORC_BLOCK]) continue;
      double p = exp(logit[j] - mx);
      den += p;
      for (int e = 0; e < d; ++e) acc[e] += p * bf16_val(Vh[(size_t)j * d + e]);
    }
    for (int e = 0; e < d; ++e) o[e] = acc[e] / den;
  }
  free(qv);
  free(acc);
  free(logit);
  free(keep);
}

int orc_attend(int H, int Hkv, int N, int d, double scale, const uint16_t* Q,
               const uint16_t* K, const uint16_t* V, const int32_t* kv_idx,
               int W, int dense, long n_units, const int32_t* units, double* O,
               int nthreads) {
  if (N % ORC_BLOCK || H % Hkv) return -1;
  attn_ctx c = {H, Hkv, N, d, W, dense, scale, Q, K, V, kv_idx, units, O};
  orc_parallel(n_units, nthreads, attn_item, &c);
  return 0;
}

/* Exposed for the oracle's own pins: bf16 rounding of a double. */
/* ------------------------------------------------------------------ */
/* Appendix D, empirical recipe step 3: row-to-row score roughness     */
/* ------------------------------------------------------------------ */
/* For each requested unit (b, h, t): the sum over candidate blocks b' in
 * C(t) = {1..t-1} and over the 63 adjacent row pairs (r, r+1) of tile t of
 * (s[r+1, b'] - s[r, b'])^2, with the per-row block score s of A.2 (the same
 * formula as the tile score, before the max over rows), all in double.  The
 * number of terms is 63 |C(t)|. */
typedef struct {
  int backbone, H, Hkv, N, d;
  const uint16_t* Q;
  const uint16_t* meta;
  const int32_t* units;
  double* out;
} rough_ctx;

static void rough_item(long u, void* vctx) {
  rough_ctx* c = (rough_ctx*)vctx;
  int NB = c->N / ORC_BLOCK, d = c->d, G = c->H / c->Hkv;
  int b = c->units[3 * u], h = c->units[3 * u + 1], t = c->units[3 * u + 2];
  int kvh = h / G;
  double* q = (double*)malloc(sizeof(double) * (size_t)ORC_BLOCK * d);
  const uint16_t* qb = c->Q + (((size_t)b * c->H + h) * c->N + (size_t)t * ORC_BLOCK) * d;
  for (long x = 0; x < (long)ORC_BLOCK * d; ++x) q[x] = bf16_val(qb[x]);
  int width = (c->backbone == ORC_KMEAN) ? 1 : 2;
  double total = 0.0;
  for (int blk = 1; blk <= t - 1; ++blk) {
    const uint16_t* m = c->meta + (((size_t)b * c->Hkv + kvh) * NB + blk) * width * d;
    double prev = 0.0;
    for (int r = 0; r < ORC_BLOCK; ++r) {
      const double* qr = q + (size_t)r * d;
      double s = 0.0;
      if (c->backbone == ORC_KMEAN) {
        for (int e = 0; e < d; ++e) s += qr[e] * bf16_val(m[e]);
      } else {
        for (int e = 0; e < d; ++e) {
          double a = qr[e] * bf16_val(m[d + e]);
          double z = qr[e] * bf16_val(m[e]);
          s += (a > z) ? a : z;
        }
      }
      if (r > 0) total += (s - prev) * (s - prev);
      prev = s;
    }
  }
  c->out[u] = total;
  free(q);
}

int orc_row_roughness(int backbone, int H, int Hkv, int N, int d, const uint16_t* Q,
                      const uint16_t* meta, long n_units, const int32_t* units, double* out,
                      int nthreads) {
  if (N % ORC_BLOCK || H % Hkv) return -1;
  rough_ctx c = {backbone, H, Hkv, N, d, Q, meta, units, out};
  orc_parallel(n_units, nthreads, rough_item, &c);
  return 0;
}

/* ------------------------------------------------------------------ */
/* Per-row block scores (A.2 before the max over the tile's rows), for   */
/* the per-row selection variant (Section 3.2 and the Limitations of    */
/* Section 4)                                                           */
/* ------------------------------------------------------------------ */
/* For each requested unit (b, h, t): out[unit][r][blk] = the fp64 score of
 * query row r of tile t against block blk, rounded to fp32, for blk in
 * C(t) = {1..t-1}; -inf elsewhere. */
typedef struct {
  int backbone, H, Hkv, N, d;
  const uint16_t* Q;
  const uint16_t* meta;
  const int32_t* units;
  float* out;
} rows_ctx;

static void rows_item(long u, void* vctx) {
  rows_ctx* c = (rows_ctx*)vctx;
  int NB = c->N / ORC_BLOCK, d = c->d, G = c->H / c->Hkv;
  int b = c->units[3 * u], h = c->units[3 * u + 1], t = c->units[3 * u + 2];
  int kvh = h / G;
  float* out = c->out + (size_t)u * ORC_BLOCK * NB;
  for (long x = 0; x < (long)ORC_BLOCK * NB; ++x) out[x] = -INFINITY;
  const uint16_t* qb = c->Q + (((size_t)b * c->H + h) * c->N + (size_t)t * ORC_BLOCK) * d;
  int width = (c->backbone == ORC_KMEAN) ? 1 : 2;
  for (int blk = 1; blk <= t - 1; ++blk) {
    const uint16_t* m = c->meta + (((size_t)b * c->Hkv + kvh) * NB + blk) * width * d;
    for (int r = 0; r < ORC_BLOCK; ++r) {
      const uint16_t* qr = qb + (size_t)r * d;
      double s = 0.0;
      if (c->backbone == ORC_KMEAN) {
        for (int e = 0; e < d; ++e) s += bf16_val(qr[e]) * bf16_val(m[e]);
      } else {
        for (int e = 0; e < d; ++e) {
          double a = bf16_val(qr[e]) * bf16_val(m[d + e]);
          double z = bf16_val(qr[e]) * bf16_val(m[e]);
          s += (a > z) ? a : z;
        }
      }
      out[(size_t)r * NB + blk] = (float)s;
    }
  }
}

int orc_row_scores(int backbone, int H, int Hkv, int N, int d, const uint16_t* Q,
                   const uint16_t* meta, long n_units, const int32_t* units, float* out,
                   int nthreads) {
  if (N % ORC_BLOCK || H % Hkv) return -1;
  rows_ctx c = {backbone, H, Hkv, N, d, Q, meta, units, out};
  orc_parallel(n_units, nthreads, rows_item, &c);
  return 0;
}

uint16_t orc_bf16_round(double x) { return bf16_round(x); }
