/*
 * Seeded synthetic rating matrices shaped like the matrix-factorization workload of
 * Dai et al., "High-Performance Distributed ML at Scale through Parameter Server
 * Consistency Models" (arXiv 1410.8043), Section 5 (a Netflix-shaped ratings matrix:
 * users x items, integer ratings 1..5, heavy-tailed degrees).
 *
 * This module produces INPUTS only.  It holds none of the method's arithmetic (no
 * residual, gradient, update or loss); both the HIP library and the CPU oracle consume
 * what it writes.  Everything is a pure function of (arguments, seed): results do not
 * depend on the thread count.
 *
 * Random numbers: SplitMix64 (Steele, Lea & Flood, OOPSLA 2014), used two ways:
 *   - as a sequential generator: state += 0x9E3779B97F4A7C15; output = mix(state);
 *   - counter-based: the value at (seed, stream, counter) is the first output of a
 *     generator whose state is  seed ^ stream*0xD1B54A32D192ED03 ^ counter*0x9E3779B97F4A7C15.
 * Normal deviates use the Box-Muller transform on two such counters.
 *
 * Build: gcc -O2 -fPIC -shared -pthread synth.c -lm -o libps_mf_synth.so
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define SYNTH_OK 0
#define SYNTH_EINVAL -1
#define SYNTH_ENOMEM -2

#define GOLDEN 0x9E3779B97F4A7C15ULL
#define STREAM_MUL 0xD1B54A32D192ED03ULL

static inline uint64_t sm_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* sequential SplitMix64 */
static inline uint64_t sm_next(uint64_t *state) {
  *state += GOLDEN;
  return sm_mix(*state);
}

/* counter-based draw */
static inline uint64_t ctr_u64(uint64_t seed, uint64_t stream, uint64_t ctr) {
  uint64_t st = seed ^ (stream * STREAM_MUL) ^ (ctr * GOLDEN);
  return sm_next(&st);
}

/* uniform in (0, 1]: 53 random bits */
static inline double u01_open0(uint64_t x) { return ((double)(x >> 11) + 1.0) * (1.0 / 9007199254740992.0); }
/* uniform in [0, 1) */
static inline double u01(uint64_t x) { return (double)(x >> 11) * (1.0 / 9007199254740992.0); }

static inline double ctr_normal(uint64_t seed, uint64_t stream, uint64_t idx) {
  double a = u01_open0(ctr_u64(seed, stream, 2 * idx));
  double b = u01(ctr_u64(seed, stream, 2 * idx + 1));
  return sqrt(-2.0 * log(a)) * cos(6.283185307179586 * b);
}

/* bounded integer in [0, n) by 128-bit multiply (Lemire), slight bias irrelevant here */
static inline uint64_t bounded(uint64_t x, uint64_t n) {
  return (uint64_t)(((unsigned __int128)x * (unsigned __int128)n) >> 64);
}

/* streams: distinct constants so that no two uses share draws */
enum {
  ST_PERM_ROWS = 1, ST_PERM_ITEMS = 2, ST_PAIRS = 3, ST_PLANT_U = 4, ST_PLANT_V = 5,
  ST_NOISE = 6, ST_CELLS = 7, ST_USER_NORMAL = 8
};

int synth_splitmix64_next(uint64_t *state, uint64_t *out) {
  *out = sm_next(state);
  return SYNTH_OK;
}

/* ---------------- threading helper ---------------- */
typedef void (*range_fn)(void *ctx, int64_t lo, int64_t hi);
typedef struct { range_fn fn; void *ctx; int64_t lo, hi; } range_job;
static void *range_tramp(void *p) {
  range_job *j = (range_job *)p;
  j->fn(j->ctx, j->lo, j->hi);
  return NULL;
}
static void parallel_range(int nthreads, int64_t n, range_fn fn, void *ctx) {
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 64) nthreads = 64;
  if (n < 4096 || nthreads == 1) { fn(ctx, 0, n); return; }
  pthread_t th[64];
  range_job jobs[64];
  /* many small chunks per thread would balance better; rows are pre-shuffled so a
     static split is adequate */
  for (int t = 0; t < nthreads; ++t) {
    jobs[t].fn = fn; jobs[t].ctx = ctx;
    jobs[t].lo = n * t / nthreads; jobs[t].hi = n * (t + 1) / nthreads;
    pthread_create(&th[t], NULL, range_tramp, &jobs[t]);
  }
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
}

/* seeded Fisher-Yates permutation of 0..n-1 */
static void seeded_perm(int64_t n, uint64_t seed, uint64_t stream, int64_t *perm) {
  for (int64_t i = 0; i < n; ++i) perm[i] = i;
  uint64_t st = seed ^ (stream * STREAM_MUL);
  for (int64_t i = n - 1; i > 0; --i) {
    int64_t k = (int64_t)bounded(sm_next(&st), (uint64_t)(i + 1));
    int64_t t = perm[i]; perm[i] = perm[k]; perm[k] = t;
  }
}

/*
 * Zipf(a) weights by rank (rank r has weight r^-a; a = 0 gives equal weights), with
 * ranks mapped to ids by a seeded permutation.  weight_out[id].
 */
int synth_rank_weights(int64_t n, double a, uint64_t seed, int32_t which, double *weight_out) {
  if (n <= 0 || a < 0 || !weight_out) return SYNTH_EINVAL;
  int64_t *perm = (int64_t *)malloc(sizeof(int64_t) * (size_t)n);
  if (!perm) return SYNTH_ENOMEM;
  seeded_perm(n, seed, which == 0 ? ST_PERM_ROWS : ST_PERM_ITEMS, perm);
  for (int64_t r = 0; r < n; ++r) weight_out[perm[r]] = (a == 0.0) ? 1.0 : pow((double)(r + 1), -a);
  free(perm);
  return SYNTH_OK;
}

/*
 * Integer degrees summing exactly to nnz, proportional to the given weights, capped at
 * `cap` with the excess water-filled onto uncapped rows:
 *   t_i = min(cap, c * w_i), c chosen by bisection so that sum t_i = nnz;
 *   d_i = floor(t_i), and the remainder goes one each to the uncapped rows with the
 *   largest fractional parts (ties: lower id first).
 */
typedef struct { double frac; int64_t id; } fracid;
static int cmp_frac_desc(const void *a, const void *b) {
  const fracid *x = (const fracid *)a, *y = (const fracid *)b;
  if (x->frac > y->frac) return -1;
  if (x->frac < y->frac) return 1;
  return (x->id < y->id) ? -1 : (x->id > y->id);
}
int synth_degrees(int64_t n, const double *w, int64_t nnz, int64_t cap, int64_t *deg_out) {
  if (n <= 0 || nnz < 0 || cap <= 0 || !w || !deg_out) return SYNTH_EINVAL;
  if ((double)nnz > (double)n * (double)cap) return SYNTH_EINVAL;
  double wsum = 0, wmax = 0;
  for (int64_t i = 0; i < n; ++i) { if (!(w[i] > 0)) return SYNTH_EINVAL; wsum += w[i]; if (w[i] > wmax) wmax = w[i]; }
  double lo = 0, hi = (double)nnz / w[0] + 1.0;
  for (int64_t i = 0; i < n; ++i) { double c = (double)cap / w[i]; if (c > hi) hi = c; }
  hi *= 2;
  for (int it = 0; it < 200; ++it) {
    double mid = 0.5 * (lo + hi), s = 0;
    for (int64_t i = 0; i < n; ++i) { double t = mid * w[i]; s += t < (double)cap ? t : (double)cap; }
    if (s < (double)nnz) lo = mid; else hi = mid;
  }
  double c = lo;
  int64_t tot = 0;
  fracid *fr = (fracid *)malloc(sizeof(fracid) * (size_t)n);
  if (!fr) return SYNTH_ENOMEM;
  int64_t nfr = 0;
  for (int64_t i = 0; i < n; ++i) {
    double t = c * w[i];
    if (t >= (double)cap) { deg_out[i] = cap; }
    else { deg_out[i] = (int64_t)floor(t); fr[nfr].frac = t - floor(t); fr[nfr].id = i; ++nfr; }
    tot += deg_out[i];
  }
  int64_t rem = nnz - tot;
  if (rem < 0 || rem > nfr) { free(fr); return SYNTH_EINVAL; }
  qsort(fr, (size_t)nfr, sizeof(fracid), cmp_frac_desc);
  for (int64_t k = 0; k < rem; ++k) deg_out[fr[k].id] += 1;
  free(fr);
  return SYNTH_OK;
}

/* ---------------- pair sampling ---------------- */
/* Vose alias table */
typedef struct { double *prob; int32_t *alias; int64_t n; } alias_t;
static int alias_build(alias_t *t, const double *w, int64_t n) {
  t->n = n;
  t->prob = (double *)malloc(sizeof(double) * (size_t)n);
  t->alias = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
  int64_t *small = (int64_t *)malloc(sizeof(int64_t) * (size_t)n);
  int64_t *large = (int64_t *)malloc(sizeof(int64_t) * (size_t)n);
  double *p = (double *)malloc(sizeof(double) * (size_t)n);
  if (!t->prob || !t->alias || !small || !large || !p) { free(small); free(large); free(p); return SYNTH_ENOMEM; }
  double s = 0;
  for (int64_t i = 0; i < n; ++i) s += w[i];
  int64_t ns = 0, nl = 0;
  for (int64_t i = 0; i < n; ++i) {
    p[i] = w[i] * (double)n / s;
    if (p[i] < 1.0) small[ns++] = i; else large[nl++] = i;
  }
  while (ns > 0 && nl > 0) {
    int64_t l = small[--ns], g = large[--nl];
    t->prob[l] = p[l]; t->alias[l] = (int32_t)g;
    p[g] = (p[g] + p[l]) - 1.0;
    if (p[g] < 1.0) small[ns++] = g; else large[nl++] = g;
  }
  while (nl > 0) { int64_t g = large[--nl]; t->prob[g] = 1.0; t->alias[g] = (int32_t)g; }
  while (ns > 0) { int64_t l = small[--ns]; t->prob[l] = 1.0; t->alias[l] = (int32_t)l; }
  free(small); free(large); free(p);
  return SYNTH_OK;
}
static inline int32_t alias_draw(const alias_t *t, uint64_t *st) {
  uint64_t x = sm_next(st);
  int64_t k = (int64_t)bounded(x, (uint64_t)t->n);
  double u = u01(sm_next(st));
  return u < t->prob[k] ? (int32_t)k : t->alias[k];
}

typedef struct { double key; int32_t id; } keyid;
static int cmp_key_desc(const void *a, const void *b) {
  const keyid *x = (const keyid *)a, *y = (const keyid *)b;
  if (x->key > y->key) return -1;
  if (x->key < y->key) return 1;
  return (x->id < y->id) ? -1 : (x->id > y->id);
}
/* quickselect: move the d largest keys to the front */
static void select_top(keyid *a, int64_t n, int64_t d) {
  int64_t lo = 0, hi = n - 1;
  while (lo < hi) {
    keyid piv = a[lo + (hi - lo) / 2];
    int64_t i = lo, j = hi;
    while (i <= j) {
      while (cmp_key_desc(&a[i], &piv) < 0) ++i;
      while (cmp_key_desc(&a[j], &piv) > 0) --j;
      if (i <= j) { keyid t = a[i]; a[i] = a[j]; a[j] = t; ++i; --j; }
    }
    if (d - 1 <= j) hi = j; else if (d - 1 >= i) lo = i; else break;
  }
}

typedef struct {
  int64_t N, M;
  const int64_t *deg, *off;
  const double *w;
  const alias_t *al;
  uint64_t seed;
  int32_t *user_out, *item_out;
  int err;
} pairs_ctx;

static void pairs_range(void *vctx, int64_t lo, int64_t hi) {
  pairs_ctx *cx = (pairs_ctx *)vctx;
  int64_t M = cx->M;
  int64_t *stamp = (int64_t *)malloc(sizeof(int64_t) * (size_t)M);
  keyid *keys = NULL;
  if (!stamp) { cx->err = SYNTH_ENOMEM; return; }
  for (int64_t j = 0; j < M; ++j) stamp[j] = -1;
  for (int64_t u = lo; u < hi; ++u) {
    int64_t d = cx->deg[u];
    if (d == 0) continue;
    int32_t *uo = cx->user_out + cx->off[u];
    int32_t *io = cx->item_out + cx->off[u];
    uint64_t st = cx->seed ^ ((uint64_t)ST_PAIRS * STREAM_MUL) ^ ((uint64_t)(u + 1) * GOLDEN);
    for (int64_t t = 0; t < d; ++t) uo[t] = (int32_t)u;
    if (d * 4 > M) {
      /* Efraimidis-Spirakis keys: taking the d largest of log(U_j)/w_j draws d distinct
         items with the same law as successive weighted sampling without replacement */
      if (!keys) { keys = (keyid *)malloc(sizeof(keyid) * (size_t)M); if (!keys) { cx->err = SYNTH_ENOMEM; break; } }
      for (int64_t j = 0; j < M; ++j) { keys[j].key = log(u01_open0(sm_next(&st))) / cx->w[j]; keys[j].id = (int32_t)j; }
      if (d < M) select_top(keys, M, d);
      qsort(keys, (size_t)d, sizeof(keyid), cmp_key_desc);
      for (int64_t t = 0; t < d; ++t) io[t] = keys[t].id;
    } else {
      /* successive weighted draws, rejecting items this user already has */
      int64_t got = 0;
      while (got < d) {
        int32_t j = alias_draw(cx->al, &st);
        if (stamp[j] == u) continue;
        stamp[j] = u;
        io[got++] = j;
      }
    }
  }
  free(keys);
  free(stamp);
}

/*
 * For each user u draw deg[u] distinct items, item j chosen with probability
 * proportional to item_w[j] among the items u does not have yet.  Output is user-major
 * (users in id order), items in draw order.  Requires deg[u] <= M.
 */
int synth_pairs(int64_t N, int64_t M, const int64_t *deg, const double *item_w, uint64_t seed, int32_t nthreads,
                int32_t *user_out, int32_t *item_out) {
  if (N <= 0 || M <= 0 || M > 0x7fffffff || N > 0x7fffffff || !deg || !item_w || !user_out || !item_out) return SYNTH_EINVAL;
  int64_t *off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(N + 1));
  if (!off) return SYNTH_ENOMEM;
  off[0] = 0;
  for (int64_t u = 0; u < N; ++u) {
    if (deg[u] < 0 || deg[u] > M) { free(off); return SYNTH_EINVAL; }
    off[u + 1] = off[u] + deg[u];
  }
  alias_t al;
  if (alias_build(&al, item_w, M) != SYNTH_OK) { free(off); return SYNTH_ENOMEM; }
  pairs_ctx cx = {N, M, deg, off, item_w, &al, seed, user_out, item_out, SYNTH_OK};
  parallel_range(nthreads, N, pairs_range, &cx);
  free(al.prob); free(al.alias); free(off);
  return cx.err;
}

/* nnz distinct cells of the N x M grid drawn uniformly without replacement (draw order). */
int synth_uniform_cells(int64_t N, int64_t M, int64_t nnz, uint64_t seed, int32_t *user_out, int32_t *item_out) {
  if (N <= 0 || M <= 0 || nnz < 0 || (double)N * (double)M > 4294967296.0 || nnz > N * M) return SYNTH_EINVAL;
  uint64_t cells = (uint64_t)(N * M);
  uint8_t *bits = (uint8_t *)calloc((size_t)((cells + 7) / 8), 1);
  if (!bits) return SYNTH_ENOMEM;
  uint64_t st = seed ^ ((uint64_t)ST_CELLS * STREAM_MUL);
  for (int64_t t = 0; t < nnz;) {
    uint64_t c = bounded(sm_next(&st), cells);
    if (bits[c >> 3] & (1u << (c & 7))) continue;
    bits[c >> 3] |= (uint8_t)(1u << (c & 7));
    user_out[t] = (int32_t)(c / (uint64_t)M);
    item_out[t] = (int32_t)(c % (uint64_t)M);
    ++t;
  }
  free(bits);
  return SYNTH_OK;
}

/* ---------------- normals and planted ratings ---------------- */
typedef struct { uint64_t seed, stream; double sd; float *out; } normal_ctx;
static void normal_range(void *v, int64_t lo, int64_t hi) {
  normal_ctx *c = (normal_ctx *)v;
  for (int64_t i = lo; i < hi; ++i) c->out[i] = (float)(c->sd * ctr_normal(c->seed, c->stream, (uint64_t)i));
}
/* out[i] = sd * Normal(seed, stream, i), rounded to fp32 */
int synth_normal(int64_t n, double sd, uint64_t seed, uint64_t stream, int32_t nthreads, float *out) {
  if (n < 0 || !(sd >= 0) || (!out && n > 0)) return SYNTH_EINVAL;
  normal_ctx c = {seed, 1000 + stream, sd, out};
  parallel_range(nthreads, n, normal_range, &c);
  return SYNTH_OK;
}

typedef struct {
  const int32_t *user, *item; const double *U, *V; int32_t r; double noise_sd; uint64_t seed; float *val;
  double lo, hi;
} rating_ctx;
static void rating_range(void *v, int64_t lo, int64_t hi) {
  rating_ctx *c = (rating_ctx *)v;
  for (int64_t t = lo; t < hi; ++t) {
    const double *u = c->U + (int64_t)c->user[t] * c->r;
    const double *w = c->V + (int64_t)c->item[t] * c->r;
    double s = 0;
    for (int32_t k = 0; k < c->r; ++k) s += u[k] * w[k];
    s += c->noise_sd * ctr_normal(c->seed, ST_NOISE, (uint64_t)t);
    s = rint(s);
    if (s < c->lo) s = c->lo;
    if (s > c->hi) s = c->hi;
    c->val[t] = (float)s;
  }
}
/*
 * Planted ratings: U (N x r), V (M x r) with i.i.d. N(0, factor_sd) entries, and
 *   val[t] = clip(rint(U_u . V_j + N(0, noise_sd)), lo, hi)
 * for each pair t (rint = round half to even).
 */
int synth_ratings(int64_t N, int64_t M, int64_t nnz, const int32_t *user, const int32_t *item, int32_t r,
                  double factor_sd, double noise_sd, double lo, double hi, uint64_t seed, int32_t nthreads,
                  float *val_out) {
  if (N <= 0 || M <= 0 || nnz < 0 || r <= 0) return SYNTH_EINVAL;
  double *U = (double *)malloc(sizeof(double) * (size_t)(N * r));
  double *V = (double *)malloc(sizeof(double) * (size_t)(M * r));
  if (!U || !V) { free(U); free(V); return SYNTH_ENOMEM; }
  for (int64_t i = 0; i < N * r; ++i) U[i] = factor_sd * ctr_normal(seed, ST_PLANT_U, (uint64_t)i);
  for (int64_t i = 0; i < M * r; ++i) V[i] = factor_sd * ctr_normal(seed, ST_PLANT_V, (uint64_t)i);
  for (int64_t t = 0; t < nnz; ++t)
    if (user[t] < 0 || user[t] >= N || item[t] < 0 || item[t] >= M) { free(U); free(V); return SYNTH_EINVAL; }
  rating_ctx c = {user, item, U, V, r, noise_sd, seed, val_out, lo, hi};
  parallel_range(nthreads, nnz, rating_range, &c);
  free(U); free(V);
  return SYNTH_OK;
}
