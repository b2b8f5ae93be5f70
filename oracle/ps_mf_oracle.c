/*
 * ORACLE — test infrastructure only.  A plain, slow, single-threaded CPU implementation
 * of the clocked SSP/ESSP matrix-factorization SGD that the HIP library computes.  Only
 * the tests, the package smoke check and the benchmark's CPU-baseline leg may load it;
 * the product path never does.  It shares no code with the HIP library.
 *
 * What it computes (Dai et al., arXiv 1410.8043):
 *   - objective: sum over observed (i,j) of (D_ij - L_i . R_j)^2 + lambda(|L|_F^2 + |R|_F^2)
 *     (Section 3.1); the factor 2 of the gradient is absorbed into the step (Section 3.1);
 *   - per-rating update (Section 3.1):  e_ij = D_ij - L_i . R_j,
 *       L_i += eta (e_ij R_j - lambda L_i),   R_j += eta (e_ij L_i - lambda R_j);
 *   - P workers own disjoint rating shards (Section 3.1: data partitioned over workers);
 *     a clock is one minibatch of each worker's shard (Section 5, Clock() per minibatch);
 *   - SSP bounded staleness (Section 3.2, formal SSP condition): the view of worker p at
 *     clock c contains every update of clocks <= c-s-1 plus any subset of the window;
 *     ESSP (Section 2.2, Section 4) is an implementation that pushes fresh rows eagerly;
 *   - the reference sequence x_{c+1} = x_c + sum_p u_{p,c} (Section 3.2, the "true"
 *     sequence); updates are coalesced and applied at the clock boundary (Section 4).
 *
 * Readings of points the paper leaves open (each is listed in the design notes):
 *   - one fixed view per (worker, clock); a worker's contributions within a clock are
 *     summed (no read-my-writes inside a clock);
 *   - the view is a whole committed version v = max(0, c - d(p,c)), d chosen by a
 *     deterministic policy: SSP_LAZY d = (c + p mod (s+1)) mod (s+1); SSP_WORST d = s;
 *     ESSP d = min(s, 1);
 *   - or, under the per-row policies, every row has its own version in the cache of the
 *     worker's client (Section 4: each PS process caches rows, a row served only while
 *     fresh enough, read as version >= c - s).  SSP_ROW (SSPTable: refreshed only when
 *     too stale): a row read at clock c that is not cached or cached at a version < c - s
 *     is fetched at version c, else the cached version is read.  ESSP_ROW (ESSPTable: the
 *     server pushes every registered row once all clients ticked; the push lands one
 *     clock later): the first read fetches version c, later reads see c - min(s, 1);
 *   - or VAP (Section 2.1 / Section 3, the VAP condition): the in-transit updates of a
 *     view, x_c - x_v, must satisfy |x_c - x_v|_inf <= v_t = v0 / sqrt(t), t = c + 1; every
 *     worker reads the stalest version v = c - d, d <= min(c, s), within that bound (the
 *     max-norm of fp32 differences, compared in fp64);
 *   - optional step schedule eta_c = eta / sqrt(c + 1) (the schedule of Section 3's
 *     theorems), else constant eta;
 *   - step normalisation: SUM uses the summed per-rating steps; ROWMEAN divides each
 *     row's summed contribution by that row's rating count in the clock's minibatch;
 *   - or SEQ: each worker applies the Section 3.1 update rating by rating to its own copy
 *     of the rows it reads (read-my-writes inside the clock), starting from its view (under
 *     a per-row policy, each row at the version its client's cache holds); at
 *     the clock boundary it commits (copy - view) for every row it touched, and the
 *     server adds the commits of all workers (Section 4: updates coalesced per clock).
 *     The order inside a worker is stratified into G sub-epochs: user group
 *     ug(i) = (i div P) mod G, item group ig(j) = j mod G, and rating (i, j) belongs to
 *     sub-epoch (ig(j) - ug(i)) mod G; the sub-epochs run in order, each in canonical
 *     order.  One sub-epoch's (user group, item group) strata share no row, so running
 *     them side by side gives the same result;
 *   - the lambda term enters once per rating, at the view (Section 3.1 update rule);
 *   - minibatch block of a rating: splitmix64(seed ^ (i<<32 | j)) mod B, block c mod B
 *     at clock c; rows with no rating in the block are left unchanged;
 *   - ratings are visited in canonical (i, j, load index) order inside a block, so the
 *     result does not depend on which worker owns which shard;
 *   - versions are stored in fp32; all arithmetic is fp64; a new version is rounded once:
 *     V_{c+1} = fp32(fp64(V_c) + Delta);
 *   - loss (Section 5: squared loss, not the penalised objective) is
 *     sum over all ratings (D_ij - L_i . R_j)^2 at the latest version, in fp64.
 *
 * Build: gcc -O2 -fPIC -shared -std=c11 ps_mf_oracle.c -o libps_mf_oracle.so
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_OK 0
#define OR_EINVAL -1
#define OR_ENOMEM -2
#define OR_ESTATE -4

enum { OR_LAZY = 0, OR_WORST = 1, OR_ESSP = 2, OR_SSP_ROW = 3, OR_ESSP_ROW = 4, OR_VAP = 5 };
enum { OR_ROWMEAN = 0, OR_SUM = 1, OR_SEQ = 2 };
enum { OR_X_OWNER = 0, OR_X_ROW_PTR = 1, OR_X_COL = 2, OR_X_PERM = 3, OR_X_USER_COUNT = 4, OR_X_ITEM_COUNT = 5,
       OR_X_VERSION_LOG = 6, OR_X_STALENESS = 7, OR_X_ROW_VERSIONS = 8, OR_X_SEQ_ORDER = 9, OR_X_VAP_NORMS = 10 };

typedef struct {
  int64_t N, M;
  int32_t K, P, s, policy, step, B;
  double eta, lambda;
  uint64_t seed;
  int32_t *owner; /* N */
  /* ratings as loaded */
  int64_t nnz;
  int32_t *user, *item;
  float *val;
  /* canonical layout: ratings of block b are order[bstart[b] .. bstart[b+1]) */
  int64_t *bstart;  /* B+1 */
  int64_t *order;   /* nnz: load indices */
  int32_t *ucount;  /* B*N */
  int32_t *icount;  /* B*M */
  int loaded, has_factors;
  /* ring of s+1 committed versions; version v lives in slot v mod (s+1) */
  float *Lring, *Rring;
  int64_t clock;
  /* version log, clock-major: entry c*P + p = v(p,c) */
  int64_t *vlog;
  int64_t vlog_len, vlog_cap;
  /* staleness profile (Fig. 1 left): stale[d] = parameter reads at clock c that saw
     version c - d, i.e. whose clock differential (parameter age - local clock) is -(d+1);
     every rating a worker processes reads its user row and its item row */
  int64_t *stale; /* s+1 */
  double *dL, *dR;
  /* per-row caches (Section 4, the client cache of a PS process), used by the per-row
     policies: worker p runs on client p mod C, C = min(P, s+1); each client caches the rows
     its workers read with the version it holds (-1: not cached).  A user row is read only
     by its owner's client. */
  int64_t C;
  int64_t *ucache; /* N */
  int64_t *icache; /* C*M */
  uint8_t *iread;  /* C*M scratch: item rows a client reads this clock */
  /* step SEQ: G sub-epochs; sorder holds the entries of each block (load indices, at
     bstart[b] ..) in the order (sub-epoch, worker, user group, canonical); each worker's
     copies of the rows it touched this clock (fp64): Lloc [N*K], Rloc [P*M*K] */
  int32_t G;
  int64_t *sorder;
  double *Lloc, *Rloc;
  uint8_t *utouch, *itouch; /* N, P*M */
  /* policy VAP: the value bound v0, the delay d of each clock run and, per clock, the
     in-transit norms |x_c - x_{c-d}|_inf for d = 0..s (-1 where c - d < 0) */
  double v0;
  int64_t *vap_d;
  double *vap_norm;
  int64_t vap_cap;
  int eta_decay;
} oracle_t;

/* SplitMix64 (Steele, Lea & Flood 2014): one step of the sequential generator from `state`. */
static uint64_t splitmix64_next(uint64_t state) {
  uint64_t z = state + 0x9E3779B97F4A7C15ULL;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

int oracle_splitmix64(uint64_t state, uint64_t *out) {
  *out = splitmix64_next(state);
  return OR_OK;
}

/* minibatch block of rating (i, j) */
static int32_t block_of(const oracle_t *o, int64_t i, int64_t j) {
  if (o->B == 1) return 0;
  uint64_t key = o->seed ^ (((uint64_t)i << 32) | (uint64_t)(uint32_t)j);
  return (int32_t)(splitmix64_next(key) % (uint64_t)o->B);
}

/* staleness d(p, c) chosen by the policy; always in [0, s] */
static int64_t delay_of(const oracle_t *o, int64_t p, int64_t c) {
  int64_t s = o->s;
  switch (o->policy) {
    case OR_LAZY: return (c + p % (s + 1)) % (s + 1);
    case OR_WORST: return s;
    case OR_VAP: return o->vap_d[c]; /* chosen when clock c starts */
    default: return s < 1 ? s : 1; /* ESSP */
  }
}

/* the committed version worker p reads at clock c */
static int64_t view_version(const oracle_t *o, int64_t p, int64_t c) {
  int64_t v = c - delay_of(o, p, c);
  return v < 0 ? 0 : v;
}

static int per_row(const oracle_t *o) { return o->policy == OR_SSP_ROW || o->policy == OR_ESSP_ROW; }

/* the version a client's cache holds for a row it reads at clock c (cached: its current
   version, -1 if none) */
static int64_t row_read(const oracle_t *o, int64_t cached, int64_t c) {
  if (o->policy == OR_SSP_ROW) return (cached < 0 || cached < c - o->s) ? c : cached;
  /* ESSP_ROW */
  if (cached < 0) return c;
  return c - (o->s < 1 ? o->s : 1);
}

int oracle_view_version(const oracle_t *o, int64_t p, int64_t c, int64_t *v) {
  if (!o || p < 0 || p >= o->P || c < 0 || per_row(o)) return OR_EINVAL;
  if (o->policy == OR_VAP && c >= o->clock) return OR_EINVAL; /* chosen when the clock runs */
  *v = view_version(o, p, c);
  return OR_OK;
}

void oracle_destroy(oracle_t *o) {
  if (!o) return;
  free(o->owner); free(o->user); free(o->item); free(o->val);
  free(o->bstart); free(o->order); free(o->ucount); free(o->icount);
  free(o->Lring); free(o->Rring); free(o->vlog); free(o->dL); free(o->dR); free(o->stale);
  free(o->ucache); free(o->icache); free(o->iread);
  free(o->sorder); free(o->Lloc); free(o->Rloc); free(o->utouch); free(o->itouch);
  free(o->vap_d); free(o->vap_norm);
  free(o);
}

int oracle_create(int64_t N, int64_t M, int32_t K, int32_t P, int32_t s, double eta, double lambda, int32_t policy,
                  int32_t step, int32_t B, uint64_t seed, const int32_t *owner, oracle_t **out) {
  if (!out) return OR_EINVAL;
  *out = NULL;
  if (N <= 0 || M <= 0 || K <= 0 || P <= 0 || s < 0 || B < 1 || N > 0x7fffffff || M > 0x7fffffff) return OR_EINVAL;
  if (policy < OR_LAZY || policy > OR_VAP || step < OR_ROWMEAN || step > OR_SEQ) return OR_EINVAL;
  if (!isfinite(eta) || !isfinite(lambda)) return OR_EINVAL;
  oracle_t *o = (oracle_t *)calloc(1, sizeof(oracle_t));
  if (!o) return OR_ENOMEM;
  o->N = N; o->M = M; o->K = K; o->P = P; o->s = s; o->eta = eta; o->lambda = lambda;
  o->policy = policy; o->step = step; o->B = B; o->seed = seed;
  o->G = 256;
  o->v0 = INFINITY;
  o->owner = (int32_t *)malloc(sizeof(int32_t) * (size_t)N);
  o->stale = (int64_t *)calloc((size_t)s + 1, sizeof(int64_t));
  o->C = P < (int64_t)s + 1 ? P : (int64_t)s + 1;
  o->ucache = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
  o->icache = (int64_t *)malloc(sizeof(int64_t) * (size_t)(o->C * M));
  o->iread = (uint8_t *)calloc((size_t)(o->C * M), 1);
  if (!o->owner || !o->stale || !o->ucache || !o->icache || !o->iread) { oracle_destroy(o); return OR_ENOMEM; }
  for (int64_t i = 0; i < N; ++i) o->ucache[i] = -1;
  for (int64_t x = 0; x < o->C * M; ++x) o->icache[x] = -1;
  for (int64_t i = 0; i < N; ++i) {
    int32_t p = owner ? owner[i] : (int32_t)(i % P);
    if (p < 0 || p >= P) { oracle_destroy(o); return OR_EINVAL; }
    o->owner[i] = p;
  }
  *out = o;
  return OR_OK;
}

/* number of sub-epochs G of the SEQ step (default 256); before load */
int oracle_set_strata(oracle_t *o, int32_t G) {
  if (!o || G < 1) return OR_EINVAL;
  if (o->loaded) return OR_ESTATE;
  o->G = G;
  return OR_OK;
}

/* the value bound v0 of the VAP policy (default: unbounded); before load; v0 >= 0 */
int oracle_set_value_bound(oracle_t *o, double v0) {
  if (!o || !(v0 >= 0)) return OR_EINVAL;
  if (o->loaded) return OR_ESTATE;
  o->v0 = v0;
  return OR_OK;
}

/* step schedule eta_c = eta / sqrt(c + 1) (on != 0) or constant eta; before load */
int oracle_set_eta_decay(oracle_t *o, int32_t on) {
  if (!o) return OR_EINVAL;
  if (o->loaded) return OR_ESTATE;
  o->eta_decay = on != 0;
  return OR_OK;
}

/* sub-epoch of rating (i, j) under the SEQ step */
static int64_t sub_epoch(const oracle_t *o, int64_t i, int64_t j) {
  const int64_t ug = (i / o->P) % o->G, ig = j % o->G;
  return ((ig - ug) % o->G + o->G) % o->G;
}

/* stable counting sort of a[0..n) by key(x) in [0, range) into out */
static int stable_by_key(const oracle_t *o, const int64_t *a, int64_t n, int64_t range, int which, int64_t *out) {
  int64_t *cnt = (int64_t *)calloc((size_t)range + 1, sizeof(int64_t));
  if (!cnt) return OR_ENOMEM;
  for (int64_t q = 0; q < n; ++q) {
    const int64_t i = o->user[a[q]], j = o->item[a[q]];
    const int64_t k = which == 0 ? (i / o->P) % o->G : sub_epoch(o, i, j) * o->P + o->owner[i];
    cnt[k + 1] += 1;
  }
  for (int64_t k = 0; k < range; ++k) cnt[k + 1] += cnt[k];
  for (int64_t q = 0; q < n; ++q) {
    const int64_t i = o->user[a[q]], j = o->item[a[q]];
    const int64_t k = which == 0 ? (i / o->P) % o->G : sub_epoch(o, i, j) * o->P + o->owner[i];
    out[cnt[k]++] = a[q];
  }
  free(cnt);
  return OR_OK;
}

/* canonical order inside a block: (user, item, load index) */
static const oracle_t *g_sort_ctx;
static int cmp_canonical(const void *a, const void *b) {
  int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
  const oracle_t *o = g_sort_ctx;
  if (o->user[x] != o->user[y]) return o->user[x] < o->user[y] ? -1 : 1;
  if (o->item[x] != o->item[y]) return o->item[x] < o->item[y] ? -1 : 1;
  return x < y ? -1 : (x > y);
}

int oracle_load(oracle_t *o, const int32_t *user, const int32_t *item, const float *val, int64_t nnz) {
  if (!o || nnz < 0 || (nnz > 0 && (!user || !item || !val))) return OR_EINVAL;
  if (o->loaded) return OR_ESTATE;
  for (int64_t t = 0; t < nnz; ++t)
    if (user[t] < 0 || user[t] >= o->N || item[t] < 0 || item[t] >= o->M || !isfinite(val[t])) return OR_EINVAL;
  size_t n = (size_t)(nnz > 0 ? nnz : 1);
  o->user = (int32_t *)malloc(sizeof(int32_t) * n);
  o->item = (int32_t *)malloc(sizeof(int32_t) * n);
  o->val = (float *)malloc(sizeof(float) * n);
  o->order = (int64_t *)malloc(sizeof(int64_t) * n);
  o->bstart = (int64_t *)calloc((size_t)o->B + 1, sizeof(int64_t));
  o->ucount = (int32_t *)calloc((size_t)(o->B * o->N), sizeof(int32_t));
  o->icount = (int32_t *)calloc((size_t)(o->B * o->M), sizeof(int32_t));
  int32_t *blk = (int32_t *)malloc(sizeof(int32_t) * n);
  int64_t *fill = (int64_t *)calloc((size_t)o->B, sizeof(int64_t));
  if (!o->user || !o->item || !o->val || !o->order || !o->bstart || !o->ucount || !o->icount || !blk || !fill) {
    free(blk); free(fill);
    return OR_ENOMEM;
  }
  o->nnz = nnz;
  if (nnz > 0) {
    memcpy(o->user, user, sizeof(int32_t) * (size_t)nnz);
    memcpy(o->item, item, sizeof(int32_t) * (size_t)nnz);
    memcpy(o->val, val, sizeof(float) * (size_t)nnz);
  }
  /* bucket by block, then sort each bucket canonically */
  for (int64_t t = 0; t < nnz; ++t) {
    blk[t] = block_of(o, user[t], item[t]);
    o->bstart[blk[t] + 1] += 1;
    o->ucount[(int64_t)blk[t] * o->N + user[t]] += 1;
    o->icount[(int64_t)blk[t] * o->M + item[t]] += 1;
  }
  for (int32_t b = 0; b < o->B; ++b) o->bstart[b + 1] += o->bstart[b];
  for (int64_t t = 0; t < nnz; ++t) o->order[o->bstart[blk[t]] + fill[blk[t]]++] = t;
  g_sort_ctx = o;
  for (int32_t b = 0; b < o->B; ++b)
    qsort(o->order + o->bstart[b], (size_t)(o->bstart[b + 1] - o->bstart[b]), sizeof(int64_t), cmp_canonical);
  free(blk); free(fill);
  if (o->step == OR_SEQ) {
    /* the order each worker applies its ratings in: canonical order, stably sorted by user
       group, then by (sub-epoch, worker) */
    o->sorder = (int64_t *)malloc(sizeof(int64_t) * n);
    int64_t *tmp = (int64_t *)malloc(sizeof(int64_t) * n);
    if (!o->sorder || !tmp) { free(tmp); return OR_ENOMEM; }
    for (int32_t b = 0; b < o->B; ++b) {
      const int64_t lo = o->bstart[b], nb = o->bstart[b + 1] - lo;
      int rc = stable_by_key(o, o->order + lo, nb, o->G, 0, tmp);
      if (!rc) rc = stable_by_key(o, tmp, nb, (int64_t)o->G * o->P, 1, o->sorder + lo);
      if (rc) { free(tmp); return rc; }
    }
    free(tmp);
  }
  o->loaded = 1;
  return OR_OK;
}

int oracle_set_factors(oracle_t *o, const float *L0, const float *R0) {
  if (!o || !L0 || !R0) return OR_EINVAL;
  size_t nl = (size_t)(o->N * o->K), nr = (size_t)(o->M * o->K);
  for (size_t x = 0; x < nl; ++x) if (!isfinite(L0[x])) return OR_EINVAL;
  for (size_t x = 0; x < nr; ++x) if (!isfinite(R0[x])) return OR_EINVAL;
  if (!o->Lring) {
    o->Lring = (float *)malloc(sizeof(float) * nl * (size_t)(o->s + 1));
    o->Rring = (float *)malloc(sizeof(float) * nr * (size_t)(o->s + 1));
    o->dL = (double *)malloc(sizeof(double) * nl);
    o->dR = (double *)malloc(sizeof(double) * nr);
    if (!o->Lring || !o->Rring || !o->dL || !o->dR) return OR_ENOMEM;
  }
  /* version 0 in slot 0 */
  memcpy(o->Lring, L0, sizeof(float) * nl);
  memcpy(o->Rring, R0, sizeof(float) * nr);
  o->clock = 0;
  o->vlog_len = 0;
  memset(o->stale, 0, sizeof(int64_t) * ((size_t)o->s + 1));
  for (int64_t i = 0; i < o->N; ++i) o->ucache[i] = -1;
  for (int64_t x = 0; x < o->C * o->M; ++x) o->icache[x] = -1;
  o->has_factors = 1;
  return OR_OK;
}

static float *L_of(const oracle_t *o, int64_t v) { return o->Lring + (size_t)(v % (o->s + 1)) * (size_t)(o->N * o->K); }
static float *R_of(const oracle_t *o, int64_t v) { return o->Rring + (size_t)(v % (o->s + 1)) * (size_t)(o->M * o->K); }

/* the version worker p's view holds for user row i / item row j at clock c: the worker's
   whole view, or under a per-row policy the version its client's cache holds */
static int64_t seq_view_L(const oracle_t *o, int64_t i, int64_t c) {
  return per_row(o) ? o->ucache[i] : view_version(o, o->owner[i], c);
}
static int64_t seq_view_R(const oracle_t *o, int64_t p, int64_t j, int64_t c) {
  return per_row(o) ? o->icache[(p % o->C) * o->M + j] : view_version(o, p, c);
}

/* the SEQ step of one clock: every worker runs its ratings in its order on its own copies
   of the rows, which start at its view; dL and dR receive sum over workers of
   (copy - view) for the rows each touched */
static int seq_sweep(oracle_t *o, int64_t c, int32_t b, double eta) {
  const int64_t K = o->K, M = o->M;
  if (!o->Lloc) {
    o->Lloc = (double *)malloc(sizeof(double) * (size_t)(o->N * K));
    o->Rloc = (double *)malloc(sizeof(double) * (size_t)(o->P * M * K));
    o->utouch = (uint8_t *)calloc((size_t)o->N, 1);
    o->itouch = (uint8_t *)calloc((size_t)(o->P * M), 1);
    if (!o->Lloc || !o->Rloc || !o->utouch || !o->itouch) return OR_ENOMEM;
  }
  for (int64_t q = o->bstart[b]; q < o->bstart[b + 1]; ++q) {
    const int64_t t = o->sorder[q];
    const int64_t i = o->user[t], j = o->item[t], p = o->owner[i];
    const int64_t vL = seq_view_L(o, i, c), vR = seq_view_R(o, p, j, c);
    double *Li = o->Lloc + i * K, *Rj = o->Rloc + (p * M + j) * K;
    if (!o->utouch[i]) { /* first read of L_i this clock: the view */
      const float *src = L_of(o, vL) + i * K;
      for (int64_t k = 0; k < K; ++k) Li[k] = (double)src[k];
      o->utouch[i] = 1;
    }
    if (!o->itouch[p * M + j]) { /* first read of R_j by worker p this clock */
      const float *src = R_of(o, vR) + j * K;
      for (int64_t k = 0; k < K; ++k) Rj[k] = (double)src[k];
      o->itouch[p * M + j] = 1;
    }
    o->stale[c - vL] += 1; /* the rating reads L_i ... */
    o->stale[c - vR] += 1; /* ... and R_j of the worker's view */
    double dot = 0.0;
    for (int64_t k = 0; k < K; ++k) dot += Li[k] * Rj[k];
    const double e = (double)o->val[t] - dot;
    for (int64_t k = 0; k < K; ++k) {
      const double l = Li[k], r = Rj[k];
      Li[k] = l + eta * (e * r - o->lambda * l);
      Rj[k] = r + eta * (e * l - o->lambda * r);
    }
  }
  for (int64_t i = 0; i < o->N; ++i) {
    if (!o->utouch[i]) continue;
    const float *Lv = L_of(o, seq_view_L(o, i, c)) + i * K;
    for (int64_t k = 0; k < K; ++k) o->dL[i * K + k] = o->Lloc[i * K + k] - (double)Lv[k];
    o->utouch[i] = 0;
  }
  for (int64_t p = 0; p < o->P; ++p) {
    for (int64_t j = 0; j < M; ++j) {
      if (!o->itouch[p * M + j]) continue;
      const double *Rl = o->Rloc + (p * M + j) * K;
      const float *Rv = R_of(o, seq_view_R(o, p, j, c)) + j * K;
      for (int64_t k = 0; k < K; ++k) o->dR[j * K + k] += Rl[k] - (double)Rv[k];
      o->itouch[p * M + j] = 0;
    }
  }
  return OR_OK;
}

/* VAP: the delay of clock c, the largest d <= min(c, s) whose in-transit updates
   x_c - x_{c-d} stay within v0 / sqrt(c + 1) in max-norm (d = 0 always does) */
static int vap_choose(oracle_t *o, int64_t c) {
  const int64_t S1 = (int64_t)o->s + 1;
  if (c >= o->vap_cap) {
    int64_t cap = o->vap_cap ? 2 * o->vap_cap : 64;
    while (cap <= c) cap *= 2;
    int64_t *nd = (int64_t *)realloc(o->vap_d, sizeof(int64_t) * (size_t)cap);
    if (!nd) return OR_ENOMEM;
    o->vap_d = nd;
    double *nn = (double *)realloc(o->vap_norm, sizeof(double) * (size_t)(cap * S1));
    if (!nn) return OR_ENOMEM;
    o->vap_norm = nn;
    o->vap_cap = cap;
  }
  const double bound = o->v0 / sqrt((double)(c + 1));
  int64_t d = 0;
  for (int64_t k = 0; k < S1; ++k) {
    double nrm = -1.0;
    if (k <= c) {
      float m = 0.0f;
      const float *a = L_of(o, c), *b = L_of(o, c - k);
      for (int64_t x = 0; x < o->N * o->K; ++x) { float t = fabsf(a[x] - b[x]); if (t > m) m = t; }
      a = R_of(o, c); b = R_of(o, c - k);
      for (int64_t x = 0; x < o->M * o->K; ++x) { float t = fabsf(a[x] - b[x]); if (t > m) m = t; }
      nrm = (double)m;
      if (nrm <= bound) d = k;
    }
    o->vap_norm[c * S1 + k] = nrm;
  }
  o->vap_d[c] = d;
  return OR_OK;
}

/* one clock: every worker computes its update from its view; the sum is committed */
static int one_clock(oracle_t *o) {
  const int64_t c = o->clock, K = o->K;
  const int32_t b = (int32_t)(c % o->B);
  if (o->policy == OR_VAP) {
    int rc = vap_choose(o, c);
    if (rc) return rc;
  }
  const double eta_c = o->eta_decay ? o->eta / sqrt((double)(c + 1)) : o->eta;
  memset(o->dL, 0, sizeof(double) * (size_t)(o->N * K));
  memset(o->dR, 0, sizeof(double) * (size_t)(o->M * K));
  if (per_row(o)) {
    /* the rows each client reads this clock take the version its cache serves */
    for (int64_t i = 0; i < o->N; ++i)
      if (o->ucount[(int64_t)b * o->N + i] > 0) o->ucache[i] = row_read(o, o->ucache[i], c);
    for (int64_t q = o->bstart[b]; q < o->bstart[b + 1]; ++q) {
      const int64_t t = o->order[q];
      o->iread[(int64_t)(o->owner[o->user[t]] % o->C) * o->M + o->item[t]] = 1;
    }
    for (int64_t x = 0; x < o->C * o->M; ++x)
      if (o->iread[x]) {
        o->icache[x] = row_read(o, o->icache[x], c);
        o->iread[x] = 0;
      }
  }
  if (o->step == OR_SEQ) {
    int rc = seq_sweep(o, c, b, eta_c);
    if (rc) return rc;
  }
  for (int64_t q = o->bstart[b]; q < o->bstart[b + 1] && o->step != OR_SEQ; ++q) {
    const int64_t t = o->order[q];
    const int64_t i = o->user[t], j = o->item[t];
    int64_t vL, vR;
    if (per_row(o)) {
      vL = o->ucache[i];
      vR = o->icache[(int64_t)(o->owner[i] % o->C) * o->M + j];
    } else {
      vL = vR = view_version(o, o->owner[i], c);
    }
    const float *Li = L_of(o, vL) + i * K;
    const float *Rj = R_of(o, vR) + j * K;
    o->stale[c - vL] += 1; /* this rating reads row L_i at version vL ... */
    o->stale[c - vR] += 1; /* ... and row R_j at version vR */
    double dot = 0.0;
    for (int64_t k = 0; k < K; ++k) dot += (double)Li[k] * (double)Rj[k];
    const double e = (double)o->val[t] - dot;
    const double su = (o->step == OR_ROWMEAN) ? 1.0 / (double)o->ucount[(int64_t)b * o->N + i] : 1.0;
    const double si = (o->step == OR_ROWMEAN) ? 1.0 / (double)o->icount[(int64_t)b * o->M + j] : 1.0;
    double *dLi = o->dL + i * K, *dRj = o->dR + j * K;
    for (int64_t k = 0; k < K; ++k) {
      dLi[k] += eta_c * su * (e * (double)Rj[k] - o->lambda * (double)Li[k]);
      dRj[k] += eta_c * si * (e * (double)Li[k] - o->lambda * (double)Rj[k]);
    }
  }
  /* log the versions read at this clock (one per worker: table-level policies only) */
  if (per_row(o)) goto commit;
  if (o->vlog_len + o->P > o->vlog_cap) {
    int64_t cap = o->vlog_cap ? o->vlog_cap * 2 : 64 * (int64_t)o->P;
    while (cap < o->vlog_len + o->P) cap *= 2;
    int64_t *nv = (int64_t *)realloc(o->vlog, sizeof(int64_t) * (size_t)cap);
    if (!nv) return OR_ENOMEM;
    o->vlog = nv; o->vlog_cap = cap;
  }
  for (int64_t p = 0; p < o->P; ++p) o->vlog[o->vlog_len++] = view_version(o, p, c);
commit:;
  /* commit: V_{c+1} = fp32(V_c + Delta); the Deltas are complete, so the slot that held
     version c-s may now be overwritten */
  const float *Lc = L_of(o, c), *Rc = R_of(o, c);
  float *Ln = L_of(o, c + 1), *Rn = R_of(o, c + 1);
  for (int64_t x = 0; x < o->N * K; ++x) Ln[x] = (float)((double)Lc[x] + o->dL[x]);
  for (int64_t x = 0; x < o->M * K; ++x) Rn[x] = (float)((double)Rc[x] + o->dR[x]);
  o->clock = c + 1;
  return OR_OK;
}

int oracle_clock(oracle_t *o, int32_t n) {
  if (!o || n < 0) return OR_EINVAL;
  if (!o->loaded || !o->has_factors) return OR_ESTATE;
  for (int32_t q = 0; q < n; ++q) {
    int rc = one_clock(o);
    if (rc) return rc;
  }
  return OR_OK;
}

int oracle_get_clock(const oracle_t *o, int64_t *c) {
  if (!o || !c) return OR_EINVAL;
  *c = o->clock;
  return OR_OK;
}

/* copy committed version v (must still be in the ring: clock-s <= v <= clock) */
int oracle_get_version(const oracle_t *o, int64_t v, float *L, float *R) {
  if (!o || !L || !R) return OR_EINVAL;
  if (!o->has_factors) return OR_ESTATE;
  if (v > o->clock || v < o->clock - o->s || v < 0) return OR_EINVAL;
  memcpy(L, L_of(o, v), sizeof(float) * (size_t)(o->N * o->K));
  memcpy(R, R_of(o, v), sizeof(float) * (size_t)(o->M * o->K));
  return OR_OK;
}

/* squared loss at the latest version */
int oracle_loss(const oracle_t *o, double *out) {
  if (!o || !out) return OR_EINVAL;
  if (!o->loaded || !o->has_factors) return OR_ESTATE;
  const float *L = L_of(o, o->clock), *R = R_of(o, o->clock);
  double acc = 0.0;
  for (int64_t t = 0; t < o->nnz; ++t) {
    const float *Li = L + (int64_t)o->user[t] * o->K, *Rj = R + (int64_t)o->item[t] * o->K;
    double dot = 0.0;
    for (int64_t k = 0; k < o->K; ++k) dot += (double)Li[k] * (double)Rj[k];
    const double e = (double)o->val[t] - dot;
    acc += e * e;
  }
  *out = acc;
  return OR_OK;
}

/*
 * Rows of version (clock + nclocks) for selected users and items, advancing only those
 * rows.  Valid only while every view read in those clocks is version 0 (so the needed
 * views are the initial factors): e.g. the first clock under any policy, or clocks
 * 0..s under SSP_WORST.  The oracle's own clock does not move.
 */
int oracle_rows_from_v0(const oracle_t *o, int32_t nclocks, int64_t nu, const int64_t *users, int64_t ni,
                        const int64_t *items, float *L_out, float *R_out) {
  if (!o || nclocks < 0 || nu < 0 || ni < 0) return OR_EINVAL;
  if (!o->loaded || !o->has_factors || o->clock != 0) return OR_ESTATE;
  const int64_t K = o->K;
  if (per_row(o) && nclocks > 1) return OR_EINVAL; /* only clock 0 surely reads version 0 */
  if (o->step == OR_SEQ) return OR_EINVAL;        /* rows of a SEQ clock depend on whole chains */
  if (o->policy == OR_VAP || o->eta_decay) return OR_EINVAL;
  for (int64_t c = 0; c < nclocks && !per_row(o); ++c)
    for (int64_t p = 0; p < o->P; ++p)
      if (view_version(o, p, c) != 0) return OR_EINVAL;
  const float *L0 = L_of(o, 0), *R0 = R_of(o, 0);
  int64_t *upos = (int64_t *)malloc(sizeof(int64_t) * (size_t)o->N);
  int64_t *ipos = (int64_t *)malloc(sizeof(int64_t) * (size_t)o->M);
  double *dl = (double *)calloc((size_t)(nu * K + 1), sizeof(double));
  double *dr = (double *)calloc((size_t)(ni * K + 1), sizeof(double));
  if (!upos || !ipos || !dl || !dr) { free(upos); free(ipos); free(dl); free(dr); return OR_ENOMEM; }
  for (int64_t i = 0; i < o->N; ++i) upos[i] = -1;
  for (int64_t j = 0; j < o->M; ++j) ipos[j] = -1;
  for (int64_t a = 0; a < nu; ++a) { if (users[a] < 0 || users[a] >= o->N) goto bad; upos[users[a]] = a; }
  for (int64_t a = 0; a < ni; ++a) { if (items[a] < 0 || items[a] >= o->M) goto bad; ipos[items[a]] = a; }
  for (int64_t a = 0; a < nu; ++a) memcpy(L_out + a * K, L0 + users[a] * K, sizeof(float) * (size_t)K);
  for (int64_t a = 0; a < ni; ++a) memcpy(R_out + a * K, R0 + items[a] * K, sizeof(float) * (size_t)K);
  for (int64_t c = 0; c < nclocks; ++c) {
    const int32_t b = (int32_t)(c % o->B);
    memset(dl, 0, sizeof(double) * (size_t)(nu * K));
    memset(dr, 0, sizeof(double) * (size_t)(ni * K));
    for (int64_t q = o->bstart[b]; q < o->bstart[b + 1]; ++q) {
      const int64_t t = o->order[q];
      const int64_t i = o->user[t], j = o->item[t];
      if (upos[i] < 0 && ipos[j] < 0) continue;
      const float *Li = L0 + i * K, *Rj = R0 + j * K;
      double dot = 0.0;
      for (int64_t k = 0; k < K; ++k) dot += (double)Li[k] * (double)Rj[k];
      const double e = (double)o->val[t] - dot;
      if (upos[i] >= 0) {
        const double su = (o->step == OR_ROWMEAN) ? 1.0 / (double)o->ucount[(int64_t)b * o->N + i] : 1.0;
        double *d = dl + upos[i] * K;
        for (int64_t k = 0; k < K; ++k) d[k] += o->eta * su * (e * (double)Rj[k] - o->lambda * (double)Li[k]);
      }
      if (ipos[j] >= 0) {
        const double si = (o->step == OR_ROWMEAN) ? 1.0 / (double)o->icount[(int64_t)b * o->M + j] : 1.0;
        double *d = dr + ipos[j] * K;
        for (int64_t k = 0; k < K; ++k) d[k] += o->eta * si * (e * (double)Li[k] - o->lambda * (double)Rj[k]);
      }
    }
    for (int64_t x = 0; x < nu * K; ++x) L_out[x] = (float)((double)L_out[x] + dl[x]);
    for (int64_t x = 0; x < ni * K; ++x) R_out[x] = (float)((double)R_out[x] + dr[x]);
  }
  free(upos); free(ipos); free(dl); free(dr);
  return OR_OK;
bad:
  free(upos); free(ipos); free(dl); free(dr);
  return OR_EINVAL;
}

/*
 * Canonical integer layout, the same form the library exports:
 *   OWNER        int32 [N]
 *   ROW_PTR(b)   int64 [N+1]  prefix sums of per-user counts in block b (users in id order)
 *   COL(b)       int32 [nnz_b] items in canonical (user, item, load index) order
 *   PERM(b)      int64 [nnz_b] load indices in the same order
 *   USER_COUNT(b) int32 [N], ITEM_COUNT(b) int32 [M]
 *   VERSION_LOG  int64 [clocks * P], entry c*P + p = v(p, c)
 *   SEQ_ORDER(b) int64 [nnz_b] (step SEQ) load indices in the order the workers apply
 *                them: (sub-epoch, worker, user group, canonical)
 *   VAP_NORMS    double [clocks * (s+1)] (policy VAP) entry c*(s+1) + d = the in-transit
 *                norm |x_c - x_{c-d}|_inf seen when clock c started, -1 where c - d < 0
 */
int oracle_export(const oracle_t *o, int32_t kind, int32_t b, void *buf, int64_t cap, int64_t *len) {
  if (!o || !len) return OR_EINVAL;
  if (kind != OR_X_OWNER && kind != OR_X_VERSION_LOG && kind != OR_X_STALENESS && kind != OR_X_ROW_VERSIONS &&
      kind != OR_X_VAP_NORMS) {
    if (!o->loaded) return OR_ESTATE;
    if (b < 0 || b >= o->B) return OR_EINVAL;
  }
  int64_t n = 0;
  switch (kind) {
    case OR_X_OWNER: n = o->N; break;
    case OR_X_ROW_PTR: n = o->N + 1; break;
    case OR_X_COL: case OR_X_PERM: n = o->bstart[b + 1] - o->bstart[b]; break;
    case OR_X_USER_COUNT: n = o->N; break;
    case OR_X_ITEM_COUNT: n = o->M; break;
    case OR_X_VERSION_LOG: n = o->vlog_len; break;
    case OR_X_STALENESS: n = (int64_t)o->s + 1; break;
    case OR_X_ROW_VERSIONS: n = o->N + o->C * o->M; break;
    case OR_X_SEQ_ORDER:
      if (o->step != OR_SEQ) return OR_EINVAL;
      n = o->bstart[b + 1] - o->bstart[b];
      break;
    case OR_X_VAP_NORMS:
      if (o->policy != OR_VAP) return OR_EINVAL;
      n = o->clock * ((int64_t)o->s + 1);
      break;
    default: return OR_EINVAL;
  }
  *len = n;
  if (!buf) return OR_OK;
  if (cap < n) return OR_EINVAL;
  switch (kind) {
    case OR_X_OWNER: memcpy(buf, o->owner, sizeof(int32_t) * (size_t)n); break;
    case OR_X_ROW_PTR: {
      int64_t *rp = (int64_t *)buf;
      rp[0] = 0;
      for (int64_t i = 0; i < o->N; ++i) rp[i + 1] = rp[i] + o->ucount[(int64_t)b * o->N + i];
      break;
    }
    case OR_X_COL:
      for (int64_t q = 0; q < n; ++q) ((int32_t *)buf)[q] = o->item[o->order[o->bstart[b] + q]];
      break;
    case OR_X_PERM: memcpy(buf, o->order + o->bstart[b], sizeof(int64_t) * (size_t)n); break;
    case OR_X_USER_COUNT: memcpy(buf, o->ucount + (int64_t)b * o->N, sizeof(int32_t) * (size_t)n); break;
    case OR_X_ITEM_COUNT: memcpy(buf, o->icount + (int64_t)b * o->M, sizeof(int32_t) * (size_t)n); break;
    case OR_X_VERSION_LOG: if (n) memcpy(buf, o->vlog, sizeof(int64_t) * (size_t)n); break;
    case OR_X_STALENESS: memcpy(buf, o->stale, sizeof(int64_t) * (size_t)n); break;
    case OR_X_ROW_VERSIONS:
      memcpy(buf, o->ucache, sizeof(int64_t) * (size_t)o->N);
      memcpy((int64_t *)buf + o->N, o->icache, sizeof(int64_t) * (size_t)(o->C * o->M));
      break;
    case OR_X_SEQ_ORDER: if (n) memcpy(buf, o->sorder + o->bstart[b], sizeof(int64_t) * (size_t)n); break;
    case OR_X_VAP_NORMS: if (n) memcpy(buf, o->vap_norm, sizeof(double) * (size_t)n); break;
  }
  return OR_OK;
}
