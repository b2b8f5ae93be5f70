/*
 * ORACLE — test infrastructure only.  A plain, slow, single-threaded CPU implementation
 * of LDA by collapsed Gibbs sampling under the clocked SSP / ESSP parameter server, the
 * second workload of Dai et al., arXiv 1410.8043 (Section 5: topic modeling with collapsed
 * Gibbs sampling, half of the tokens per Clock(), log-likelihood as the quality measure).
 * Only the tests, the package smoke check and the benchmark's CPU-baseline leg load it;
 * the product path never does.  It shares no code with the HIP library.
 *
 * The sampler (collapsed Gibbs sampling for LDA, Griffiths and Steyvers 2004): a token of
 * word w in document d, currently of topic k0, takes topic k with probability
 * proportional to (n_dk + alpha)(n_wk + beta) / (n_k + V beta), every count excluding the
 * token itself.
 *
 * Readings of what the paper leaves open (listed in the design notes):
 *   - the word-topic counts n_wk and the topic totals n_k are the shared parameters, one
 *     committed version per clock in a ring of s+1 versions; the doc-topic counts n_dk and
 *     the assignments z belong to the worker that owns the document (d mod P);
 *   - a clock processes one minibatch block: token t (its load index) is in block
 *     splitmix64(seed ^ t) mod B, block c mod B at clock c;
 *   - worker p at clock c reads the committed version v = max(0, c - d(p, c)) of the
 *     shared counts (the same policies as the matrix factorization: SSP_LAZY, SSP_WORST,
 *     ESSP), plus its own changes of this clock (read-my-writes inside a clock, as the
 *     sampler needs); its tokens run in (document, load index) order; at the clock
 *     boundary it INCs its changes, and version c+1 = version c + every worker's changes;
 *   - excluding the token from a view that may predate its current topic: the view's
 *     counts minus one for k0, floored at zero;
 *   - the draw is exact integer arithmetic, so that any summation order gives the same
 *     topic: p_k is evaluated in fp64 as ((n_dk + alpha) * (n_wk + beta)) / (n_k + Vbeta),
 *     Vbeta = V * beta computed once; with e the binary exponent of the largest p_k
 *     (2^e <= max p_k < 2^(e+1)) and c_K = ceil(log2 K), topic k weighs
 *     floor(p_k * 2^(62 - c_K - e)) (a scaling by a power of two is exact, and the largest
 *     weight is at least 2^(62 - c_K), so each weight keeps p_k to within one part in
 *     2^(62 - c_K) of the largest and the K weights sum below 2^63); with W the sum of the
 *     weights and r = splitmix64(seed ^ 0x5851F42D4C957F2D ^ (c << 40) ^ t), the new topic
 *     is the first k whose prefix sum of weights exceeds floor(r * W / 2^64);
 *   - log-likelihood: the collapsed log p(w, z) in fp64.
 *
 * Build: compiled with ps_mf_oracle.c into libps_mf_oracle.so (gcc -O2, no fast math).
 */
#define _GNU_SOURCE /* qsort_r */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define LO_OK 0
#define LO_EINVAL -1
#define LO_ENOMEM -2
#define LO_ESTATE -4

enum { LO_LAZY = 0, LO_WORST = 1, LO_ESSP = 2 };

typedef struct {
  int64_t D, V;
  int32_t K, P, s, policy, B;
  double alpha, beta, Vbeta;
  uint64_t seed;
  int64_t ntok;
  int32_t *doc, *word, *z;  /* tokens in load order */
  int64_t *bstart, *order;  /* tokens of block b at bstart[b]..: (worker, document, load index) order */
  int32_t *ndk;             /* D*K */
  int32_t *ring;            /* (s+1) * (V+1)*K: version v in slot v mod (s+1); row V = topic totals */
  int32_t *delta;           /* (V+1)*K: one worker's changes of the clock */
  int64_t *acc;             /* (V+1)*K: every worker's changes of the clock */
  uint64_t *w;              /* K weights */
  double *pk;               /* K unnormalised probabilities */
  int32_t clog2k;           /* ceil(log2 K) */
  int loaded;
  int64_t clock;
  int64_t *vlog;            /* clock-major v(p, c) */
  int64_t vlog_len, vlog_cap;
} lda_t;

static uint64_t lda_splitmix64(uint64_t state) {
  uint64_t z = state + 0x9E3779B97F4A7C15ULL;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static int64_t lda_view(const lda_t *o, int64_t p, int64_t c) {
  const int64_t s = o->s;
  int64_t d;
  if (o->policy == LO_LAZY) d = (c + p % (s + 1)) % (s + 1);
  else if (o->policy == LO_WORST) d = s;
  else d = s < 1 ? s : 1;
  return c - d < 0 ? 0 : c - d;
}

static int32_t *lda_slot(const lda_t *o, int64_t v) {
  return o->ring + (size_t)(v % (o->s + 1)) * (size_t)((o->V + 1) * o->K);
}

void lda_destroy(lda_t *o) {
  if (!o) return;
  free(o->doc); free(o->word); free(o->z); free(o->bstart); free(o->order); free(o->ndk); free(o->ring);
  free(o->delta); free(o->acc); free(o->w); free(o->pk); free(o->vlog);
  free(o);
}

int lda_create(int64_t D, int64_t V, int32_t K, int32_t P, int32_t s, double alpha, double beta, int32_t policy,
               int32_t B, uint64_t seed, lda_t **out) {
  if (!out) return LO_EINVAL;
  *out = NULL;
  if (D <= 0 || V <= 0 || K <= 0 || P <= 0 || s < 0 || B < 1 || policy < LO_LAZY || policy > LO_ESSP) return LO_EINVAL;
  if (!(alpha > 0) || !(beta > 0) || !isfinite(alpha) || !isfinite(beta)) return LO_EINVAL;
  lda_t *o = (lda_t *)calloc(1, sizeof(lda_t));
  if (!o) return LO_ENOMEM;
  o->D = D; o->V = V; o->K = K; o->P = P; o->s = s; o->policy = policy; o->B = B;
  o->alpha = alpha; o->beta = beta; o->Vbeta = (double)V * beta; o->seed = seed;
  while ((1LL << o->clog2k) < (int64_t)K) o->clog2k += 1;
  o->w = (uint64_t *)calloc((size_t)K, sizeof(uint64_t));
  o->pk = (double *)calloc((size_t)K, sizeof(double));
  *out = o;
  if (!o->w || !o->pk) {
    lda_destroy(o);
    *out = NULL;
    return LO_ENOMEM;
  }
  return LO_OK;
}

static int cmp_token(const void *a, const void *b, void *arg) {
  const int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
  const lda_t *o = (const lda_t *)arg;
  const int64_t px = o->doc[x] % o->P, py = o->doc[y] % o->P;
  if (px != py) return px < py ? -1 : 1;
  if (o->doc[x] != o->doc[y]) return o->doc[x] < o->doc[y] ? -1 : 1;
  return x < y ? -1 : (x > y);
}

/* tokens (document, word, initial topic); version 0 holds the counts of z0 */
int lda_load(lda_t *o, const int32_t *doc, const int32_t *word, const int32_t *z0, int64_t n) {
  if (!o || n < 0 || (n > 0 && (!doc || !word || !z0))) return LO_EINVAL;
  if (o->loaded) return LO_ESTATE;
  for (int64_t t = 0; t < n; ++t)
    if (doc[t] < 0 || doc[t] >= o->D || word[t] < 0 || word[t] >= o->V || z0[t] < 0 || z0[t] >= o->K) return LO_EINVAL;
  {
    /* every p_k must be a normal fp64 number, so that its exponent is defined: p_k lies
       between alpha beta / (tokens + V beta) and (longest document + alpha)(tokens + beta) /
       (V beta), and both must stay inside [2^-1000, 2^1000] */
    int64_t *len = (int64_t *)calloc((size_t)o->D, sizeof(int64_t)), lmax = 0;
    if (!len) return LO_ENOMEM;
    for (int64_t t = 0; t < n; ++t)
      if (++len[doc[t]] > lmax) lmax = len[doc[t]];
    free(len);
    const double hi = ((double)lmax + o->alpha) * ((double)n + o->beta) / o->Vbeta;
    const double lo = o->alpha * o->beta / ((double)n + o->Vbeta);
    if (!(hi <= ldexp(1.0, 1000)) || !(lo >= ldexp(1.0, -1000))) return LO_EINVAL;
  }
  const size_t nn = (size_t)(n > 0 ? n : 1), KV = (size_t)((o->V + 1) * o->K);
  o->doc = (int32_t *)malloc(sizeof(int32_t) * nn);
  o->word = (int32_t *)malloc(sizeof(int32_t) * nn);
  o->z = (int32_t *)malloc(sizeof(int32_t) * nn);
  o->order = (int64_t *)malloc(sizeof(int64_t) * nn);
  o->bstart = (int64_t *)calloc((size_t)o->B + 1, sizeof(int64_t));
  o->ndk = (int32_t *)calloc((size_t)(o->D * o->K), sizeof(int32_t));
  o->ring = (int32_t *)calloc(KV * (size_t)(o->s + 1), sizeof(int32_t));
  o->delta = (int32_t *)calloc(KV, sizeof(int32_t));
  o->acc = (int64_t *)calloc(KV, sizeof(int64_t));
  int32_t *blk = (int32_t *)malloc(sizeof(int32_t) * nn);
  int64_t *fill = (int64_t *)calloc((size_t)o->B, sizeof(int64_t));
  if (!o->doc || !o->word || !o->z || !o->order || !o->bstart || !o->ndk || !o->ring || !o->delta || !o->acc || !blk ||
      !fill) {
    free(blk); free(fill);
    return LO_ENOMEM;
  }
  o->ntok = n;
  if (n > 0) {
    memcpy(o->doc, doc, sizeof(int32_t) * (size_t)n);
    memcpy(o->word, word, sizeof(int32_t) * (size_t)n);
    memcpy(o->z, z0, sizeof(int32_t) * (size_t)n);
  }
  for (int64_t t = 0; t < n; ++t) {
    blk[t] = o->B == 1 ? 0 : (int32_t)(lda_splitmix64(o->seed ^ (uint64_t)t) % (uint64_t)o->B);
    o->bstart[blk[t] + 1] += 1;
    o->ndk[(int64_t)doc[t] * o->K + z0[t]] += 1;
    o->ring[(int64_t)word[t] * o->K + z0[t]] += 1;
    o->ring[o->V * o->K + z0[t]] += 1;
  }
  for (int32_t b = 0; b < o->B; ++b) o->bstart[b + 1] += o->bstart[b];
  for (int64_t t = 0; t < n; ++t) o->order[o->bstart[blk[t]] + fill[blk[t]]++] = t;
  for (int32_t b = 0; b < o->B; ++b)
    qsort_r(o->order + o->bstart[b], (size_t)(o->bstart[b + 1] - o->bstart[b]), sizeof(int64_t), cmp_token, o);
  free(blk); free(fill);
  o->loaded = 1;
  return LO_OK;
}

/* one token: the weights of its topics (into o->w) and their sum, from counts that
   include the token (it is excluded here, each count floored at zero) */
static uint64_t lda_weights(lda_t *o, const int32_t *nd, const int32_t *vw, const int32_t *dw, const int32_t *vk,
                            const int32_t *dk, int32_t k0) {
  double pmax = 0.0;
  for (int32_t k = 0; k < o->K; ++k) {
    const int32_t self = k == k0;
    int64_t ndk = (int64_t)nd[k] - self;
    int64_t nwk = (int64_t)vw[k] + dw[k] - self;
    int64_t nk = (int64_t)vk[k] + dk[k] - self;
    if (nwk < 0) nwk = 0;
    if (nk < 0) nk = 0;
    const double a = (double)ndk + o->alpha, b = (double)nwk + o->beta, c = (double)nk + o->Vbeta;
    o->pk[k] = (a * b) / c;
    if (o->pk[k] > pmax) pmax = o->pk[k];
  }
  /* scale so that the largest weight lies in [2^(62 - c_K), 2^(63 - c_K)) */
  const int shift = 62 - o->clog2k - ilogb(pmax);
  uint64_t total = 0;
  for (int32_t k = 0; k < o->K; ++k) {
    o->w[k] = (uint64_t)floor(ldexp(o->pk[k], shift));
    total += o->w[k];
  }
  return total;
}

/* the first topic whose prefix sum of weights exceeds floor(r W / 2^64) */
static int32_t lda_pick(const lda_t *o, uint64_t total, int32_t k0, uint64_t r) {
  if (total == 0) return k0; /* not reached: the largest weight is at least 2^(62 - c_K) */
  const uint64_t target = (uint64_t)(((unsigned __int128)r * total) >> 64);
  uint64_t cum = 0;
  for (int32_t k = 0; k < o->K; ++k) {
    cum += o->w[k];
    if (cum > target) return k;
  }
  return o->K - 1; /* not reached: cum ends at total > target */
}

static int32_t lda_draw(lda_t *o, const int32_t *nd, const int32_t *vw, const int32_t *dw, const int32_t *vk,
                        const int32_t *dk, int32_t k0, uint64_t r) {
  return lda_pick(o, lda_weights(o, nd, vw, dw, vk, dk, k0), k0, r);
}

/* One token's weights and draw from its counts n_dk, n_wk and n_k (each including the
   token, which sits in topic k0) and the random number r, for the tests' pins of the draw:
   w_out[K] receives the weights, *k_out the drawn topic, *total_out their sum. */
int lda_token_draw(lda_t *o, const int32_t *nd, const int32_t *nw, const int32_t *nk, int32_t k0, uint64_t r,
                   uint64_t *w_out, uint64_t *total_out, int32_t *k_out) {
  if (!o || !nd || !nw || !nk || !w_out || !total_out || !k_out || k0 < 0 || k0 >= o->K) return LO_EINVAL;
  int32_t *zero = (int32_t *)calloc((size_t)o->K, sizeof(int32_t));
  if (!zero) return LO_ENOMEM;
  const uint64_t total = lda_weights(o, nd, nw, zero, nk, zero, k0);
  memcpy(w_out, o->w, sizeof(uint64_t) * (size_t)o->K);
  *total_out = total;
  *k_out = lda_pick(o, total, k0, r);
  free(zero);
  return LO_OK;
}

static int lda_one_clock(lda_t *o) {
  const int64_t c = o->clock, K = o->K, KV = (o->V + 1) * K;
  const int32_t b = (int32_t)(c % o->B);
  memset(o->acc, 0, sizeof(int64_t) * (size_t)KV);
  int64_t q = o->bstart[b];
  for (int64_t p = 0; p < o->P; ++p) {
    const int32_t *view = lda_slot(o, lda_view(o, p, c));
    memset(o->delta, 0, sizeof(int32_t) * (size_t)KV);
    for (; q < o->bstart[b + 1] && o->doc[o->order[q]] % o->P == p; ++q) {
      const int64_t t = o->order[q];
      const int64_t d = o->doc[t], w = o->word[t];
      const int32_t k0 = o->z[t];
      const uint64_t r = lda_splitmix64(o->seed ^ 0x5851F42D4C957F2DULL ^ ((uint64_t)c << 40) ^ (uint64_t)t);
      int32_t *nd = o->ndk + d * K;
      const int32_t k1 = lda_draw(o, nd, view + w * K, o->delta + w * K, view + o->V * K, o->delta + o->V * K, k0, r);
      if (k1 != k0) {
        nd[k0] -= 1; nd[k1] += 1;
        o->delta[w * K + k0] -= 1; o->delta[w * K + k1] += 1;
        o->delta[o->V * K + k0] -= 1; o->delta[o->V * K + k1] += 1;
        o->z[t] = k1;
      }
    }
    for (int64_t x = 0; x < KV; ++x) o->acc[x] += o->delta[x];
  }
  if (o->vlog_len + o->P > o->vlog_cap) {
    int64_t cap = o->vlog_cap ? 2 * o->vlog_cap : 64 * (int64_t)o->P;
    while (cap < o->vlog_len + o->P) cap *= 2;
    int64_t *nv = (int64_t *)realloc(o->vlog, sizeof(int64_t) * (size_t)cap);
    if (!nv) return LO_ENOMEM;
    o->vlog = nv; o->vlog_cap = cap;
  }
  for (int64_t p = 0; p < o->P; ++p) o->vlog[o->vlog_len++] = lda_view(o, p, c);
  const int32_t *cur = lda_slot(o, c);
  int32_t *next = lda_slot(o, c + 1);
  for (int64_t x = 0; x < KV; ++x) next[x] = (int32_t)((int64_t)cur[x] + o->acc[x]);
  o->clock = c + 1;
  return LO_OK;
}

int lda_clock(lda_t *o, int32_t n) {
  if (!o || n < 0) return LO_EINVAL;
  if (!o->loaded) return LO_ESTATE;
  for (int32_t i = 0; i < n; ++i) {
    const int rc = lda_one_clock(o);
    if (rc) return rc;
  }
  return LO_OK;
}

/* the collapsed log p(w, z) at the latest version, fp64 */
int lda_loglik(const lda_t *o, double *out) {
  if (!o || !out) return LO_EINVAL;
  if (!o->loaded) return LO_ESTATE;
  const int32_t *n = lda_slot(o, o->clock);
  const int64_t K = o->K;
  double ll = 0.0;
  for (int64_t k = 0; k < K; ++k) {
    double t = lgamma(o->Vbeta) - lgamma((double)n[o->V * K + k] + o->Vbeta);
    for (int64_t w = 0; w < o->V; ++w) t += lgamma((double)n[w * K + k] + o->beta) - lgamma(o->beta);
    ll += t;
  }
  const double Ka = (double)K * o->alpha;
  for (int64_t d = 0; d < o->D; ++d) {
    int64_t len = 0;
    double t = lgamma(Ka);
    for (int64_t k = 0; k < K; ++k) {
      len += o->ndk[d * K + k];
      t += lgamma((double)o->ndk[d * K + k] + o->alpha) - lgamma(o->alpha);
    }
    ll += t - lgamma((double)len + Ka);
  }
  *out = ll;
  return LO_OK;
}

/* exports: 0 = z [ntok] int32 (load order); 1 = ndk [D*K] int32; 2 = nwk [(V+1)*K] int32 of the
   latest version (row V: topic totals); 3 = version log [clocks*P] int64; 4 = block order
   of block b [nnz_b] int64 (load indices in (worker, document, load index) order) */
int lda_export(const lda_t *o, int32_t kind, int32_t b, void *buf, int64_t cap, int64_t *len) {
  if (!o || !len) return LO_EINVAL;
  if (!o->loaded && kind != 3) return LO_ESTATE;
  int64_t n;
  switch (kind) {
    case 0: n = o->ntok; break;
    case 1: n = o->D * o->K; break;
    case 2: n = (o->V + 1) * o->K; break;
    case 3: n = o->vlog_len; break;
    case 4:
      if (b < 0 || b >= o->B) return LO_EINVAL;
      n = o->bstart[b + 1] - o->bstart[b];
      break;
    default: return LO_EINVAL;
  }
  *len = n;
  if (!buf) return LO_OK;
  if (cap < n) return LO_EINVAL;
  if (n == 0) return LO_OK;
  switch (kind) {
    case 0: memcpy(buf, o->z, sizeof(int32_t) * (size_t)n); break;
    case 1: memcpy(buf, o->ndk, sizeof(int32_t) * (size_t)n); break;
    case 2: memcpy(buf, lda_slot(o, o->clock), sizeof(int32_t) * (size_t)n); break;
    case 3: memcpy(buf, o->vlog, sizeof(int64_t) * (size_t)n); break;
    case 4: memcpy(buf, o->order + o->bstart[b], sizeof(int64_t) * (size_t)n); break;
  }
  return LO_OK;
}
