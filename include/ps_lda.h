/*
 * ps_lda — LDA by collapsed Gibbs sampling under clocked SSP / ESSP on one MI355X (gfx950),
 * P logical workers emulated on one GPU.  C ABI: plain host pointers and sizes only.
 *
 * The method (Dai et al., arXiv 1410.8043, Section 5, the topic-modeling workload): the
 * shared parameters are the word-topic counts n_wk and the topic totals n_k, kept by the
 * parameter server under SSP or ESSP (Sections 2.2 and 3.2); the documents are partitioned
 * over workers, and each Clock() processes a minibatch of the tokens.  A token of word w in
 * document d, currently of topic k0, is resampled from the collapsed conditional
 * (Griffiths and Steyvers 2004)
 *     p(k) proportional to (n_dk + alpha)(n_wk + beta) / (n_k + V beta),
 * every count excluding the token itself; the quality measure is the log-likelihood.
 *
 * Semantics implemented (readings of points the paper leaves open):
 *   - document d belongs to worker d mod P, which alone keeps its doc-topic counts n_dk and
 *     its tokens' assignments z;
 *   - token t (its index in the load order) is in minibatch block splitmix64(seed ^ t) mod B
 *     (splitmix64(x): one step of the SplitMix64 generator from state x); clock c processes
 *     block c mod B;
 *   - worker p at clock c reads committed version v(p, c) = max(0, c - d(p, c)) of the
 *     shared counts, d from the policy as for ps_mf (SSP_LAZY (c + p mod (s+1)) mod (s+1),
 *     SSP_WORST s, ESSP min(s, 1)), plus its own changes of this clock (read-my-writes), and
 *     runs its tokens of the block in (document, load index) order; version c+1 = version c
 *     + every worker's changes of clock c (integer counts: exact in any summation order);
 *   - a count that excludes the token is the view's count (plus own changes) minus one for
 *     k0, floored at zero (a stale view may predate the token's current topic);
 *   - the draw is exact integer arithmetic: p_k is evaluated in IEEE fp64 as
 *     ((n_dk + alpha) * (n_wk + beta)) / (n_k + Vbeta), Vbeta = V * beta; with e the binary
 *     exponent of the token's largest p_k and c_K = ceil(log2 K), topic k weighs
 *     floor(p_k * 2^(62 - c_K - e)) (exact scaling; the weights keep every p_k to within
 *     2^-(62 - c_K) of the largest, and sum below 2^63); with W the sum of the weights and
 *     r = splitmix64(seed ^ 0x5851F42D4C957F2D ^ (c << 40) ^ t), the new topic is the first k
 *     whose prefix sum of weights exceeds floor(r W / 2^64);
 *   - log-likelihood: the collapsed log p(w, z) of the latest version and the doc-topic
 *     counts, in fp64.
 *
 * Storage: counts are int32.  The handle keeps a ring of s+2 committed versions of the
 * (V+1) x K counts (row V: the topic totals) in HBM, version v in slot v mod (s+2), so the
 * version being built never overwrites a version some worker still reads.
 *
 * Conventions: as ps_mf — PS_LDA_OK (0) or a negative code with ps_lda_last_error(); host
 * inputs are copied before the call returns; outputs belong to the caller; the handle owns
 * the device memory; calls on one handle must not overlap; kernels run on the handle's
 * stream, asynchronously unless the call says it synchronizes.
 */
#ifndef PS_LDA_H
#define PS_LDA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ps_lda ps_lda_t;

#define PS_LDA_OK 0
#define PS_LDA_EINVAL (-1) /* bad argument: sizes, ranges, non-finite or non-positive priors, keys */
#define PS_LDA_ENOMEM (-2) /* allocation failed */
#define PS_LDA_EDEVICE (-3) /* a HIP call failed */
#define PS_LDA_ESTATE (-4) /* call out of order (clock before load, options after load) */

/* option keys (ps_lda_set_option), all before ps_lda_load */
#define PS_LDA_OPT_POLICY 1    /* PS_LDA_SSP_LAZY, PS_LDA_SSP_WORST, PS_LDA_ESSP (default) */
#define PS_LDA_OPT_MB_BLOCKS 2 /* B >= 1 (default 2: half of the tokens per clock) */
#define PS_LDA_OPT_SEED 3      /* 64-bit seed of the block hash and the draws (default 0) */
#define PS_LDA_OPT_HOST_ONLY 4 /* 1: build and export the token layout only; never touch a device */
#define PS_LDA_OPT_TIMING 5    /* 1: HIP events around every sampling kernel (ps_lda_kernel_time) */
#define PS_LDA_OPT_FLAT_ADDRESSING 6 /* 1: the sampling kernel addresses its tables with 64-bit
                                        offsets (default 0: 32-bit buffer offsets whenever every
                                        table is under 2 GiB, 64-bit otherwise); same results */

#define PS_LDA_SSP_LAZY 0
#define PS_LDA_SSP_WORST 1
#define PS_LDA_ESSP 2

/* export kinds (ps_lda_export) */
#define PS_LDA_X_Z 0           /* int32 [tokens]: topic of every token, load order */
#define PS_LDA_X_NDK 1         /* int32 [D*K]: doc-topic counts, row-major */
#define PS_LDA_X_NWK 2         /* int32 [(V+1)*K]: latest version, row V the topic totals */
#define PS_LDA_X_VERSION_LOG 3 /* int64 [clocks*P]: v(p, c), clock-major */
#define PS_LDA_X_BLOCK_ORDER 4 /* int64 [tokens of block b]: load indices in processing order */

/* D documents, V words, 1 <= K <= 512 topics, P workers, staleness s; alpha, beta > 0. */
int ps_lda_create(int64_t D, int64_t V, int32_t K, int32_t P, int32_t s, double alpha, double beta,
                  ps_lda_t **out);
int ps_lda_set_option(ps_lda_t *h, int32_t key, int64_t value);
/* hip_stream: a hipStream_t of the current device, or NULL for a stream the handle creates. */
int ps_lda_set_stream(ps_lda_t *h, void *hip_stream);
/* n tokens as host arrays: document, word, initial topic (0 <= doc < D, word < V, z0 < K).
   Version 0 holds the counts of z0.  Synchronizes.  PS_LDA_EINVAL also when a weight p_k,
   its numerator (n_dk + alpha)(n_wk + beta) or its denominator n_k + V beta could leave
   [2^-700, 2^700] (p_k must be a normal fp64 number, and the sampler divides by a short form
   that is exact there): each of alpha beta, (longest document + alpha)(n + beta), V beta,
   n + V beta, alpha beta / (n + V beta) and (longest document + alpha)(n + beta) / (V beta)
   must lie in that range. */
int ps_lda_load(ps_lda_t *h, const int32_t *doc, const int32_t *word, const int32_t *z0, int64_t n);
/* run n clocks (asynchronous) */
int ps_lda_clock(ps_lda_t *h, int32_t n);
/* collapsed log p(w, z) of the latest state; synchronizes */
int ps_lda_loglik(ps_lda_t *h, double *out);
int ps_lda_get_clock(ps_lda_t *h, int64_t *clock);
/* copy an export into buf (capacity cap elements); *len = its length; buf NULL: length only.
   Synchronizes. */
int ps_lda_export(ps_lda_t *h, int32_t kind, int32_t block, void *buf, int64_t cap, int64_t *len);
/* summed milliseconds and count of the sampling kernel's launches (PS_LDA_OPT_TIMING) */
int ps_lda_kernel_time(ps_lda_t *h, double *ms, int64_t *count);
const char *ps_lda_last_error(const ps_lda_t *h);
void ps_lda_destroy(ps_lda_t *h);

#ifdef __cplusplus
}
#endif

#endif
