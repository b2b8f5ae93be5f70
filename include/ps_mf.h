/*
 * ps_mf — clocked SSP / ESSP matrix-factorization SGD on one MI355X (gfx950), P logical
 * workers emulated on one GPU.  C ABI: plain host or device pointers and sizes only.
 *
 * The method (Dai et al., "High-Performance Distributed ML at Scale through Parameter
 * Server Consistency Models", arXiv 1410.8043):
 *   - Section 3.1: factor an N x M ratings matrix D into L (N x K) and R (K x M) by SGD;
 *     per observed rating e_ij = D_ij - L_i . R_j and
 *         L_i += eta (e_ij R_j - lambda L_i),   R_j += eta (e_ij L_i - lambda R_j)
 *     (the factor 2 absorbed into eta); L and R live in the parameter server, the
 *     ratings are partitioned over workers.
 *   - Section 3.2 (formal SSP condition): worker p at clock c reads a view that holds
 *     every update of clocks <= c-s-1 plus any subset of the in-window updates.
 *   - Section 2.2 / Section 4: ESSP pushes fresh rows eagerly; GET / INC / CLOCK, with
 *     the updates of a clock coalesced and applied at the clock boundary.
 *   - Section 5: one Clock() processes one minibatch; the squared loss is reported.
 *
 * Semantics implemented (readings of points the paper leaves open):
 *   - each (worker p, clock c) reads ONE committed version v(p,c) = max(0, c - d(p,c)),
 *     with d from the policy: SSP_LAZY d = (c + p mod (s+1)) mod (s+1) (staleness spread
 *     uniformly over 0..s, as a lazily refreshed cache does); SSP_WORST d = s (exactly the
 *     guaranteed pre-window); ESSP d = min(s, 1) (the eager push lands one clock later);
 *   - version c+1 = version c + the sum over workers of their clock-c updates, each
 *     computed at the worker's view (no read-my-writes inside a clock);
 *   - STEP ROWMEAN (default) divides a row's summed contribution by its number of ratings
 *     in the clock's minibatch (items: across all workers); STEP SUM does not;
 *   - or STEP SEQ: each worker applies the Section 3.1 rule rating by rating to its own
 *     copy of the rows it touches (reading its own writes inside the clock), starting
 *     from its view (under a per-row policy, each row at its cached version), and at the clock boundary version c+1 = version c + the sum over
 *     workers of (copy - view) of the rows each touched.  A worker's ratings run in G
 *     sub-epochs (PS_MF_OPT_SEQ_STRATA): user group (i div P) mod G, item group j mod G,
 *     rating (i, j) in sub-epoch (item group - user group) mod G; sub-epochs in order,
 *     each in (user, item, load index) order.  The strata of one sub-epoch share no row,
 *     so they run side by side;
 *   - minibatch block of rating (i, j) = splitmix64(seed ^ (i << 32 | j)) mod B, where
 *     splitmix64(x) is one step of the SplitMix64 generator from state x; clock c
 *     processes block c mod B; rows with no rating in the block are unchanged;
 *   - duplicate (i, j) ratings are separate terms.
 *
 * Storage: factors are fp32.  R is stored items x K row-major (the transpose of the
 * paper's K x M layout).  The handle keeps a ring of s+1 committed versions in HBM;
 * version v lives in slot v mod (s+1).
 *
 * Conventions for every call:
 *   - returns PS_MF_OK (0) or a negative code; ps_mf_last_error() gives the message;
 *   - host input arrays are copied before the call returns; output buffers belong to
 *     the caller; the handle owns all device memory it allocates;
 *   - a handle is not thread-safe; calls on one handle must not overlap;
 *   - kernels run on the handle's stream (ps_mf_set_stream), asynchronously unless the
 *     call says it synchronizes.
 */
#ifndef PS_MF_H
#define PS_MF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ps_mf ps_mf_t;

/* return codes */
#define PS_MF_OK 0
#define PS_MF_EINVAL (-1) /* bad argument: sizes, ranges, non-finite values, unknown keys */
#define PS_MF_ENOMEM (-2) /* host or device allocation failed; the handle stays destroyable */
#define PS_MF_EDEVICE (-3) /* a HIP call failed (no device, launch error, fault) */
#define PS_MF_ESTATE (-4) /* call out of order (e.g. clock before load and set_factors) */
#define PS_MF_EINTERNAL (-5) /* the library's own consistency check of its layout failed (a bug) */

/* option keys (ps_mf_set_option); all must be set before ps_mf_load_ratings */
#define PS_MF_OPT_POLICY 1    /* PS_MF_SSP_LAZY (default), PS_MF_SSP_WORST, PS_MF_ESSP, PS_MF_SSP_ROW,
                                 PS_MF_ESSP_ROW, PS_MF_VAP */
#define PS_MF_OPT_STEP 2      /* PS_MF_STEP_ROWMEAN (default), PS_MF_STEP_SUM, PS_MF_STEP_SEQ */
#define PS_MF_OPT_MB_BLOCKS 3 /* B >= 1 minibatch blocks (default 1: full shard per clock) */
#define PS_MF_OPT_MB_SEED 4   /* 64-bit seed of the block hash (default 0) */
#define PS_MF_OPT_HOST_ONLY 5 /* 1: build, self-check and export the integer layout only; never touch
                                 a device (a failed self-check returns PS_MF_EINTERNAL) */
#define PS_MF_OPT_TIMING 6    /* 1: record HIP events around every kernel (ps_mf_kernel_time) */
#define PS_MF_OPT_TILE_BYTES 7 /* bytes of user rows per tile of the item-major sweep (default 6 MiB:
                                  about one XCD's 4 MiB L2; larger tiles mean fewer partial rows);
                                  >= 1 */
#define PS_MF_OPT_UNIT_MAX 8   /* ratings per sweep work unit (default 256); >= 1 */
#define PS_MF_OPT_CELLS 9      /* 1 (default): sweep the dense part (users with many ratings) through
                                  LDS-staged cells; 0: every rating through the L2 work units */
#define PS_MF_OPT_HEAVY_MIN 10 /* ratings in a block from which a user's ratings go to the cells;
                                  -1 (default): 16 x items / LDS sub-tile rows, at least 256,
                                  when the blocks average at least 2^24 ratings, else no cells */
#define PS_MF_OPT_TWO_STREAMS 11 /* 1 (default): run the L2 work units on a second and the LDS cells
                                    on a third internal stream (default priority) beside the
                                    dense tiles; 0: one stream */
#define PS_MF_OPT_HOT_STEPS 12 /* LDS sub-tiles of a block's most rated items whose ratings by the
                                  remaining (light) users also go to cells; 0: none;
                                  -1 (default): automatic (none when dense tiles are in
                                  use or the blocks average fewer than 2^24 ratings, else
                                  one sub-tile).  Needs
                                  PS_MF_OPT_CELLS = 1; at most 1024 */
#define PS_MF_OPT_DENSE_MIN 13 /* ratings from which a 64 x 64 tile (64 users of one worker class
                                  ranked by rating count x 64 items ranked by rating count) is
                                  swept with matrix-core products as a dense block; 0: none;
                                  -1 (default): automatic (800, i.e. 20% full, when the padded
                                  rank is in [16, 256] and the blocks average at least 2^24
                                  ratings, else none); at most 4096.  A value > 0
                                  with a padded rank outside [16, 256] makes
                                  ps_mf_load_ratings fail with PS_MF_EINVAL */
#define PS_MF_OPT_SEQ_STRATA 14 /* G: sub-epochs per clock of PS_MF_STEP_SEQ (default 256), in
                                   [1, 4096].  Part of the semantics: it fixes the order in which
                                   a worker applies its ratings */
#define PS_MF_OPT_ETA_DECAY 15  /* 1: step eta / sqrt(c + 1) at clock c (the schedule of Section 3's
                                   theorems); 0 (default): constant eta */
#define PS_MF_OPT_SEQ_GRAPHS 16 /* 1 (default): under PS_MF_STEP_SEQ, capture each clock's sub-epoch
                                   launches once per (block, view schedule) into a HIP graph on the
                                   handle's stream and replay it (not with PS_MF_OPT_ETA_DECAY);
                                   0: launch them one by one */
#define PS_MF_OPT_ITEM_TILE_BYTES 17 /* bytes of item rows per tile of the user-major sweep's work
                                        units (each tile is read from one XCD's L2); -1 (default):
                                        4 x PS_MF_OPT_TILE_BYTES; >= 1 otherwise */
#define PS_MF_OPT_DEVICE 18     /* HIP device ordinal the handle runs on; -1 (default): the device
                                   current at the handle's first device call.  A device that does
                                   not exist makes that call fail with PS_MF_EDEVICE */
#define PS_MF_OPT_POISON 19     /* debug, fixed-view steps only: 1 fills, before every commit, each
                                   row of the new version's ring slot that the commit does not
                                   read with NaN, so a row the commit failed to write shows as
                                   NaN (s = 0: the commit updates in place; nothing is filled);
                                   0 (default): off.  With PS_MF_STEP_SEQ load fails (EINVAL) */
#define PS_MF_OPT_SWEEP_GRAPHS 20 /* 1: under the fixed-view steps, capture each clock's sweep
                                     launches (work units, LDS cells, dense tiles and the fork
                                     and join of their streams) once per (block, view schedule)
                                     into a HIP graph on the handle's stream and replay it; a
                                     stream the caller is already capturing gets the launches
                                     one by one.  0 (default): launch them one by one (measured
                                     faster on ROCm 7: the replay's cross-stream edges cost more
                                     than the launches they replace) */
#define PS_MF_OPT_UNIT_COMMIT 21 /* 1 (default): under the fixed-view steps, a user whose ratings of
                                    the block all lie in one work unit has its new version written
                                    by that unit (the commit's formula, same arithmetic) when its
                                    view is not the new version's ring slot, and the commit skips
                                    it; 0 (and with PS_MF_OPT_SWEEP_GRAPHS): every user through
                                    the commit.  Same results */

/* Views (Section 3.2 SSP condition; Section 4 ESSPTable).  The table-level policies give
   worker p at clock c one whole version v = max(0, c - d):
     PS_MF_SSP_LAZY  d = (c + p mod (s+1)) mod (s+1) (a lazily refreshed cache, staggered);
     PS_MF_SSP_WORST d = s (exactly the guaranteed pre-window);
     PS_MF_ESSP      d = min(s, 1) (pushes land one clock later).
   The per-row policies keep a version per row in the cache of each client: worker p runs
   on client p mod min(P, s+1), a user row is read by its owner's client, an item row by
   every client with a rating of it in the clock's minibatch:
     PS_MF_SSP_ROW   a row that is not cached, or cached at a version < c - s, is fetched at
                     version c; otherwise the cached version is read (SSPTable);
     PS_MF_ESSP_ROW  the first read fetches version c, later reads see the server's push of
                     version c - min(s, 1) (ESSPTable).
   Under the per-row policies the version log stays empty; PS_MF_IDX_STALENESS and
   PS_MF_IDX_ROW_VERSIONS report the reads.
   The value-bounded policy (Section 2.1 and Section 3, the VAP condition: the in-transit
   updates of a worker's view are bounded in max-norm by v_t = v0 / sqrt(t)):
     PS_MF_VAP       every worker reads the stalest version v = c - d, d <= min(c, s), with
                     |x_c - x_v|_inf <= v0 / sqrt(c + 1); the norm is the maximum of the fp32
                     differences of the stored versions, compared in fp64.  v0 is set by
                     ps_mf_set_value_bound (default: unbounded, i.e. PS_MF_SSP_WORST);
                     s bounds how far back the ring reaches. */
#define PS_MF_SSP_LAZY 0
#define PS_MF_SSP_WORST 1
#define PS_MF_ESSP 2
#define PS_MF_SSP_ROW 3
#define PS_MF_ESSP_ROW 4
#define PS_MF_VAP 5

#define PS_MF_STEP_ROWMEAN 0
#define PS_MF_STEP_SUM 1
#define PS_MF_STEP_SEQ 2

/* index kinds (ps_mf_export_index) */
#define PS_MF_IDX_OWNER 0       /* int32 [users]: worker of each user */
#define PS_MF_IDX_ROW_PTR 1     /* int64 [users+1]: prefix sums of USER_COUNT(b), users in id order */
#define PS_MF_IDX_COL 2         /* int32 [nnz_b]: items of block b in (user, item, load index) order */
#define PS_MF_IDX_PERM 3        /* int64 [nnz_b]: load indices in the same order */
#define PS_MF_IDX_USER_COUNT 4  /* int32 [users]: ratings of each user in block b */
#define PS_MF_IDX_ITEM_COUNT 5  /* int32 [items]: ratings of each item in block b (all workers) */
#define PS_MF_IDX_VERSION_LOG 6 /* int64 [clocks*P]: v(p,c) at entry c*P + p (clock-major, Section 3.2) */
#define PS_MF_IDX_SPLIT 7       /* int64 [8]: how block b's ratings are swept: ratings in dense
                                   (matrix-core) tiles, in LDS-staged cells and in L2 work units,
                                   for the user-major then the item-major direction (each triple
                                   sums to the block's rating count); then the partial rows
                                   (Kp floats each) the user-major and the item-major sweep
                                   write per clock for the commit to sum.  Under
                                   PS_MF_STEP_SEQ: the chains, the user runs (a user's
                                   ratings inside one chain) and the ratings of block b,
                                   then zeros */
#define PS_MF_IDX_STALENESS 8   /* int64 [s+1]: staleness profile of the clocks run since the last
                                   ps_mf_set_factors (Section 2.2, Fig. 1 left): entry d counts
                                   the parameter reads that saw version c - d at clock c, i.e.
                                   whose clock differential (parameter age - local clock) is
                                   -(d+1); every rating a worker processes reads its user row
                                   and its item row at the worker's view.  BSP (s = 0) puts
                                   every read at d = 0 (differential -1) */
#define PS_MF_IDX_ROW_VERSIONS 9 /* int64 [users + C*items], C = min(P, s+1): under a per-row
                                   policy, the version each client's cache holds after the
                                   last clock: user rows (read by their owner's client), then
                                   client 0's item rows, client 1's, ...; -1 = never read.
                                   Other policies: length 0 */
#define PS_MF_IDX_SEQ_ORDER 10  /* int64 [nnz_b] under PS_MF_STEP_SEQ: load indices of block b in the
                                   order the workers apply them, (sub-epoch, worker, user group,
                                   user, item, load index); other steps: PS_MF_EINVAL */
#define PS_MF_IDX_VAP_NORMS 11  /* double [clocks * (s+1)] under PS_MF_VAP: entry c*(s+1) + d is the
                                   in-transit norm |x_c - x_{c-d}|_inf when clock c started
                                   (-1 where c - d < 0); other policies: PS_MF_EINVAL */

/* kernel ids (ps_mf_kernel_time) */
#define PS_MF_KERNEL_SWEEP 0  /* residual, dL segment-sum and dR accumulation of one clock */
#define PS_MF_KERNEL_COMMIT 1 /* clock commit: R (and untouched L rows) of the new version */

/*
 * Create a handle for an N x M problem of rank K with P workers and staleness s
 * (Section 3.1 problem statement; Section 3.2 staleness).  No device memory is touched.
 * Limits: 1 <= users, items <= 2^31-1; 1 <= K <= 512; 1 <= P <= 65536; 0 <= s <= 1024;
 * users * Kp * 4 and items * Kp * 4 below 2^32 bytes (Kp = K rounded up to a power of two,
 * at least 8); eta and lambda finite.  EINVAL otherwise; *out is NULL on failure.
 */
int ps_mf_create(int64_t users, int64_t items, int32_t K, int32_t P, int32_t s, float eta, float lambda,
                 ps_mf_t **out);

/* Set an option (keys above) before ps_mf_load_ratings; ESTATE after it, EINVAL for an
   unknown key or value. */
int ps_mf_set_option(ps_mf_t *h, int32_t key, int64_t value);

/* The value bound v0 of PS_MF_VAP (Section 3: v_t = v0 / sqrt(t), t = c + 1 at clock c);
   v0 >= 0, INFINITY allowed (the default).  Before load: ESTATE after it, EINVAL for a
   negative or NaN bound. */
int ps_mf_set_value_bound(ps_mf_t *h, double v0);

/* Optional explicit data partition (Section 3.1: ratings partitioned over workers):
   owner[users] with values in [0, P); default owner(i) = i mod P.  Before load. */
int ps_mf_set_owner_map(ps_mf_t *h, const int32_t *owner);

/* Launch everything on this HIP stream (a hipStream_t, e.g. torch's current stream);
   NULL selects the handle's own stream.  The caller keeps the stream alive. */
int ps_mf_set_stream(ps_mf_t *h, void *hip_stream);

/* Load the observed ratings D_obs as host COO arrays of length n (Section 3.1): user in
   [0, users), item in [0, items), finite value.  Builds the per-block layout (integer
   work, on the host) and uploads it.  Once per handle (ESTATE on a second call).
   Synchronizes. */
int ps_mf_load_ratings(ps_mf_t *h, const int32_t *user, const int32_t *item, const float *value, int64_t n);

/* Set version 0 from host arrays L (users x K) and R (items x K), row-major fp32,
   finite.  Resets the clock to 0 and the version log.  Synchronizes. */
int ps_mf_set_factors(ps_mf_t *h, const float *L, const float *R);

/* All P workers advance n >= 0 clocks in lockstep (Section 3.2): for each clock c the
   worker views are chosen, the sweep runs over block c mod B and version c+1 is
   committed.  Asynchronous on the handle's stream.  ESTATE before load and set_factors. */
int ps_mf_clock(ps_mf_t *h, int32_t n);

/* Squared loss (Section 5): sum over every loaded rating of (D_ij - L_i . R_j)^2 at the
   latest version, accumulated in fp64.  Synchronizes. */
int ps_mf_loss(ps_mf_t *h, double *out);

/* ps_mf_loss for callers that cannot allocate device memory (code under HIP graph capture,
   tight serving loops, harnesses that forbid hipMalloc): the same value, computed by the
   same kernels in the same order, with the fp64 partial sums in a fixed static array of
   2^18 + 1 doubles (2 MiB) that each GPU holds until the process ends, instead of the
   handle's buffer.  Calls no hipMalloc or hipFree.  EINVAL (before touching the device)
   when the loaded ratings need more than 2^18 partial sums (one per 256-thread workgroup of
   the loss: about (users + ratings / 512) * (lanes per row, 2 to 16) / 256); ESTATE as
   ps_mf_loss.
   Every call on one GPU shares that GPU's array: calls that overlap on one GPU (from
   several host threads) race.  Synchronizes. */
int ps_mf_loss_noalloc(ps_mf_t *h, double *out);

/* Copy the latest committed version into host arrays L (users x K), R (items x K).
   Synchronizes. */
int ps_mf_get_factors(ps_mf_t *h, float *L, float *R);

/* Copy committed version v (clock-s <= v <= clock: still in the ring).  Synchronizes. */
int ps_mf_get_version(ps_mf_t *h, int64_t v, float *L, float *R);

/* Number of clocks committed since set_factors. */
int ps_mf_get_clock(ps_mf_t *h, int64_t *clock);

/* Copy an integer index (kinds above) of block `block` into buf (capacity `cap`
   elements); *len receives the element count.  buf = NULL only queries *len.  EINVAL
   if cap is too small.  Works in host-only mode. */
int ps_mf_export_index(ps_mf_t *h, int32_t kind, int32_t block, void *buf, int64_t cap, int64_t *len);

/* With PS_MF_OPT_TIMING on: total milliseconds and launch count of a kernel id over all
   clocks run so far (HIP events on the handle's stream).  Synchronizes. */
int ps_mf_kernel_time(ps_mf_t *h, int32_t kernel, double *ms, int64_t *count);

/* Message of the last failed call on this handle (never NULL). */
const char *ps_mf_last_error(const ps_mf_t *h);

/* Free everything the handle owns; NULL-safe; valid after any failure. */
void ps_mf_destroy(ps_mf_t *h);

#ifdef __cplusplus
}
#endif

#endif /* PS_MF_H */
