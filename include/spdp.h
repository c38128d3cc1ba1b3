/*
 * spdp.h -- C ABI of the MI355X (gfx950) SPDP Gibbs-sweep library.
 *
 * The library runs the data-parallel hot path of the Shadow Poisson Dirichlet
 * Process (SPDP) differential topic model of Li (2012), "Multi-GPU Distributed
 * Parallel Bayesian Differential Topic Modelling" (arXiv:1510.06549): the
 * collapsed-Gibbs resampling of every token's (topic z, table indicator r)
 * against Pitman-Yor customer counts n[g,k,w] and table counts t[g,k,w] whose
 * tables share a per-topic shadow base (chapter "Shared Topic Modelling Using
 * Shadow Poisson Dirichlet Process", Eq. SPDP-sampling-w-z-r0 and
 * Eq. SPDP-sampling-w-z-r1, with identity transformation matrices P^i).
 * Documents are resampled in parallel against a snapshot of the shared counts
 * taken at the start of the sweep, the document-parallel approximation of the
 * thesis's Improved-GPU-SPDP (section "Parallelism With Improved Accuracy: Word
 * Order Rearrangement"), each document's own doc-topic row staying live and its
 * tokens running in order; the counts are then rebuilt exactly.
 *
 * Conventions shared by every entry point:
 *   - Return value: SPDP_OK (0) or a negative SPDP_E_* code; the text of the
 *     last error of the calling thread is returned by spdp_last_error().  No
 *     C++ exception crosses this boundary.
 *   - Ownership: host inputs are deep-copied before the call returns.  Outputs
 *     go to caller-allocated buffers of the documented size; `where` = 0 means
 *     a host pointer, 1 a device pointer on the state's GPU.  The state owns
 *     all its device memory until spdp_destroy().
 *   - Streams: all device work of a state runs in order on the HIP stream given
 *     at creation (NULL = the null stream).  spdp_sweep() only enqueues; calls
 *     that return data to the host synchronise that stream.
 *   - Threading: a state may be used by one host thread at a time.
 *   - Determinism: results are a pure function of (corpus, groups, K,
 *     hyperparameters, init seed, sequence of (sweep, seed)), independent of
 *     launch configuration and scheduling.
 *
 * Layouts: n and t are exported as [g][k][w] (group, then topic, then word:
 * the order of the thesis's n_{i,k,w}); the shadow-base table counts B as
 * [w][k] (topics contiguous); per-restaurant totals as [g][k].
 * The (z, r) state is per token in corpus order.
 */
#ifndef SPDP_H
#define SPDP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPDP_OK 0
#define SPDP_E_ARG (-1)   /* invalid argument (null pointer, value out of range) */
#define SPDP_E_NOMEM (-2) /* device or host allocation failed                   */
#define SPDP_E_HIP (-3)   /* a HIP runtime call failed                          */
#define SPDP_E_RANGE (-4) /* a size limit of the state would be exceeded          */
#define SPDP_E_STATE (-5) /* an invariant of the count state is violated         */

#define SPDP_MAX_K 1024
#define SPDP_MAX_SOURCES 8 /* longest source list of a word association row */

typedef struct spdp_state spdp_state; /* opaque */

/* A corpus: N tokens in D documents, stored document after document. */
typedef struct {
    int64_t n_tokens;           /* N, 0 <= N < 2^31                                */
    int32_t n_docs;             /* D >= 1                                          */
    int32_t vocab;              /* V >= 1                                          */
    const int32_t *words;       /* host [N], 0 <= words[i] < V                     */
    const int64_t *doc_offsets; /* host [D+1], [0] = 0, nondecreasing, [D] = N     */
    uint64_t init_seed;         /* key of the Philox stream that draws the initial z */
    void *hip_stream;           /* hipStream_t for all work of the state, or NULL   */
} spdp_corpus;

/* The groups ("collections" of the differential model, index i of the thesis). */
typedef struct {
    int32_t n_groups;           /* G >= 1, G * V < 2^31                             */
    const int32_t *doc_group;   /* host [D], 0 <= doc_group[d] < G                  */
} spdp_groups;

/*
 * Word associations: the transformation matrices P^g of the full SPDP model
 * (chapter "Shared Topic Modelling Using Shadow Poisson Dirichlet Process":
 * group g's topic k is a Pitman-Yor process around P^g phi0_k, so a new table
 * takes a source word v from the shadow base and serves word w with
 * probability p_{g,w,v}; Eq. SPDP-joint-prob-with-v).  P^g is given sparse, by
 * rows: row q = g V + w lists the sources v with p_{g,w,v} > 0 in entries
 * [row_off[q], row_off[q + 1]).  Column v of P^g is meant to be a
 * distribution over words (the sampler does not need it; the group estimate
 * then sums to one).
 */
typedef struct {
    int32_t max_sources;        /* S: the longest row, 1 <= S <= SPDP_MAX_SOURCES   */
    const int64_t *row_off;     /* host [G V + 1], [0] = 0, every row non-empty       */
    const int32_t *src;         /* host [nnz] source words, 0 <= v < V, distinct per row */
    const double *p;            /* host [nnz] p_{g,w,v}, finite and > 0               */
} spdp_assoc;

/*
 * Create a sampler state: validate, upload the corpus, tabulate the
 * generalised Stirling numbers S^n_{t,a} (recurrence of the PYP joint,
 * Corollary 17 passage) in fp64 log space for every n the corpus can reach,
 * draw the initial topics (z uniform from Philox, r = 0), rebuild the counts
 * and promote the smallest-index token of every non-empty cell to table head.
 *   K      number of topics, 1 <= K <= SPDP_MAX_K
 *   alpha  symmetric Dirichlet prior of document-topic proportions, > 0
 *   a      Pitman-Yor discount, 0 <= a < 1
 *   b      Pitman-Yor concentration, > 0
 *   gamma  symmetric Dirichlet prior of the shadow base phi0_k, > 0
 * Errors: E_ARG, E_NOMEM, E_HIP, E_RANGE (a (group, word) pair occurring more
 * than 65535 times: counts are held in 16 bits).  The Stirling cache takes
 * about 16 (ncap + 1)^2 bytes of device memory for ncap customers of the most
 * frequent pair: 17.2 GB at 32767, 68.7 GB at 65535.
 * On success *out holds the new state; on error *out is NULL.
 */
int spdp_create(const spdp_corpus *corpus, const spdp_groups *groups, int32_t K, double alpha,
                double a, double b, double gamma, spdp_state **out);

/*
 * The same for the model with word associations (`assoc`, copied at the
 * call).  Each table head then carries a source word, stored as its slot s in
 * its row's list (0 <= s < the row's length), and the shadow-base counts are
 * keyed by source: B[v][k] counts the heads of topic k whose source is v.
 * Initialisation and repair give a new head its row's most probable source
 * (the first on ties).  Every entry point below works on such a state, with
 * the differences stated there.  Errors: as spdp_create, and E_ARG for a bad
 * association list (an empty or over-long row, a source out of range or
 * repeated in its row, p not finite and > 0, max_sources not the longest
 * row).
 */
int spdp_create_assoc(const spdp_corpus *corpus, const spdp_groups *groups,
                      const spdp_assoc *assoc, int32_t K, double alpha, double a, double b,
                      double gamma, spdp_state **out);

/*
 * One Gibbs sweep (asynchronous on the state's stream): every token's (z, r)
 * is resampled from the 2K outcomes of Eq. SPDP-sampling-w-z-r0/-r1, with the
 * shared counts of the sweep start and the live row of its own document;
 * outcome j = 2k is (k, r = 1), j = 2k + 1 is (k, r = 0); the uniform of token
 * i is Philox4x32-10 keyed by `seed` at counter (i lo, i hi, sweep, 0), and the
 * draw is the first j whose prefix sum exceeds u * total.  A token that is the
 * only head of a cell with other customers keeps its state.  Counts are then
 * updated exactly and every cell left with customers but no table gets its
 * smallest-index token as head.  Errors: E_ARG, E_HIP.
 * With word associations a token has K (S + 1) outcomes, per topic k the head
 * outcomes (k, r = 1, slot s) for s = 0 .. S - 1, then (k, r = 0):
 *   j = k (S + 1) + s is (k, 1, s),  j = k (S + 1) + S is (k, 0),
 * with W(k, 1, s) = p_{g,w,v_s} times the plain r = 1 weight evaluated on the
 * shadow-base count of source v_s (Eq. SPDP-sampling-w-z-r1 with p_{i,w,v});
 * slots past a row's length weigh 0.  The only head of a cell with other
 * customers keeps its topic and r but redraws its source, in proportion to
 * p_{g,w,v} (gamma + B'[v][k]).
 */
int spdp_sweep(spdp_state *s, uint32_t sweep, uint64_t seed);

/*
 * Ablation (not the library's sweep): one sweep of the thesis's asynchronous
 * scheme (section "Parallel Word Sampling": each token reads the global
 * counts as they are, removes itself and adds itself back with atomics, no
 * locks; subsection "Word Order Rearrangement": tokens taken up round robin
 * over the position inside the document, documents in index order at each
 * position).  `waves` wavefronts take the tokens of the visiting order in
 * turn (wave w: positions w, w + waves, ...); 0 takes the library's default
 * (16 per compute unit).  The word, shadow-base and document counts are live;
 * the sums N_gk, T_gk, B_k are live too if live_totals != 0, else held at
 * their sweep-start values during the pass (the thesis lets them drift and
 * corrects them regularly; live sums serialise on their few counters).  With
 * waves = 1 and live_totals = 1 the sweep is exactly sequential collapsed
 * Gibbs in the visiting order (same outcomes, uniforms and sole-head rule as
 * spdp_sweep, counts live after every token); with more waves it is racy and
 * its result depends on scheduling.  The counts are then regenerated exactly
 * from the new state, with the repair of spdp_sweep.  The first call builds
 * the visiting order and allocates 8 N + 4 D Kp bytes of device memory.
 * Asynchronous on the state's stream.  Errors: E_ARG (NULL state, waves < 0,
 * a state with word associations), E_NOMEM, E_HIP.
 */
int spdp_sweep_async(spdp_state *s, uint32_t sweep, uint64_t seed, int32_t waves,
                     int32_t live_totals);

/*
 * Export customer counts n and table counts t of groups [g_begin, g_end) as
 * [g_end - g_begin][K][V] int32 each: element ((g - g_begin) K + k) V + w is
 * n[g][k][w] (either pointer may be NULL to skip it).  Synchronises.
 * Errors: E_ARG, E_HIP.
 */
int spdp_counts(const spdp_state *s, int32_t g_begin, int32_t g_end, int32_t *n_gkw,
                int32_t *t_gkw, int where);

/*
 * Export the totals: customers N[g][k] = sum_w n, tables T[g][k] = sum_w t,
 * shadow-base table counts B[w][k] = sum_g t and B[k] = sum_w B[w][k] (with
 * word associations B[v][k] counts the heads of topic k whose source is v).
 * Any pointer may be NULL.  Synchronises.  Errors: E_ARG, E_HIP.
 */
int spdp_totals(const spdp_state *s, int32_t *N_gk, int32_t *T_gk, int32_t *B_wk, int32_t *B_k,
                int where);

/*
 * Joint log p(W, Z, R | alpha, a, b, gamma) of the current state in fp64 (the
 * collapsed joint of the thesis's blocked-Gibbs derivation with P = I):
 * document Dirichlet-multinomial terms, per-restaurant (b|a)_T / (b)_N,
 * per-cell S^n_{t,a} / C(n, t), and the shadow-base Dirichlet-multinomial of
 * each topic; with word associations the base counts are keyed by source and
 * the sum over table heads of log p_{g,w,v} of the head's source is added.
 * Deterministic reduction order.  Synchronises.
 * Errors: E_ARG, E_HIP, E_STATE (a cell with t > n or t = 0 < n).
 */
int spdp_loglik(spdp_state *s, double *out);

/* Free all resources of the state (NULL is ignored). */
void spdp_destroy(spdp_state *s);

/*
 * Point estimates of the current state (the thesis's estimates after
 * convergence: Eq. spdp-topic-doc-estimate, Eq. spdp-word-topic-estimate and
 * Eq. spdp-group-word-topic-estimate, with P = I), in fp64:
 *   theta [D][K]   theta[d][k] = (c_dk + alpha) / (L_d + K alpha)
 *   phi0  [V][K]   phi0[w][k]  = (gamma + B_wk) / (V gamma + B_k)
 *   phi   [g_end - g_begin][V][K]
 *                  phi[g][w][k] = (n - a t + (b + a T_gk) phi0[w][k]) / (b + N_gk)
 * (the base weight b + a T is the Pitman-Yor seating rule's; the printed
 * a T does not normalise).  With word associations phi0 is over source words
 * and the group's base is P^g phi0: phi0[w][k] above is replaced by
 * sum_v p_{g,w,v} phi0[v][k].  Any pointer may be NULL; the group range applies
 * to phi only.  `where` as for spdp_counts.  Synchronises.
 * Errors: E_ARG (bad range), E_HIP.
 */
int spdp_estimates(spdp_state *s, int32_t g_begin, int32_t g_end, double *theta, double *phi0,
                   double *phi, int where);

/*
 * Held-out perplexity (section "Perplexity") of test documents given as their
 * own corpus (same vocabulary; `init_seed` and `hip_stream` are not used) and
 * groups (same n_groups).  Each test document is folded in with phi fixed at
 * the group estimate of the current state: topics drawn uniformly (first
 * Philox word keyed by `seed` with purpose 3 at counter (test token, 0), times
 * K, high 32 bits), then n_sweeps Gibbs sweeps over its tokens in order with
 * p(z_n = k | rest) proportional to (c_k without token n + alpha) phi[g][w_n][k]
 * (uniform: purpose 2 at counter (test token, sweep); first k whose prefix
 * exceeds u * total); then log p(w_d) = sum_n log sum_k phi[g][w_n][k]
 * theta_d[k] with theta_d from the final counts, in fp64.
 * out2[0] = perplexity exp(-sum_d log p(w_d) / N_test) (NaN if N_test = 0),
 * out2[1] = sum_d log p(w_d) (host pointer).  z_out [N_test] int32 receives
 * the final fold-in topics (may be NULL; `where` applies to it).  The state
 * is not changed.  Synchronises.
 * Errors: E_ARG (sizes, vocabulary or groups differ, ids out of range), E_HIP.
 */
int spdp_heldout(spdp_state *s, const spdp_corpus *test, const spdp_groups *test_groups,
                 int32_t n_sweeps, uint64_t seed, double *out2, int32_t *z_out, int where);

/*
 * Hellinger distances between the topics of two models (chapter
 * "Experiments", subsection "Hellinger Distance"):
 *   h[i][j] = sqrt(max(0, 1 - sum_v sqrt(p[v][i]) sqrt(q[v][j]))),
 * which is (1/sqrt 2) || sqrt(p_i) - sqrt(q_j) ||_2 for distributions.
 * p [n_outcomes][kp] and q [n_outcomes][kq] hold one distribution per column
 * (topics contiguous, the layout spdp_estimates writes phi0 and phi in);
 * entries must be >= 0 (a negative entry gives NaN).  p = NULL takes the
 * state's shadow-base estimate phi0 (then kp = K, n_outcomes = V).  h
 * [kp][kq] fp64.  `where` applies to p, q and h alike.  The contraction runs
 * on the fp64 matrix cores; it allocates slices * kp * kq doubles of device
 * scratch (at most 2048 slices, fewer as kp * kq grows) plus device copies of
 * host inputs.  Uses the state's device and stream only; the state is not
 * changed.  Synchronises.
 * Errors: E_ARG (NULL q or h, negative size, kp or kq above SPDP_MAX_K, p NULL
 * with kp != K or n_outcomes != V), E_HIP.
 */
int spdp_hellinger(spdp_state *s, const double *p, int32_t kp, const double *q, int32_t kq,
                   int32_t n_outcomes, double *h, int where);

/*
 * For callers that cannot allocate device memory (code under stream capture,
 * tight serving loops, harnesses that forbid hipMalloc): spdp_hellinger on
 * device buffers that allocates nothing.  p [n_outcomes][kp], q
 * [n_outcomes][kq] and h [kp][kq] are fp64 device pointers on the state's
 * GPU (p may not be NULL: the state's phi0 would need a buffer), each inside
 * one device allocation that holds its size (checked against the
 * allocation, not against a caller's sub-range of it); the result equals
 * spdp_hellinger's.
 * The partial sums over outcome slices go to a static device array of
 * 2^20 doubles (8 MiB) that each GPU the library runs on holds until the
 * process ends, so kp * kq may not exceed 2^20 (always true for topic counts
 * up to SPDP_MAX_K).  Only enqueues on the state's stream (no
 * synchronisation): calls on one GPU share the array, so calls that overlap
 * (other streams or host threads) race; calls in one stream's order do not.
 * Errors: E_ARG (NULL pointer, negative size, topic count above SPDP_MAX_K,
 * a buffer that is not device memory or too short), E_RANGE (kp * kq above
 * 2^20), E_HIP.
 */
int spdp_hellinger_noalloc(spdp_state *s, const double *p, int32_t kp, const double *q,
                           int32_t kq, int32_t n_outcomes, double *h);

/*
 * Topic alignment for comparing two models (the topics are reordered to line up in the
 * Hellinger comparison): the one-to-one matching of the kp rows of h
 * [kp][kq] (kp <= kq; e.g. distances from spdp_hellinger) to columns that
 * minimises the summed entries.  match [kp] int32 receives the column of each
 * row, *total the minimum sum.  Host arrays only; runs on the host
 * (Hungarian method with potentials, O(kp^2 kq)); needs no state and no GPU.
 * Errors: E_ARG (NULL pointer, kp < 0 or kp > kq, an entry not finite).
 */
int spdp_align_topics(const double *h, int32_t kp, int32_t kq, int32_t *match, double *total);

/*
 * Checkpoint: export z [N] int32 and r [N] uint8 (either may be NULL).
 * Synchronises.  Errors: E_ARG, E_HIP.
 */
int spdp_get_assignments(const spdp_state *s, int32_t *z, uint8_t *r, int where);

/*
 * Resume: replace the state by (z, r) (z in [0, K), r in {0, 1}), rebuild the
 * counts and promote the smallest-index token of every cell with customers but
 * no table.  Synchronises.  Errors: E_ARG (value out of range), E_HIP.
 */
int spdp_set_assignments(spdp_state *s, const int32_t *z, const uint8_t *r, int where);

/*
 * Word associations: export the source slot of every token's table ([N]
 * uint8, 0 for r = 0), or resume from (z, r, slot) (as spdp_set_assignments;
 * a head's slot must index a source of its row, r = 0 tokens store slot 0).
 * spdp_set_assignments on such a state gives every head slot 0.  *S receives
 * the longest source list (0 for a state without associations).
 * Synchronise.  Errors: E_ARG (null pointer, a state without associations for
 * the resume, a value out of range), E_HIP.
 */
int spdp_get_slots(const spdp_state *s, uint8_t *slot, int where);
int spdp_set_assignments_assoc(spdp_state *s, const int32_t *z, const uint8_t *r,
                               const uint8_t *slot, int where);
int spdp_max_sources(const spdp_state *s, int32_t *S);

/*
 * Test hook: run the sampling step of sweep (sweep, seed) on the current state
 * WITHOUT committing it, and export, for tokens i in [tok_begin, tok_end), the
 * fp32 unnormalised weights of all 2K outcomes (w_out, [(tok_end - tok_begin)
 * * 2K], outcome order as in spdp_sweep), the uniform (u_out, -1 for a token
 * kept by the sole-head rule) and the sampled packed outcome (zr_out, value
 * 2 z + r, may be NULL).  With word associations w_out holds K (S + 1)
 * weights per token, every token draws (no -1), and zr_out holds
 * s << 16 | 2 z + r.  With w_out and u_out both NULL no trace is kept and
 * any token range may be requested (the sampled state before the count update
 * and repair).  Uses the same kernel as spdp_sweep.  Synchronises.
 * Errors: E_ARG, E_NOMEM, E_HIP.
 */
int spdp_debug_conditionals(spdp_state *s, uint32_t sweep, uint64_t seed, int64_t tok_begin,
                            int64_t tok_end, float *w_out, float *u_out, int32_t *zr_out,
                            int where);

/*
 * Statistics of the last sweep: tokens whose (z, r) changed and table heads
 * promoted by the repair step.  Synchronises.  Errors: E_ARG, E_HIP.
 */
int spdp_stats(const spdp_state *s, int64_t *changed, int64_t *repaired);

/*
 * Per-kernel timing with HIP events on the state's stream.  enable = 1 starts
 * recording (and clears the accumulators), 0 stops.  spdp_kernel_times writes
 * the accumulated milliseconds and launch counts of the SPDP_NKERNELS kernel
 * classes, in this order: sampling; count rebuild with repair (which also
 * sums the shadow-base counts); the 16-bit copy of the shadow base;
 * per-restaurant totals and per-sweep constants.  Synchronises.
 */
#define SPDP_NKERNELS 4
int spdp_kernel_timing(spdp_state *s, int enable);
int spdp_kernel_times(spdp_state *s, double *ms, int64_t *launches);

/*
 * Invariant check of the count state: the stored counts are recounted from
 * the tokens' (z, r) (and sources, with word associations) and compared, and
 * every cell must satisfy 0 <= t <= n with t > 0 exactly when n > 0 (a cell
 * with customers but no table has joint probability zero).  Checked: every
 * count row (and the 16-bit copy of a narrow row), the totals N_gk, T_gk,
 * B_k, the shadow-base counts B and their 16-bit copy and width flag, and
 * every token's topic and source slot.  The read-only counterpart of the
 * count regeneration the thesis runs on the host after a parallel iteration
 * (Algorithm MGPU-DP-SPDP Host).  *bad (may be NULL) receives the number of
 * failing cells, tokens and totals.  Allocates and frees device scratch of
 * (2 G + 1) Kp ints (+ V Kp with word associations).  Synchronises.
 * Errors: E_ARG, E_NOMEM, E_HIP, E_STATE (some check failed; the message
 * gives the counts).
 */
int spdp_check(spdp_state *s, int64_t *bad);

/*
 * Test hook: add dn customers and dt tables to the stored count cell of
 * (group g, word w, topic k) -- in the copy the samplers read (the 16-bit
 * copy of a narrow row, else the 32-bit row), nothing else -- so that tests
 * can make the state inconsistent and see spdp_check report it (any later
 * rebuild, e.g. spdp_set_assignments, restores consistent counts).
 * Synchronises.  Errors: E_ARG (cell out of range, or a count would leave
 * [0, 255] in a narrow row or [0, 65535] in a wide one), E_HIP.
 */
int spdp_debug_poke(spdp_state *s, int32_t g, int32_t w, int32_t k, int32_t dn, int32_t dt);

/*
 * Shape of the state: out[0] = N, [1] = D, [2] = V, [3] = G, [4] = K,
 * [5] = row stride of the count arrays (topics, >= K), [6] = largest
 * per-(group, word) token count (the Stirling rows needed), [7] = device bytes
 * held.  Errors: E_ARG.
 */
int spdp_info(const spdp_state *s, int64_t *out8);

/*
 * Read-bandwidth probe of the device: the ceiling against which the sampler's
 * bytes per second are read (a measurement aid, not part of the sampling
 * path).  Reads the device buffer buf (bytes long, 16-byte aligned, inside one
 * device allocation; the caller owns it) and returns in *ms the elapsed
 * milliseconds of the launch, from HIP events on stream (a hipStream_t, or
 * NULL for the null stream).
 *   row_bytes = 0     the whole buffer once, front to back, by waves
 *                     wavefronts' worth of threads (rows is ignored);
 *   row_bytes = 1024, 2048, 3072, 4096 or 8192
 *                     waves wavefronts read rows rows in all, one whole row at a
 *                     time per wavefront at pseudo-random row positions among
 *                     bytes / row_bytes, two rows in flight per wavefront (as
 *                     the sampler reads a token's count row).
 * The bytes read are bytes (row_bytes = 0) or ceil(rows / waves) * waves *
 * row_bytes.  Synchronises.  Errors: E_ARG (NULL buf or ms, misaligned buf,
 * other row_bytes, bytes below one row, waves outside [1, 2^20], rows < 1 with
 * rows read, buf not device memory or bytes past its allocation), E_HIP.
 */
int spdp_read_probe(const void *buf, int64_t bytes, int32_t row_bytes, int64_t rows,
                    int32_t waves, void *stream, double *ms);

/* Text of the calling thread's last error ("" if none). */
const char *spdp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SPDP_H */
