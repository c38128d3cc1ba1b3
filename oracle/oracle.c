/*
 * oracle.c -- plain fp64 CPU oracle of the SPDP snapshot-parallel Gibbs sweep.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or calls
 * this file: only the test suite, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header, table or constant generator
 * with the HIP library; its own Philox and Stirling table are written here from
 * their published definitions.
 *
 * Model: Li (2012), "Multi-GPU Distributed Parallel Bayesian Differential Topic
 * Modelling" (arXiv:1510.06549), chapter "Shared Topic Modelling Using Shadow
 * Poisson Dirichlet Process", with every transformation matrix P^i = I (the
 * setting of the thesis's experiments, section "MGPU-DP-SPDP" / identity P).
 * Then the word-association variables v collapse, q = t, and p_{i,w,v} = 1.
 *
 * Notation (thesis -> here):
 *   m_{ikw}  customers of word w at restaurant (group i, topic k)  -> n[g][k][w]
 *   t_{ikw}  tables ("multiplicity") of word w at (i,k)            -> t[g][k][w]
 *   n_{idk}  tokens of document d with topic k                     -> ndk / c[k]
 *   m_{ik.}, t_{ik.}                                               -> Ngk, Tgk
 *   sum_i t_{ikw} (shadow-base table counts), sum over w           -> Bkw, Bk
 *   alpha_{ik} (doc prior), a_k (discount), b_k (concentration),
 *   gamma_v (base prior)                                           -> alpha, a, b, gam
 *
 * Readings of passages the thesis leaves open (each one is listed in the
 * design notes of the repository):
 *   - shared counts come from a snapshot taken at sweep start; the document's
 *     own doc-topic row is live and its tokens run in index order;
 *   - r is stored per token; removal uses the stored r;
 *   - removing the only head of a cell that still has other customers has
 *     joint probability zero for every alternative, so the token keeps its
 *     state (point mass) and no uniform is consumed;
 *   - after the sweep, counts are rebuilt from (z, r) and every cell with
 *     n > 0 and t = 0 gets its smallest-index token promoted to head;
 *   - outcome j = 2k is (k, r=1), j = 2k+1 is (k, r=0) (even/odd work-item
 *     convention of the thesis's ParallelSampleWord kernel); the draw takes
 *     the first j whose inclusive prefix sum exceeds u * total;
 *   - uniforms come from Philox4x32-10 keyed by the seed, counter =
 *     (token lo, token hi, sweep, purpose); u = (x0 >> 8) * 2^-24.
 *
 * Build:  gcc -O2 -fopenmp -fPIC -shared oracle.c -lm -o liboracle.so
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_PURPOSE_SAMPLE 0u
#define OR_PURPOSE_INIT 1u
/* (purposes 2 and 3 are the held-out fold-in, defined with it below) */

/* ------------------------------------------------------------------------ */
/* Model description.  All arrays are owned by the caller.                   */
/* ------------------------------------------------------------------------ */
typedef struct {
    int64_t n_tokens;
    int32_t n_docs, vocab, n_groups, K;
    const int32_t *words;     /* [N]   word id per token                     */
    const int64_t *doc_off;   /* [D+1] CSR offsets of documents               */
    const int32_t *doc_group; /* [D]   group of each document                 */
    double alpha, a, b, gam;  /* doc prior, PYP discount, PYP conc., base prior */
    int32_t ncap;             /* the Stirling table covers 0 <= t <= n <= ncap */
    const double *logS;       /* triangle, row n at n(n+1)/2                   */
} or_model;

/* Counts, logical layout of the thesis: n_{i,k,w} -> n[(g*K + k)*V + w]. */
typedef struct {
    int32_t *n, *t;     /* [G][K][V] */
    int32_t *Ngk, *Tgk; /* [G][K]    */
    int32_t *Bkw;       /* [K][V]    */
    int32_t *Bk;        /* [K]       */
} or_counts;

static inline int64_t tri(int64_t n, int64_t t) { return n * (n + 1) / 2 + t; }

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as   */
/* easy as 1, 2, 3", SC'11): 10 rounds of the 4x32 Philox S-box with the     */
/* Weyl key schedule.                                                        */
/* ------------------------------------------------------------------------ */
void or_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) { k0 += W0; k1 += W1; }
        uint64_t p0 = (uint64_t)M0 * c0;
        uint64_t p1 = (uint64_t)M1 * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* First output word for (seed; token i, sweep, purpose). */
uint32_t or_philox_word0(uint64_t seed, int64_t i, uint32_t sweep, uint32_t purpose)
{
    uint32_t ctr[4] = {(uint32_t)(uint64_t)i, (uint32_t)((uint64_t)i >> 32), sweep, purpose};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t out[4];
    or_philox4x32_10(ctr, key, out);
    return out[0];
}

/* 24-bit uniform in [0,1): exact in both fp32 and fp64. */
double or_uniform(uint64_t seed, int64_t i, uint32_t sweep)
{
    uint32_t x = or_philox_word0(seed, i, sweep, OR_PURPOSE_SAMPLE);
    return (double)(x >> 8) * (1.0 / 16777216.0);
}

/* ------------------------------------------------------------------------ */
/* Generalised Stirling numbers S^n_{t,a} (thesis, section on the SPDP joint, */
/* the Corollary 17 passage): S^{n+1}_{t} = S^n_{t-1} + (n - t a) S^n_t,      */
/* S^n_t = 0 for t > n, S^n_0 = delta_{n,0}.  Tabulated as log S in fp64,     */
/* -inf where S = 0.  Output: triangle of (nmax+1)(nmax+2)/2 doubles.        */
/* ------------------------------------------------------------------------ */
static double log_add(double x, double y)
{
    if (x == -INFINITY) return y;
    if (y == -INFINITY) return x;
    double m = x > y ? x : y;
    return m + log1p(exp(-fabs(x - y)));
}

int or_stirling_log_table(int32_t nmax, double a, double *logS)
{
    if (nmax < 0 || !(a >= 0.0 && a < 1.0) || !logS) return -1;
    logS[0] = 0.0; /* S^0_0 = 1 */
    for (int64_t n = 0; n < nmax; ++n) {
        const double *row = logS + tri(n, 0);
        double *next = logS + tri(n + 1, 0);
        next[0] = -INFINITY; /* S^{n+1}_0 = 0 */
        for (int64_t t = 1; t <= n + 1; ++t) {
            double from_left = row[t - 1];                        /* S^n_{t-1} */
            double from_same = (t <= n) ? row[t] : -INFINITY;     /* S^n_t     */
            double term = (from_same == -INFINITY) ? -INFINITY
                                                   : log((double)n - (double)t * a) + from_same;
            next[t] = log_add(from_left, term);
        }
    }
    return 0;
}

static inline double log_stirling(const or_model *m, int64_t n, int64_t t)
{
    if (t < 0 || t > n) return -INFINITY;
    return m->logS[tri(n, t)];
}

/* ------------------------------------------------------------------------ */
/* Initialisation: z_i uniform over topics by integer multiply-shift of the  */
/* first Philox word with purpose INIT; r_i = 0 (repair then makes one head  */
/* per non-empty cell).                                                      */
/* ------------------------------------------------------------------------ */
void or_init(const or_model *m, uint64_t init_seed, int32_t *z, uint8_t *r)
{
    for (int64_t i = 0; i < m->n_tokens; ++i) {
        uint32_t x = or_philox_word0(init_seed, i, 0u, OR_PURPOSE_INIT);
        z[i] = (int32_t)(((uint64_t)x * (uint64_t)m->K) >> 32);
        r[i] = 0;
    }
}

/* ------------------------------------------------------------------------ */
/* Counts as pure functions of (z, r): the definitions of the count           */
/* statistics used by the collapsed joint (thesis, SPDP joint derivation).    */
/* ------------------------------------------------------------------------ */
void or_rebuild(const or_model *m, const int32_t *z, const uint8_t *r, or_counts *c)
{
    const int64_t G = m->n_groups, K = m->K, V = m->vocab;
    memset(c->n, 0, sizeof(int32_t) * (size_t)(G * K * V));
    memset(c->t, 0, sizeof(int32_t) * (size_t)(G * K * V));
    memset(c->Ngk, 0, sizeof(int32_t) * (size_t)(G * K));
    memset(c->Tgk, 0, sizeof(int32_t) * (size_t)(G * K));
    memset(c->Bkw, 0, sizeof(int32_t) * (size_t)(K * V));
    memset(c->Bk, 0, sizeof(int32_t) * (size_t)K);
    for (int32_t d = 0; d < m->n_docs; ++d) {
        const int64_t g = m->doc_group[d];
        for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) {
            const int64_t k = z[i], w = m->words[i];
            c->n[(g * K + k) * V + w] += 1;
            c->Ngk[g * K + k] += 1;
            if (r[i]) {
                c->t[(g * K + k) * V + w] += 1;
                c->Tgk[g * K + k] += 1;
                c->Bkw[k * V + w] += 1;
                c->Bk[k] += 1;
            }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Repair: scan tokens in increasing index; a token with r = 0 in a cell      */
/* that has no table becomes that cell's head.  Returns the number promoted. */
/* ------------------------------------------------------------------------ */
int64_t or_repair(const or_model *m, const int32_t *z, uint8_t *r, or_counts *c)
{
    const int64_t K = m->K, V = m->vocab;
    int64_t promoted = 0;
    for (int32_t d = 0; d < m->n_docs; ++d) {
        const int64_t g = m->doc_group[d];
        for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) {
            const int64_t k = z[i], w = m->words[i];
            if (r[i] == 0 && c->t[(g * K + k) * V + w] == 0) {
                r[i] = 1;
                c->t[(g * K + k) * V + w] += 1;
                c->Tgk[g * K + k] += 1;
                c->Bkw[k * V + w] += 1;
                c->Bk[k] += 1;
                ++promoted;
            }
        }
    }
    return promoted;
}

/* ------------------------------------------------------------------------ */
/* The 2K unnormalised conditionals of one token (thesis Eq.                  */
/* SPDP-sampling-w-z-r0 and Eq. SPDP-sampling-w-z-r1, P = I), evaluated on    */
/* the counts `s` with the token's own contribution removed at its current    */
/* cell, and on the document row `crow` (which still includes the token).    */
/*                                                                           */
/* Returns 1 (and leaves w untouched) when the token is the only head of a    */
/* cell that still has other customers: every other outcome then has zero    */
/* joint probability, so the conditional is a point mass on the current      */
/* state.  Otherwise fills w[2k] = weight of (k, r=1), w[2k+1] = (k, r=0).   */
/* ------------------------------------------------------------------------ */
int or_token_weights(const or_model *m, const or_counts *s, const int32_t *crow, int32_t g,
                     int32_t wd, int32_t k0, int32_t r0, double *w)
{
    const int64_t K = m->K, V = m->vocab;
    const int64_t cell0 = ((int64_t)g * K + k0) * V + wd;
    if (r0 == 1 && s->t[cell0] == 1 && s->n[cell0] > 1) return 1;
    const double alpha = m->alpha, a = m->a, b = m->b, gam = m->gam;
    for (int64_t k = 0; k < K; ++k) {
        const int del = (k == k0);
        const int64_t cell = ((int64_t)g * K + k) * V + wd;
        const int64_t nw = s->n[cell] - del;            /* m_{ikw} without token */
        const int64_t tw = s->t[cell] - del * r0;       /* t_{ikw} without token */
        const int64_t Nk = s->Ngk[g * K + k] - del;     /* m_{ik.}               */
        const int64_t Tk = s->Tgk[g * K + k] - del * r0;/* t_{ik.}               */
        const int64_t Bw = s->Bkw[k * V + wd] - del * r0;  /* sum_i t_{ikw}        */
        const int64_t Bt = s->Bk[k] - del * r0;            /* sum_i sum_w t_{ikw}  */
        const double ck = (double)(crow[k] - del);      /* n_{idk} without token */
        double q0, q1;
        if (nw == 0) {
            /* empty cell: S^1_0 / S^0_0 = 0 and S^1_1 / S^0_0 = 1 */
            q0 = 0.0;
            q1 = 1.0;
        } else {
            const double ls = log_stirling(m, nw, tw);
            /* (m - t + 1)/(m + 1) * S^{m+1}_t / S^m_t */
            q0 = (double)(nw - tw + 1) / (double)(nw + 1) * exp(log_stirling(m, nw + 1, tw) - ls);
            /* (t + 1)/(m + 1) * S^{m+1}_{t+1} / S^m_t */
            q1 = (double)(tw + 1) / (double)(nw + 1) * exp(log_stirling(m, nw + 1, tw + 1) - ls);
        }
        const double doc = alpha + ck;
        w[2 * k + 1] = doc / (b + (double)Nk) * q0;
        w[2 * k] = doc * (b + a * (double)Tk) / (b + (double)Nk) * (gam + (double)Bw) /
                   ((double)m->vocab * gam + (double)Bt) * q1;
    }
    return 0;
}

/* First outcome whose inclusive prefix sum exceeds u * total. */
static int draw_outcome(const double *w, int64_t nout, double u)
{
    double total = 0.0;
    for (int64_t j = 0; j < nout; ++j) total += w[j];
    const double target = u * total;
    double acc = 0.0;
    for (int64_t j = 0; j < nout; ++j) {
        acc += w[j];
        if (acc > target) return (int)j;
    }
    return -1; /* unreachable: u < 1 and total > 0 */
}

/* ------------------------------------------------------------------------ */
/* Sampling step of one sweep over documents [d_begin, d_end), against the   */
/* snapshot `s` (read only).  z, r are updated in place; each document only  */
/* touches its own tokens, so documents may run in any order or in parallel. */
/* Optional trace: for tokens i in [tr_begin, tr_end) the weights (2K each),  */
/* the uniform and a skip flag are written.                                   */
/* Returns the number of tokens whose (z, r) changed.                        */
/* ------------------------------------------------------------------------ */
int64_t or_sample_docs(const or_model *m, const or_counts *s, int32_t *z, uint8_t *r,
                       uint32_t sweep, uint64_t seed, int32_t d_begin, int32_t d_end,
                       double *tr_w, double *tr_u, uint8_t *tr_skip, int64_t tr_begin,
                       int64_t tr_end)
{
    const int64_t K = m->K;
    int64_t changed = 0;
#pragma omp parallel reduction(+ : changed)
    {
        int32_t *crow = (int32_t *)malloc(sizeof(int32_t) * (size_t)K);
        double *w = (double *)malloc(sizeof(double) * (size_t)(2 * K));
#pragma omp for schedule(dynamic, 16)
        for (int32_t d = d_begin; d < d_end; ++d) {
            const int32_t g = m->doc_group[d];
            memset(crow, 0, sizeof(int32_t) * (size_t)K);
            for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) crow[z[i]] += 1;
            for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) {
                const int32_t k0 = z[i], r0 = r[i];
                const int skip = or_token_weights(m, s, crow, g, m->words[i], k0, r0, w);
                const int tr = (tr_w != NULL && i >= tr_begin && i < tr_end);
                if (tr) tr_skip[i - tr_begin] = (uint8_t)skip;
                if (skip) continue;
                const double u = or_uniform(seed, i, sweep);
                if (tr) {
                    memcpy(tr_w + (i - tr_begin) * 2 * K, w, sizeof(double) * (size_t)(2 * K));
                    tr_u[i - tr_begin] = u;
                }
                const int j = draw_outcome(w, 2 * K, u);
                const int32_t k1 = j / 2, r1 = 1 - (j % 2);
                crow[k0] -= 1;
                crow[k1] += 1;
                if (k1 != k0 || r1 != r0) ++changed;
                z[i] = k1;
                r[i] = (uint8_t)r1;
            }
        }
        free(crow);
        free(w);
    }
    return changed;
}

/* ------------------------------------------------------------------------ */
/* One full sweep.  mode 0: snapshot-parallel (sampling step against the      */
/* sweep-start counts, then exact rebuild and repair).  mode 1: sequential    */
/* collapsed Gibbs (Algorithm SPDP-Full-Gibbs with stored r): live counts,    */
/* updated after every token; the state stays valid so repair never fires.   */
/* out_stats[0] = tokens changed, out_stats[1] = heads promoted by repair.    */
/* ------------------------------------------------------------------------ */
static void apply_token(const or_model *m, or_counts *c, int32_t g, int32_t wd, int32_t k,
                        int32_t rr, int sgn)
{
    const int64_t K = m->K, V = m->vocab;
    const int64_t cell = ((int64_t)g * K + k) * V + wd;
    c->n[cell] += sgn;
    c->Ngk[(int64_t)g * K + k] += sgn;
    if (rr) {
        c->t[cell] += sgn;
        c->Tgk[(int64_t)g * K + k] += sgn;
        c->Bkw[(int64_t)k * V + wd] += sgn;
        c->Bk[k] += sgn;
    }
}

int or_sweep(const or_model *m, or_counts *c, int32_t *z, uint8_t *r, uint32_t sweep,
             uint64_t seed, int mode, int64_t *out_stats)
{
    int64_t changed = 0, promoted = 0;
    if (mode == 0) {
        changed = or_sample_docs(m, c, z, r, sweep, seed, 0, m->n_docs, NULL, NULL, NULL, 0, 0);
        or_rebuild(m, z, r, c);
        promoted = or_repair(m, z, r, c);
    } else if (mode == 1) {
        const int64_t K = m->K;
        int32_t *crow = (int32_t *)malloc(sizeof(int32_t) * (size_t)K);
        double *w = (double *)malloc(sizeof(double) * (size_t)(2 * K));
        for (int32_t d = 0; d < m->n_docs; ++d) {
            const int32_t g = m->doc_group[d];
            memset(crow, 0, sizeof(int32_t) * (size_t)K);
            for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) crow[z[i]] += 1;
            for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) {
                const int32_t k0 = z[i], r0 = r[i], wd = m->words[i];
                if (or_token_weights(m, c, crow, g, wd, k0, r0, w)) continue;
                const int j = draw_outcome(w, 2 * K, or_uniform(seed, i, sweep));
                const int32_t k1 = j / 2, r1 = 1 - (j % 2);
                apply_token(m, c, g, wd, k0, r0, -1);
                apply_token(m, c, g, wd, k1, r1, +1);
                crow[k0] -= 1;
                crow[k1] += 1;
                if (k1 != k0 || r1 != r0) ++changed;
                z[i] = k1;
                r[i] = (uint8_t)r1;
            }
        }
        free(crow);
        free(w);
    } else {
        return -1;
    }
    if (out_stats) { out_stats[0] = changed; out_stats[1] = promoted; }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Joint log p(W, Z, R | alpha, a, b, gamma) with P = I: the collapsed joint  */
/* of the thesis's blocked-Gibbs derivation (Eq. SPDP-Blocked-Gibbs-Joint-    */
/* Prob and the final product), read as                                      */
/*   doc terms      prod_d Beta_K(alpha + n_d) / Beta_K(alpha)                */
/*   PYP normaliser prod_{g,k} (b|a)_{T_gk} / (b)_{N_gk}                      */
/*   cells          prod_{g,k,w} S^{n}_{t,a} / C(n, t)                        */
/*   shadow base    prod_k Beta_V(gamma + B_k.) / Beta_V(gamma)               */
/* Returns -inf for a state with zero probability (some t > n, or t = 0 < n). */
/* ------------------------------------------------------------------------ */
static double log_pochhammer_step(double x, double y, int64_t T)
{
    /* log (x|y)_T = sum_{j<T} log(x + j y) */
    if (T <= 0) return 0.0;
    if (y == 0.0) return (double)T * log(x);
    return (double)T * log(y) + lgamma(x / y + (double)T) - lgamma(x / y);
}

double or_loglik(const or_model *m, const int32_t *z, const uint8_t *r, const or_counts *c)
{
    (void)r;
    const int64_t G = m->n_groups, K = m->K, V = m->vocab;
    const double alpha = m->alpha, a = m->a, b = m->b, gam = m->gam;
    double ll_doc = 0.0, ll_pyp = 0.0, ll_cell = 0.0, ll_base = 0.0;
    int bad = 0;

    /* documents */
    int32_t *crow = (int32_t *)calloc((size_t)K, sizeof(int32_t));
    for (int32_t d = 0; d < m->n_docs; ++d) {
        memset(crow, 0, sizeof(int32_t) * (size_t)K);
        const int64_t L = m->doc_off[d + 1] - m->doc_off[d];
        for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) crow[z[i]] += 1;
        double s = lgamma((double)K * alpha) - lgamma((double)K * alpha + (double)L);
        for (int64_t k = 0; k < K; ++k) s += lgamma(alpha + crow[k]) - lgamma(alpha);
        ll_doc += s;
    }
    free(crow);

    /* restaurants (g, k) */
    for (int64_t g = 0; g < G; ++g)
        for (int64_t k = 0; k < K; ++k) {
            const int64_t N = c->Ngk[g * K + k], T = c->Tgk[g * K + k];
            ll_pyp += log_pochhammer_step(b, a, T) - log_pochhammer_step(b, 1.0, N);
        }

    /* cells */
    for (int64_t g = 0; g < G; ++g)
        for (int64_t k = 0; k < K; ++k)
            for (int64_t w = 0; w < V; ++w) {
                const int64_t n = c->n[(g * K + k) * V + w], t = c->t[(g * K + k) * V + w];
                if (n == 0 && t == 0) continue;
                if (n > m->ncap) return NAN; /* Stirling table too small */
                if (t > n || t <= 0) { bad = 1; continue; }
                ll_cell += log_stirling(m, n, t) -
                           (lgamma((double)n + 1.0) - lgamma((double)t + 1.0) -
                            lgamma((double)(n - t) + 1.0));
            }

    /* shadow base */
    for (int64_t k = 0; k < K; ++k) {
        double s = lgamma((double)V * gam) - lgamma((double)V * gam + (double)c->Bk[k]);
        for (int64_t w = 0; w < V; ++w) s += lgamma(gam + (double)c->Bkw[k * V + w]) - lgamma(gam);
        ll_base += s;
    }
    if (bad) return -INFINITY;
    return ll_doc + ll_pyp + ll_cell + ll_base;
}

/* Largest per-(group, word) token count: every n[g][k][w] is bounded by it, */
/* so it fixes how many Stirling rows any state of this corpus can need.     */
int32_t or_max_group_word_count(const or_model *m)
{
    const int64_t G = m->n_groups, V = m->vocab;
    int32_t *cnt = (int32_t *)calloc((size_t)(G * V), sizeof(int32_t));
    int32_t best = 0;
    for (int32_t d = 0; d < m->n_docs; ++d) {
        const int64_t g = m->doc_group[d];
        for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) {
            int32_t v = ++cnt[g * V + m->words[i]];
            if (v > best) best = v;
        }
    }
    free(cnt);
    return best;
}

int or_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the OpenMP loops that follow (n >= 1); returns the new count. */
int or_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
    return omp_get_max_threads();
#else
    (void)n;
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Word order rearrangement (thesis, subsection "Parallelism With Improved    */
/* Accuracy: Word Order Rearrangement"): tokens are visited round robin over  */
/* their position inside the document -- every document's first token, then  */
/* every document's second token, and so on -- so that tokens taken up at     */
/* about the same time come from different documents.  Documents are taken   */
/* in index order at every position.  order [N] receives token indices.      */
/* ------------------------------------------------------------------------ */
void or_interleaved_order(const or_model *m, int32_t *order)
{
    int64_t longest = 0, out = 0;
    for (int32_t d = 0; d < m->n_docs; ++d)
        if (m->doc_off[d + 1] - m->doc_off[d] > longest) longest = m->doc_off[d + 1] - m->doc_off[d];
    for (int64_t pos = 0; pos < longest; ++pos)
        for (int32_t d = 0; d < m->n_docs; ++d)
            if (m->doc_off[d] + pos < m->doc_off[d + 1]) order[out++] = (int32_t)(m->doc_off[d] + pos);
}

/* ------------------------------------------------------------------------ */
/* Sequential collapsed Gibbs (Algorithm SPDP-Full-Gibbs with stored r, live */
/* counts) visiting the tokens in a given order (a permutation of 0..N-1):   */
/* the exact single-site sampler whose racy concurrent execution the        */
/* thesis's asynchronous GPU kernel is.  Each document's topic counts stay   */
/* live across the sweep.  The uniform of token i is that of or_sweep.       */
/* stale_totals = 1: the auxiliary sums N_gk, T_gk and B_k enter the         */
/* conditionals at their sweep-start values (the token's own contribution    */
/* removed), while n, t, B_kw and the document counts stay live -- the       */
/* thesis lets the sums drift during an iteration and corrects them          */
/* regularly; this variant is not exact Gibbs.  It is pinned by a re-walk   */
/* that keeps the live and the held counts itself (tests).                  */
/* ------------------------------------------------------------------------ */
int or_sweep_ordered(const or_model *m, or_counts *c, int32_t *z, uint8_t *r, uint32_t sweep,
                     uint64_t seed, const int32_t *order, int stale_totals, int64_t *out_stats)
{
    const int64_t K = m->K, N = m->n_tokens, G = m->n_groups;
    /* the counts the conditionals read: live, or live with frozen sums */
    or_counts view = *c;
    int32_t *frozen = NULL;
    if (stale_totals) {
        frozen = (int32_t *)malloc(sizeof(int32_t) * (size_t)(2 * G * K + K));
        memcpy(frozen, c->Ngk, sizeof(int32_t) * (size_t)(G * K));
        memcpy(frozen + G * K, c->Tgk, sizeof(int32_t) * (size_t)(G * K));
        memcpy(frozen + 2 * G * K, c->Bk, sizeof(int32_t) * (size_t)K);
        view.Ngk = frozen;
        view.Tgk = frozen + G * K;
        view.Bk = frozen + 2 * G * K;
    }
    int32_t *cdk = (int32_t *)calloc((size_t)(m->n_docs > 0 ? m->n_docs : 1) * (size_t)K,
                                     sizeof(int32_t));
    int32_t *tok_doc = (int32_t *)malloc(sizeof(int32_t) * (size_t)(N > 0 ? N : 1));
    double *w = (double *)malloc(sizeof(double) * (size_t)(2 * K));
    for (int32_t d = 0; d < m->n_docs; ++d)
        for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) {
            tok_doc[i] = d;
            cdk[(int64_t)d * K + z[i]] += 1;
        }
    int64_t changed = 0;
    int bad = 0;
    for (int64_t p = 0; p < N; ++p) {
        const int64_t i = order[p];
        if (i < 0 || i >= N) { bad = 1; break; }
        const int32_t d = tok_doc[i], g = m->doc_group[d];
        int32_t *crow = cdk + (int64_t)d * K;
        const int32_t k0 = z[i], r0 = r[i], wd = m->words[i];
        if (or_token_weights(m, &view, crow, g, wd, k0, r0, w)) continue;
        const int j = draw_outcome(w, 2 * K, or_uniform(seed, i, sweep));
        const int32_t k1 = j / 2, r1 = 1 - (j % 2);
        apply_token(m, c, g, wd, k0, r0, -1);
        apply_token(m, c, g, wd, k1, r1, +1);
        crow[k0] -= 1;
        crow[k1] += 1;
        if (k1 != k0 || r1 != r0) ++changed;
        z[i] = k1;
        r[i] = (uint8_t)r1;
    }
    free(cdk);
    free(tok_doc);
    free(w);
    free(frozen);
    if (bad) return -1;
    if (out_stats) { out_stats[0] = changed; out_stats[1] = 0; }
    return 0;
}

/* Chain histogram of the ordered sequential sweep (encoding as below). */
int or_chain_histogram_ordered(const or_model *m, or_counts *c, int32_t *z, uint8_t *r,
                               uint32_t first_sweep, int64_t n_sweeps, uint64_t seed,
                               const int32_t *order, int64_t *hist, int64_t n_bins)
{
    const int64_t base = 2 * (int64_t)m->K;
    for (int64_t s = 0; s < n_sweeps; ++s) {
        if (or_sweep_ordered(m, c, z, r, first_sweep + (uint32_t)s, seed, order, 0, NULL) != 0)
            return -1;
        int64_t code = 0, mul = 1;
        for (int64_t i = 0; i < m->n_tokens; ++i) {
            code += (2 * (int64_t)z[i] + 1 - r[i]) * mul;
            mul *= base;
        }
        if (code < 0 || code >= n_bins) return -2;
        hist[code] += 1;
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Test helper: run `n_sweeps` sweeps (mode as in or_sweep, sweep index =    */
/* first_sweep + s) and histogram the visited states.  A state is encoded in  */
/* base 2K with digit (2 z_i + 1 - r_i) for token i (least significant first), */
/* so the histogram needs (2K)^N bins; only for tiny corpora.                 */
/* ------------------------------------------------------------------------ */
int or_chain_histogram(const or_model *m, or_counts *c, int32_t *z, uint8_t *r,
                       uint32_t first_sweep, int64_t n_sweeps, uint64_t seed, int mode,
                       int64_t *hist, int64_t n_bins)
{
    const int64_t base = 2 * (int64_t)m->K;
    for (int64_t s = 0; s < n_sweeps; ++s) {
        if (or_sweep(m, c, z, r, first_sweep + (uint32_t)s, seed, mode, NULL) != 0) return -1;
        int64_t code = 0, mul = 1;
        for (int64_t i = 0; i < m->n_tokens; ++i) {
            code += (2 * (int64_t)z[i] + 1 - r[i]) * mul;
            mul *= base;
        }
        if (code < 0 || code >= n_bins) return -2;
        hist[code] += 1;
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Point estimates of a state (thesis: estimates after convergence,         */
/* Eq. spdp-topic-doc-estimate, Eq. spdp-word-topic-estimate and            */
/* Eq. spdp-group-word-topic-estimate, with P = I so that q = t):            */
/*   theta[d][k] = (c_dk + alpha) / (L_d + K alpha)                          */
/*   phi0[k][w]  = (gamma + B_kw) / (V gamma + B_k)                          */
/*   phig[g][k][w] = (n - a t + (b + a T_gk) phi0[k][w]) / (b + N_gk)        */
/* The printed group estimate weights the base by a T / (b + N), which sums */
/* over words to N / (b + N); the Pitman-Yor posterior predictive (a new    */
/* customer joins a table serving w with weight n_w - a t_w, or opens a new */
/* table with weight b + a T and takes its dish from the base) weights it   */
/* by (b + a T) / (b + N), which sums to one: that is the reading here.     */
/* Any output pointer may be NULL.                                           */
/* ------------------------------------------------------------------------ */
void or_estimates(const or_model *m, const int32_t *z, const or_counts *c, double *theta,
                  double *phi0, double *phig)
{
    const int64_t G = m->n_groups, K = m->K, V = m->vocab;
    if (theta) {
        for (int32_t d = 0; d < m->n_docs; ++d) {
            double *row = theta + (int64_t)d * K;
            for (int64_t k = 0; k < K; ++k) row[k] = 0.0;
            for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) row[z[i]] += 1.0;
            const double len = (double)(m->doc_off[d + 1] - m->doc_off[d]);
            for (int64_t k = 0; k < K; ++k)
                row[k] = (row[k] + m->alpha) / (len + (double)K * m->alpha);
        }
    }
    double *p0 = phi0 ? phi0 : (phig ? (double *)malloc(sizeof(double) * (size_t)(K * V)) : NULL);
    if (p0) {
        for (int64_t k = 0; k < K; ++k)
            for (int64_t w = 0; w < V; ++w)
                p0[k * V + w] = (m->gam + (double)c->Bkw[k * V + w]) /
                                ((double)V * m->gam + (double)c->Bk[k]);
    }
    if (phig) {
        for (int64_t g = 0; g < G; ++g)
            for (int64_t k = 0; k < K; ++k) {
                const double N = (double)c->Ngk[g * K + k], T = (double)c->Tgk[g * K + k];
                for (int64_t w = 0; w < V; ++w) {
                    const int64_t cell = (g * K + k) * V + w;
                    phig[cell] = ((double)c->n[cell] - m->a * (double)c->t[cell] +
                                  (m->b + m->a * T) * p0[k * V + w]) /
                                 (m->b + N);
                }
            }
    }
    if (p0 && !phi0) free(p0);
}

/* ------------------------------------------------------------------------ */
/* Held-out documents (thesis, section "Perplexity": documents held out per  */
/* group; p(w_d | rest) = prod_n sum_k phi^i_{k,w_n} theta_{d,k}).  The      */
/* thesis leaves open how a held-out document's theta is obtained; reading: */
/* fold-in (query sampling) with phi fixed at the point estimate phig of    */
/* the training state:                                                      */
/*   1. z_n drawn uniformly: first Philox word with purpose FOLDIN_INIT (3), */
/*      counter (test token n, 0), times K, high 32 bits;                    */
/*   2. n_sweeps Gibbs sweeps, each over the document's tokens in order:     */
/*      p(z_n = k | rest) proportional to (c_k without n + alpha) phig[g][k][w_n], */
/*      u from Philox purpose FOLDIN (2) at counter (n, sweep), first k     */
/*      whose inclusive prefix sum exceeds u * total;                        */
/*   3. theta_k = (c_k + alpha) / (L + K alpha) from the final counts, and   */
/*      log p(w_d) = sum_n log sum_k phig[g][k][w_n] theta_k.                */
/* Documents are independent (any order, in parallel).  The test corpus has */
/* its own token numbering.  z_out [N_test] receives the final topics;       */
/* ll_doc [D_test] the per-document log p (either may be NULL).  Returns the */
/* sum of log p over documents, added in document order.                     */
/* ------------------------------------------------------------------------ */
#define OR_PURPOSE_FOLDIN 2u
#define OR_PURPOSE_FOLDIN_INIT 3u

double or_heldout(const or_model *m, const double *phig, int32_t d_test, const int32_t *words,
                  const int64_t *doc_off, const int32_t *doc_group, int32_t n_sweeps,
                  uint64_t seed, int32_t *z_out, double *ll_doc)
{
    const int64_t K = m->K, V = m->vocab;
    double *lld = ll_doc ? ll_doc : (double *)malloc(sizeof(double) * (size_t)(d_test > 0 ? d_test : 1));
    int32_t *zz = z_out ? z_out : (int32_t *)malloc(sizeof(int32_t) * (size_t)(doc_off[d_test] > 0 ? doc_off[d_test] : 1));
#pragma omp parallel
    {
        int64_t *c = (int64_t *)malloc(sizeof(int64_t) * (size_t)K);
        double *w = (double *)malloc(sizeof(double) * (size_t)K);
#pragma omp for schedule(dynamic, 16)
        for (int32_t d = 0; d < d_test; ++d) {
            const int64_t g = doc_group[d], beg = doc_off[d], end = doc_off[d + 1];
            const double *ph = phig + g * K * V;
            for (int64_t k = 0; k < K; ++k) c[k] = 0;
            for (int64_t i = beg; i < end; ++i) {
                const uint32_t x = or_philox_word0(seed, i, 0u, OR_PURPOSE_FOLDIN_INIT);
                zz[i] = (int32_t)(((uint64_t)x * (uint64_t)K) >> 32);
                c[zz[i]] += 1;
            }
            for (int32_t s = 0; s < n_sweeps; ++s) {
                for (int64_t i = beg; i < end; ++i) {
                    c[zz[i]] -= 1;
                    for (int64_t k = 0; k < K; ++k)
                        w[k] = ((double)c[k] + m->alpha) * ph[k * V + words[i]];
                    const uint32_t x = or_philox_word0(seed, i, (uint32_t)s, OR_PURPOSE_FOLDIN);
                    const double u = (double)(x >> 8) * (1.0 / 16777216.0);
                    const int k1 = draw_outcome(w, K, u);
                    zz[i] = k1;
                    c[k1] += 1;
                }
            }
            const double len = (double)(end - beg);
            double ll = 0.0;
            for (int64_t i = beg; i < end; ++i) {
                double p = 0.0;
                for (int64_t k = 0; k < K; ++k)
                    p += ph[k * V + words[i]] * ((double)c[k] + m->alpha) / (len + (double)K * m->alpha);
                ll += log(p);
            }
            lld[d] = ll;
        }
        free(c);
        free(w);
    }
    double total = 0.0;
    for (int32_t d = 0; d < d_test; ++d) total += lld[d];
    if (!ll_doc) free(lld);
    if (!z_out) free(zz);
    return total;
}

/* ======================================================================== */
/* Word associations: non-identity transformation matrices P^i.            */
/*                                                                          */
/* The full model of the SPDP chapter: group i's topic k is a Pitman-Yor     */
/* process around P^i phi0_k, so a new table first takes a source word v     */
/* from the shadow base and then serves word w with probability p_{i,w,v}    */
/* (column v of P^i is a distribution over w).  Each table head carries its  */
/* source (the thesis's v_{ikwt}); q_{ikwv} counts the tables of (i, k, w)   */
/* with source v, and the shadow base counts tables by SOURCE:               */
/*   Bkw[k][v] = sum_i sum_w q_{ikwv},   Bk[k] = sum_v Bkw[k][v] = sum T_gk.  */
/* Eq. SPDP-joint-prob-with-v and the blocked-Gibbs joint add the factor     */
/* prod over heads of p_{i,w,v(head)}; Eq. SPDP-sampling-w-z-r1 gains        */
/* p_{i,w,v} and (gamma_v + sum q_{.k.v}) in place of (gamma + B_kw).        */
/*                                                                          */
/* P^i is sparse: row (g, w) lists its sources v with p_{g,w,v} > 0          */
/* (at most S of them).  A head's source is stored as its index s within     */
/* its row's list.  Readings (listed in the design notes):                   */
/*   - outcomes of one token, per topic k, in the order (k, r=1, s) for       */
/*     s = 0..S-1, then (k, r=0): j = k (S + 1) + s and j = k (S + 1) + S;    */
/*     list slots s >= S_w of a shorter row have weight 0.  With S = 1 and    */
/*     v = w this is the identity order j = 2k + 1 - r;                       */
/*   - a token with r = 0 stores s = 0;                                       */
/*   - repair promotes the smallest-index token of a cell with customers but  */
/*     no table and gives it the row's most probable source (the first one    */
/*     on ties);                                                              */
/*   - initialisation as with P = I (z from Philox, r = 0, s = 0), then       */
/*     rebuild and repair.                                                    */
/* ======================================================================== */
typedef struct {
    int32_t S;              /* longest source list                          */
    const int64_t *row_off; /* [G V + 1] CSR offsets of the rows (g, w)       */
    const int32_t *src;     /* [nnz] source word v of each entry             */
    const double *p;        /* [nnz] p_{g,w,v}                               */
} or_assoc;

static inline int64_t arow(const or_model *m, int64_t g, int64_t w) { return g * m->vocab + w; }

/* index of the row's most probable source (first on ties) */
int32_t or_head_source(const or_model *m, const or_assoc *A, int32_t g, int32_t w)
{
    const int64_t q = arow(m, g, w), beg = A->row_off[q], end = A->row_off[q + 1];
    int32_t best = 0;
    for (int64_t e = beg + 1; e < end; ++e)
        if (A->p[e] > A->p[beg + best]) best = (int32_t)(e - beg);
    return best;
}

static inline int32_t source_of(const or_model *m, const or_assoc *A, int64_t g, int64_t w,
                                int32_t s)
{
    return A->src[A->row_off[arow(m, g, w)] + s];
}

void or_rebuild_assoc(const or_model *m, const or_assoc *A, const int32_t *z, const uint8_t *r,
                      const uint8_t *s, or_counts *c)
{
    const int64_t G = m->n_groups, K = m->K, V = m->vocab;
    memset(c->n, 0, sizeof(int32_t) * (size_t)(G * K * V));
    memset(c->t, 0, sizeof(int32_t) * (size_t)(G * K * V));
    memset(c->Ngk, 0, sizeof(int32_t) * (size_t)(G * K));
    memset(c->Tgk, 0, sizeof(int32_t) * (size_t)(G * K));
    memset(c->Bkw, 0, sizeof(int32_t) * (size_t)(K * V));
    memset(c->Bk, 0, sizeof(int32_t) * (size_t)K);
    for (int32_t d = 0; d < m->n_docs; ++d) {
        const int64_t g = m->doc_group[d];
        for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) {
            const int64_t k = z[i], w = m->words[i];
            c->n[(g * K + k) * V + w] += 1;
            c->Ngk[g * K + k] += 1;
            if (r[i]) {
                c->t[(g * K + k) * V + w] += 1;
                c->Tgk[g * K + k] += 1;
                c->Bkw[k * V + source_of(m, A, g, w, s[i])] += 1;
                c->Bk[k] += 1;
            }
        }
    }
}

int64_t or_repair_assoc(const or_model *m, const or_assoc *A, const int32_t *z, uint8_t *r,
                        uint8_t *s, or_counts *c)
{
    const int64_t K = m->K, V = m->vocab;
    int64_t promoted = 0;
    for (int32_t d = 0; d < m->n_docs; ++d) {
        const int64_t g = m->doc_group[d];
        for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) {
            const int64_t k = z[i], w = m->words[i];
            if (r[i] == 0 && c->t[(g * K + k) * V + w] == 0) {
                const int32_t hs = or_head_source(m, A, (int32_t)g, (int32_t)w);
                r[i] = 1;
                s[i] = (uint8_t)hs;
                c->t[(g * K + k) * V + w] += 1;
                c->Tgk[g * K + k] += 1;
                c->Bkw[k * V + source_of(m, A, g, w, hs)] += 1;
                c->Bk[k] += 1;
                ++promoted;
            }
        }
    }
    return promoted;
}

/* The K (S + 1) unnormalised conditionals of one token (Eq. SPDP-sampling-  */
/* w-z-r0 and Eq. SPDP-sampling-w-z-r1 with p_{i,w,v}), on the counts `c`    */
/* with the token's own contribution removed (its customer, and if it is a   */
/* head its table and its source's base count), and the document row `crow` */
/* (which still includes the token): w[k (S+1) + s] = (k, r=1, source slot   */
/* s) and w[k (S+1) + S] = (k, r=0).                                          */
/* The only head of a cell that keeps other customers must stay that cell's  */
/* head (every other topic or r has joint probability zero), but its source  */
/* is free: then only its own topic's head slots are non-zero, in proportion */
/* to the joint, p_{g,w,v} (gamma + Bkw[k0][v] without the token's source).  */
/* Always returns 0 (no point mass: some slot is always positive).          */
int or_token_weights_assoc(const or_model *m, const or_assoc *A, const or_counts *c,
                           const int32_t *crow, int32_t g, int32_t wd, int32_t k0, int32_t r0,
                           int32_t s0, double *w)
{
    const int64_t K = m->K, V = m->vocab, S = A->S;
    const int64_t cell0 = ((int64_t)g * K + k0) * V + wd;
    const int64_t q = arow(m, g, wd), beg = A->row_off[q], nsrc = A->row_off[q + 1] - beg;
    const int32_t v0 = A->src[beg + s0];
    if (r0 == 1 && c->t[cell0] == 1 && c->n[cell0] > 1) {
        for (int64_t j = 0; j < K * (S + 1); ++j) w[j] = 0.0;
        for (int64_t sl = 0; sl < nsrc; ++sl) {
            const int32_t v = A->src[beg + sl];
            w[k0 * (S + 1) + sl] =
                A->p[beg + sl] * (m->gam + (double)(c->Bkw[(int64_t)k0 * V + v] - (v == v0)));
        }
        return 0;
    }
    const double alpha = m->alpha, a = m->a, b = m->b, gam = m->gam;
    for (int64_t k = 0; k < K; ++k) {
        const int del = (k == k0);
        const int64_t cell = ((int64_t)g * K + k) * V + wd;
        const int64_t nw = c->n[cell] - del;
        const int64_t tw = c->t[cell] - del * r0;
        const int64_t Nk = c->Ngk[g * K + k] - del;
        const int64_t Tk = c->Tgk[g * K + k] - del * r0;
        const int64_t Bt = c->Bk[k] - del * r0;
        const double ck = (double)(crow[k] - del);
        double q0, q1;
        if (nw == 0) {
            q0 = 0.0;
            q1 = 1.0;
        } else {
            const double ls = log_stirling(m, nw, tw);
            q0 = (double)(nw - tw + 1) / (double)(nw + 1) * exp(log_stirling(m, nw + 1, tw) - ls);
            q1 = (double)(tw + 1) / (double)(nw + 1) * exp(log_stirling(m, nw + 1, tw + 1) - ls);
        }
        const double doc = alpha + ck;
        double *wk = w + k * (S + 1);
        for (int64_t sl = 0; sl < S; ++sl) {
            if (sl >= nsrc) { wk[sl] = 0.0; continue; }
            const int32_t v = A->src[beg + sl];
            const int64_t Bv = c->Bkw[k * V + v] - ((del && r0 && v == v0) ? 1 : 0);
            wk[sl] = A->p[beg + sl] * doc * (b + a * (double)Tk) / (b + (double)Nk) *
                     (gam + (double)Bv) / ((double)V * gam + (double)Bt) * q1;
        }
        wk[S] = doc / (b + (double)Nk) * q0;
    }
    return 0;
}

/* Sampling step of one sweep over documents [d_begin, d_end) against the    */
/* snapshot `c` (read only); as or_sample_docs, with the source slot s.       */
/* Trace: K (S + 1) weights per token.                                        */
int64_t or_sample_docs_assoc(const or_model *m, const or_assoc *A, const or_counts *c,
                             int32_t *z, uint8_t *r, uint8_t *s, uint32_t sweep, uint64_t seed,
                             int32_t d_begin, int32_t d_end, double *tr_w, double *tr_u,
                             uint8_t *tr_skip, int64_t tr_begin, int64_t tr_end)
{
    const int64_t K = m->K, S1 = A->S + 1, nout = K * S1;
    int64_t changed = 0;
#pragma omp parallel reduction(+ : changed)
    {
        int32_t *crow = (int32_t *)malloc(sizeof(int32_t) * (size_t)K);
        double *w = (double *)malloc(sizeof(double) * (size_t)nout);
#pragma omp for schedule(dynamic, 16)
        for (int32_t d = d_begin; d < d_end; ++d) {
            const int32_t g = m->doc_group[d];
            memset(crow, 0, sizeof(int32_t) * (size_t)K);
            for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) crow[z[i]] += 1;
            for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) {
                const int32_t k0 = z[i], r0 = r[i], s0 = s[i];
                const int skip =
                    or_token_weights_assoc(m, A, c, crow, g, m->words[i], k0, r0, s0, w);
                const int tr = (tr_w != NULL && i >= tr_begin && i < tr_end);
                if (tr) tr_skip[i - tr_begin] = (uint8_t)skip;
                if (skip) continue;
                const double u = or_uniform(seed, i, sweep);
                if (tr) {
                    memcpy(tr_w + (i - tr_begin) * nout, w, sizeof(double) * (size_t)nout);
                    tr_u[i - tr_begin] = u;
                }
                const int j = draw_outcome(w, nout, u);
                const int32_t k1 = (int32_t)(j / S1), sl = (int32_t)(j % S1);
                const int32_t r1 = sl < A->S ? 1 : 0, s1 = r1 ? sl : 0;
                crow[k0] -= 1;
                crow[k1] += 1;
                if (k1 != k0 || r1 != r0 || s1 != s0) ++changed;
                z[i] = k1;
                r[i] = (uint8_t)r1;
                s[i] = (uint8_t)s1;
            }
        }
        free(crow);
        free(w);
    }
    return changed;
}

static void apply_token_assoc(const or_model *m, const or_assoc *A, or_counts *c, int32_t g,
                              int32_t wd, int32_t k, int32_t rr, int32_t sl, int sgn)
{
    const int64_t K = m->K, V = m->vocab;
    const int64_t cell = ((int64_t)g * K + k) * V + wd;
    c->n[cell] += sgn;
    c->Ngk[(int64_t)g * K + k] += sgn;
    if (rr) {
        c->t[cell] += sgn;
        c->Tgk[(int64_t)g * K + k] += sgn;
        c->Bkw[(int64_t)k * V + source_of(m, A, g, wd, sl)] += sgn;
        c->Bk[k] += sgn;
    }
}

/* One sweep: mode 0 snapshot-parallel (sampling, then rebuild and repair),  */
/* mode 1 sequential collapsed Gibbs (Algorithm SPDP-Full-Gibbs with stored  */
/* r and source: live counts after every token).                             */
int or_sweep_assoc(const or_model *m, const or_assoc *A, or_counts *c, int32_t *z, uint8_t *r,
                   uint8_t *s, uint32_t sweep, uint64_t seed, int mode, int64_t *out_stats)
{
    int64_t changed = 0, promoted = 0;
    const int64_t K = m->K, S1 = A->S + 1, nout = K * S1;
    if (mode == 0) {
        changed = or_sample_docs_assoc(m, A, c, z, r, s, sweep, seed, 0, m->n_docs, NULL, NULL,
                                       NULL, 0, 0);
        or_rebuild_assoc(m, A, z, r, s, c);
        promoted = or_repair_assoc(m, A, z, r, s, c);
    } else if (mode == 1) {
        int32_t *crow = (int32_t *)malloc(sizeof(int32_t) * (size_t)K);
        double *w = (double *)malloc(sizeof(double) * (size_t)nout);
        for (int32_t d = 0; d < m->n_docs; ++d) {
            const int32_t g = m->doc_group[d];
            memset(crow, 0, sizeof(int32_t) * (size_t)K);
            for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) crow[z[i]] += 1;
            for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) {
                const int32_t k0 = z[i], r0 = r[i], s0 = s[i], wd = m->words[i];
                if (or_token_weights_assoc(m, A, c, crow, g, wd, k0, r0, s0, w)) continue;
                const int j = draw_outcome(w, nout, or_uniform(seed, i, sweep));
                const int32_t k1 = (int32_t)(j / S1), sl = (int32_t)(j % S1);
                const int32_t r1 = sl < A->S ? 1 : 0, s1 = r1 ? sl : 0;
                apply_token_assoc(m, A, c, g, wd, k0, r0, s0, -1);
                apply_token_assoc(m, A, c, g, wd, k1, r1, s1, +1);
                crow[k0] -= 1;
                crow[k1] += 1;
                if (k1 != k0 || r1 != r0 || s1 != s0) ++changed;
                z[i] = k1;
                r[i] = (uint8_t)r1;
                s[i] = (uint8_t)s1;
            }
        }
        free(crow);
        free(w);
    } else {
        return -1;
    }
    if (out_stats) { out_stats[0] = changed; out_stats[1] = promoted; }
    return 0;
}

/* Joint log p(W, Z, V, R): the P = I joint evaluated on counts whose shadow */
/* base is keyed by source (or_rebuild_assoc), times the association factor  */
/* prod_{g,w,v} p_{g,w,v}^{sum_k q_{gkwv}} = prod over heads of p of the     */
/* head's source.                                                            */
double or_loglik_assoc(const or_model *m, const or_assoc *A, const int32_t *z, const uint8_t *r,
                       const uint8_t *s, const or_counts *c)
{
    double ll = or_loglik(m, z, r, c);
    double lp = 0.0;
    for (int32_t d = 0; d < m->n_docs; ++d) {
        const int64_t g = m->doc_group[d];
        for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i)
            if (r[i]) lp += log(A->p[A->row_off[arow(m, g, m->words[i])] + s[i]]);
    }
    return ll + lp;
}

/* Estimates with associations: theta as before; phi0[k][v] over sources;    */
/* the group estimate takes the base of its Pitman-Yor process, P^g phi0_k:  */
/*   phig[g][k][w] = (n - a t + (b + a T_gk) sum_v p_{g,w,v} phi0[k][v]) / (b + N_gk). */
void or_estimates_assoc(const or_model *m, const or_assoc *A, const int32_t *z,
                        const or_counts *c, double *theta, double *phi0, double *phig)
{
    const int64_t G = m->n_groups, K = m->K, V = m->vocab;
    double *p0 = (double *)malloc(sizeof(double) * (size_t)(K * V > 0 ? K * V : 1));
    or_estimates(m, z, c, theta, p0, NULL);
    if (phi0) memcpy(phi0, p0, sizeof(double) * (size_t)(K * V));
    if (phig) {
        for (int64_t g = 0; g < G; ++g)
            for (int64_t k = 0; k < K; ++k) {
                const double N = (double)c->Ngk[g * K + k], T = (double)c->Tgk[g * K + k];
                for (int64_t w = 0; w < V; ++w) {
                    const int64_t cell = (g * K + k) * V + w, q = arow(m, g, w);
                    double base = 0.0;
                    for (int64_t e = A->row_off[q]; e < A->row_off[q + 1]; ++e)
                        base += A->p[e] * p0[k * V + A->src[e]];
                    phig[cell] = ((double)c->n[cell] - m->a * (double)c->t[cell] +
                                  (m->b + m->a * T) * base) /
                                 (m->b + N);
                }
            }
    }
    free(p0);
}

/* Chain histogram with associations: a state is encoded per token with the  */
/* digit (S + 1) z + (r ? s : S) in base K (S + 1) (least significant first). */
int or_chain_histogram_assoc(const or_model *m, const or_assoc *A, or_counts *c, int32_t *z,
                             uint8_t *r, uint8_t *s, uint32_t first_sweep, int64_t n_sweeps,
                             uint64_t seed, int mode, int64_t *hist, int64_t n_bins)
{
    const int64_t S1 = A->S + 1, base = (int64_t)m->K * S1;
    for (int64_t sw = 0; sw < n_sweeps; ++sw) {
        if (or_sweep_assoc(m, A, c, z, r, s, first_sweep + (uint32_t)sw, seed, mode, NULL) != 0)
            return -1;
        int64_t code = 0, mul = 1;
        for (int64_t i = 0; i < m->n_tokens; ++i) {
            code += (S1 * (int64_t)z[i] + (r[i] ? s[i] : A->S)) * mul;
            mul *= base;
        }
        if (code < 0 || code >= n_bins) return -2;
        hist[code] += 1;
    }
    return 0;
}
