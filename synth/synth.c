/*
 * synth.c -- seeded synthetic corpora drawn from the SPDP generative process.
 *
 * Input generator shared by the tests and the benchmark.  It holds none of the
 * sampler's arithmetic (no conditionals, no Stirling numbers, no Philox): it
 * only draws corpora from the generative model of the thesis (chapter "Shared
 * Topic Modelling Using Shadow Poisson Dirichlet Process", graphical model of
 * SPDP, with identity transformation matrices):
 *
 *   phi0_k        ~ a Zipf(s) law over a per-topic random permutation of the
 *                   vocabulary (stand-in for the Dirichlet-distributed shadow
 *                   base: heavy-tailed and with distinct head words per topic)
 *   theta_d       ~ Dirichlet(alpha 1_K)
 *   L_d           ~ Poisson(lambda), redrawn while 0
 *   z_{d,l}       ~ Categorical(theta_d)
 *   w_{d,l}       ~ PYP(a, b, phi0_k) per restaurant (group g, topic k), run
 *                   as a Chinese restaurant in corpus order: a new table with
 *                   probability (b + a T)/(b + N), serving a dish drawn from
 *                   phi0_k (r = 1); otherwise an existing dish w with
 *                   probability proportional to (n_w - a t_w) (r = 0).
 *
 * Randomness: xoshiro256** streams seeded through splitmix64 from (seed,
 * stream kind, index), so every draw is independent of thread count and
 * scheduling.  Documents are laid out group by group; document d belongs to
 * group d / docs_per_group.
 *
 * Build:  gcc -O2 -fopenmp -fPIC -shared synth.c -lm -o libsynth.so
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int32_t n_groups, docs_per_group, vocab, K;
    double doc_len_mean; /* Poisson mean of document length */
    double zipf_s;       /* Zipf exponent of the shadow base */
    double alpha, a, b;  /* generative doc prior, PYP discount, concentration */
} synth_params;

/* ---------------------------- random numbers ---------------------------- */
typedef struct { uint64_t s[4]; } rng_t;

static uint64_t splitmix64(uint64_t *x)
{
    uint64_t z = (*x += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static void rng_seed(rng_t *r, uint64_t seed, uint64_t kind, uint64_t idx)
{
    uint64_t x = seed ^ (kind * 0xD1B54A32D192ED03ull) ^ (idx * 0x8CB92BA72F3D8DD7ull);
    x = splitmix64(&x) ^ idx;
    for (int i = 0; i < 4; ++i) r->s[i] = splitmix64(&x);
}

static inline uint64_t rotl(uint64_t x, int k) { return (x << k) | (x >> (64 - k)); }

static inline uint64_t rng_next(rng_t *r)
{
    uint64_t *s = r->s;
    const uint64_t result = rotl(s[1] * 5, 7) * 9;
    const uint64_t t = s[1] << 17;
    s[2] ^= s[0];
    s[3] ^= s[1];
    s[1] ^= s[2];
    s[0] ^= s[3];
    s[2] ^= t;
    s[3] = rotl(s[3], 45);
    return result;
}

/* uniform in (0,1) */
static inline double u01(rng_t *r) { return ((double)(rng_next(r) >> 11) + 0.5) * (1.0 / 9007199254740992.0); }

static inline uint64_t below(rng_t *r, uint64_t n) { return (uint64_t)(u01(r) * (double)n) % n; }

static double std_normal(rng_t *r)
{
    /* Box-Muller */
    double u1 = u01(r), u2 = u01(r);
    return sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
}

/* log of a Gamma(shape, 1) draw: Marsaglia & Tsang (2000), with the
 * U^{1/shape} boost for shape < 1 applied in log space (no underflow). */
static double log_gamma_draw(rng_t *r, double shape)
{
    double boost = 0.0;
    if (shape < 1.0) {
        boost = log(u01(r)) / shape;
        shape += 1.0;
    }
    const double d = shape - 1.0 / 3.0, c = 1.0 / sqrt(9.0 * d);
    for (;;) {
        double x, v;
        do {
            x = std_normal(r);
            v = 1.0 + c * x;
        } while (v <= 0.0);
        v = v * v * v;
        const double u = u01(r);
        if (u < 1.0 - 0.0331 * x * x * x * x || log(u) < 0.5 * x * x + d * (1.0 - v + log(v)))
            return log(d * v) + boost;
    }
}

/* Poisson: multiplication method for small means, Hormann's PTRS
 * transformed rejection ("The transformed rejection method for generating
 * Poisson random variables", 1993) otherwise. */
static int64_t poisson_draw(rng_t *r, double lam)
{
    if (lam < 10.0) {
        const double L = exp(-lam);
        int64_t k = 0;
        double p = u01(r);
        while (p > L) { ++k; p *= u01(r); }
        return k;
    }
    const double slam = sqrt(lam), loglam = log(lam);
    const double bb = 0.931 + 2.53 * slam;
    const double aa = -0.059 + 0.02483 * bb;
    const double inv_alpha = 1.1239 + 1.1328 / (bb - 3.4);
    const double vr = 0.9277 - 3.6224 / (bb - 2.0);
    for (;;) {
        const double U = u01(r) - 0.5, V = u01(r);
        const double us = 0.5 - fabs(U);
        const int64_t k = (int64_t)floor((2.0 * aa / us + bb) * U + lam + 0.43);
        if (us >= 0.07 && V <= vr) return k;
        if (k < 0 || (us < 0.013 && V > us)) continue;
        if (log(V) + log(inv_alpha) - log(aa / (us * us) + bb) <= -lam + (double)k * loglam - lgamma((double)k + 1.0))
            return k;
    }
}

static int64_t doc_length(const synth_params *p, uint64_t seed, int64_t d)
{
    rng_t r;
    rng_seed(&r, seed, 1, (uint64_t)d);
    int64_t L;
    do { L = poisson_draw(&r, p->doc_len_mean); } while (L <= 0);
    return L;
}

/* Phase 1: document lengths (D = G * docs_per_group).  Returns total tokens. */
int64_t synth_doc_lengths(const synth_params *p, uint64_t seed, int32_t *len)
{
    const int64_t D = (int64_t)p->n_groups * p->docs_per_group;
    int64_t total = 0;
#pragma omp parallel for reduction(+ : total) schedule(static)
    for (int64_t d = 0; d < D; ++d) {
        int64_t L = doc_length(p, seed, d);
        len[d] = (int32_t)L;
        total += L;
    }
    return total;
}

/* ------------------------- small open-addressing map --------------------- */
typedef struct { int32_t key, n, t, pad; } slot_t;
typedef struct { slot_t *s; int64_t cap, used; } wmap_t;

static void wmap_init(wmap_t *m, int64_t hint)
{
    int64_t cap = 64;
    while (cap < 2 * hint) cap <<= 1;
    m->s = (slot_t *)malloc(sizeof(slot_t) * (size_t)cap);
    for (int64_t i = 0; i < cap; ++i) m->s[i].key = -1;
    m->cap = cap;
    m->used = 0;
}

static slot_t *wmap_get(wmap_t *m, int32_t key)
{
    uint64_t h = (uint64_t)(uint32_t)key * 0x9E3779B97F4A7C15ull;
    int64_t i = (int64_t)(h >> 20) & (m->cap - 1);
    for (;;) {
        if (m->s[i].key == key) return &m->s[i];
        if (m->s[i].key < 0) {
            if (2 * (m->used + 1) > m->cap) {
                /* grow and retry */
                slot_t *old = m->s;
                int64_t oc = m->cap;
                m->cap <<= 1;
                m->s = (slot_t *)malloc(sizeof(slot_t) * (size_t)m->cap);
                for (int64_t j = 0; j < m->cap; ++j) m->s[j].key = -1;
                m->used = 0;
                for (int64_t j = 0; j < oc; ++j)
                    if (old[j].key >= 0) {
                        slot_t *ns = wmap_get(m, old[j].key);
                        ns->n = old[j].n;
                        ns->t = old[j].t;
                    }
                free(old);
                return wmap_get(m, key);
            }
            m->s[i].key = key;
            m->s[i].n = 0;
            m->s[i].t = 0;
            m->used++;
            return &m->s[i];
        }
        i = (i + 1) & (m->cap - 1);
    }
}

/* ------------------------------------------------------------------------ */
/* Phase 2: fill words, the generating topics z and table indicators r.      */
/* doc_off must hold the CSR offsets implied by the phase-1 lengths.         */
/* Scratch: about 4 N + 4 K V bytes.                                         */
/* ------------------------------------------------------------------------ */
/* shadow base: Zipf CDF over ranks (cdf [V]), one word permutation per topic
 * (perm [K][V]: the word of rank i in topic k) */
static void base_law(const synth_params *p, uint64_t seed, double *cdf, int32_t *perm)
{
    const int64_t K = p->K, V = p->vocab;
    double acc = 0.0;
    for (int64_t i = 0; i < V; ++i) {
        acc += pow((double)(i + 1), -p->zipf_s);
        cdf[i] = acc;
    }
    for (int64_t i = 0; i < V; ++i) cdf[i] /= acc;
    cdf[V - 1] = 1.0;
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < K; ++k) {
        rng_t r;
        rng_seed(&r, seed, 2, (uint64_t)k);
        int32_t *pk = perm + k * V;
        for (int64_t i = 0; i < V; ++i) pk[i] = (int32_t)i;
        for (int64_t i = V - 1; i > 0; --i) { /* Fisher-Yates */
            int64_t j = (int64_t)below(&r, (uint64_t)(i + 1));
            int32_t tmp = pk[i]; pk[i] = pk[j]; pk[j] = tmp;
        }
    }
}

/* The generating shadow base phi0 [K][V] of the corpus drawn with (p, seed):
 * the probability with which a new table of topic k serves word w, i.e. the
 * CDF step of w's rank (the law new tables draw from in synth_fill). */
int synth_phi0(const synth_params *p, uint64_t seed, double *phi0)
{
    const int64_t K = p->K, V = p->vocab;
    double *cdf = (double *)malloc(sizeof(double) * (size_t)V);
    int32_t *perm = (int32_t *)malloc(sizeof(int32_t) * (size_t)(K * V));
    if (!cdf || !perm) { free(cdf); free(perm); return -1; }
    base_law(p, seed, cdf, perm);
    for (int64_t k = 0; k < K; ++k)
        for (int64_t i = 0; i < V; ++i)
            phi0[k * V + perm[k * V + i]] = cdf[i] - (i > 0 ? cdf[i - 1] : 0.0);
    free(cdf);
    free(perm);
    return 0;
}

int synth_fill(const synth_params *p, uint64_t seed, const int64_t *doc_off, int32_t *words,
               int32_t *z, uint8_t *rr)
{
    const int64_t G = p->n_groups, K = p->K, V = p->vocab;
    const int64_t D = G * p->docs_per_group;
    const int64_t N = doc_off[D];

    double *cdf = (double *)malloc(sizeof(double) * (size_t)V);
    int32_t *perm = (int32_t *)malloc(sizeof(int32_t) * (size_t)(K * V));
    if (!cdf || !perm) return -1;
    base_law(p, seed, cdf, perm);

    /* topics: theta_d ~ Dir(alpha), z ~ theta_d */
#pragma omp parallel
    {
        double *cum = (double *)malloc(sizeof(double) * (size_t)K);
#pragma omp for schedule(dynamic, 64)
        for (int64_t d = 0; d < D; ++d) {
            rng_t r;
            rng_seed(&r, seed, 3, (uint64_t)d);
            double mx = -INFINITY;
            for (int64_t k = 0; k < K; ++k) {
                cum[k] = log_gamma_draw(&r, p->alpha);
                if (cum[k] > mx) mx = cum[k];
            }
            double acc = 0.0;
            for (int64_t k = 0; k < K; ++k) { acc += exp(cum[k] - mx); cum[k] = acc; }
            for (int64_t i = doc_off[d]; i < doc_off[d + 1]; ++i) {
                const double u = u01(&r) * acc;
                int64_t lo = 0, hi = K - 1;
                while (lo < hi) { int64_t mid = (lo + hi) / 2; if (cum[mid] > u) hi = mid; else lo = mid + 1; }
                z[i] = (int32_t)lo;
            }
        }
        free(cum);
    }

    /* bucket token positions by restaurant (g, k), keeping corpus order */
    const int64_t R = G * K;
    int64_t *start = (int64_t *)calloc((size_t)(R + 1), sizeof(int64_t));
    int32_t *pos = (int32_t *)malloc(sizeof(int32_t) * (size_t)(N > 0 ? N : 1));
    if (!start || !pos) return -1;
    for (int64_t d = 0; d < D; ++d) {
        const int64_t g = d / p->docs_per_group;
        for (int64_t i = doc_off[d]; i < doc_off[d + 1]; ++i) start[g * K + z[i] + 1] += 1;
    }
    for (int64_t q = 0; q < R; ++q) start[q + 1] += start[q];
    {
        int64_t *fill = (int64_t *)malloc(sizeof(int64_t) * (size_t)R);
        memcpy(fill, start, sizeof(int64_t) * (size_t)R);
        for (int64_t d = 0; d < D; ++d) {
            const int64_t g = d / p->docs_per_group;
            for (int64_t i = doc_off[d]; i < doc_off[d + 1]; ++i) pos[fill[g * K + z[i]]++] = (int32_t)i;
        }
        free(fill);
    }

    /* one Chinese restaurant per (g, k) */
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t q = 0; q < R; ++q) {
        const int64_t k = q % K;
        const int64_t cnt = start[q + 1] - start[q];
        if (cnt == 0) continue;
        rng_t r;
        rng_seed(&r, seed, 4, (uint64_t)q);
        wmap_t map;
        wmap_init(&map, cnt < 1024 ? cnt : 1024);
        int64_t T = 0;
        for (int64_t c = 0; c < cnt; ++c) {
            const int64_t i = pos[start[q] + c];
            const double pnew = (p->b + p->a * (double)T) / (p->b + (double)c);
            int32_t w;
            if (c == 0 || u01(&r) < pnew) {
                const double u = u01(&r);
                int64_t lo = 0, hi = V - 1;
                while (lo < hi) { int64_t mid = (lo + hi) / 2; if (cdf[mid] > u) hi = mid; else lo = mid + 1; }
                w = perm[k * V + lo];
                slot_t *s = wmap_get(&map, w);
                s->n += 1;
                s->t += 1;
                T += 1;
                rr[i] = 1;
            } else {
                /* existing dish w with probability (n_w - a t_w)/(N - a T):
                 * uniform previous customer, accepted w.p. 1 - a t_w / n_w */
                for (;;) {
                    const int64_t j = pos[start[q] + (int64_t)below(&r, (uint64_t)c)];
                    w = words[j];
                    slot_t *s = wmap_get(&map, w);
                    if (u01(&r) * (double)s->n < (double)s->n - p->a * (double)s->t) {
                        s->n += 1;
                        break;
                    }
                }
                rr[i] = 0;
            }
            words[i] = w;
        }
        free(map.s);
    }
    free(start);
    free(pos);
    free(cdf);
    free(perm);
    return 0;
}
