/*
 * Seeded synthetic corpus generator: Zipf unigram with a topic mixture.
 *
 * This module only produces input data (word-id streams). It holds none of
 * the word2vec arithmetic and is shared, as data, by the GPU path's tests and
 * by the CPU oracle's tests.
 *
 * Model (stands in for the Text8 corpus used in the experiment setup, §4.1):
 *   base distribution  p(r) proportional to r^-s over ranks r = 1..V, word id = r-1;
 *   topic tau < T owns a subset S_tau of round(frac*V) distinct ids drawn
 *   uniformly without replacement;
 *   document k (doc_len tokens) picks tau uniformly; its tokens are i.i.d. from
 *   p_tau(i) proportional to p(i) * (boost if i in S_tau else 1).
 *   p_tau is sampled as a mixture: with probability 1/Z_tau from the base
 *   distribution, else from p restricted to S_tau, Z_tau = 1 + (boost-1) p(S_tau).
 *   T = 0 gives plain i.i.d. Zipf.
 *
 * Every document draws from its own counter-keyed SplitMix64 stream, so the
 * output does not depend on the number of threads.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static inline uint64_t sm64_next(uint64_t *s) {
    uint64_t z = (*s += 0x9E3779B97F4A7C15ULL);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static inline uint64_t mix_key(uint64_t seed, uint64_t a, uint64_t b) {
    uint64_t s = seed ^ 0x5851F42D4C957F2DULL;
    uint64_t k = sm64_next(&s) ^ (a * 0xD1342543DE82EF95ULL);
    s = k;
    k = sm64_next(&s) ^ (b * 0x9E3779B97F4A7C15ULL);
    s = k;
    return sm64_next(&s);
}

/* uniform in [0,1) with 53 random bits */
static inline double u01(uint64_t *s) { return (double)(sm64_next(s) >> 11) * (1.0 / 9007199254740992.0); }
/* uniform integer in [0,n) (multiply-high; bias < 2^-32 for n < 2^32) */
static inline uint32_t below(uint64_t *s, uint32_t n) {
    return (uint32_t)(((sm64_next(s) >> 32) * (uint64_t)n) >> 32);
}

typedef struct {
    int32_t n;
    double *prob;    /* acceptance probability of column i */
    int32_t *alias;  /* alias column */
    int32_t *ids;    /* word id of column i (NULL = identity) */
} alias_t;

/* Vose's alias method over weights w[0..n) */
static int alias_build(alias_t *a, const double *w, int32_t n, const int32_t *ids) {
    a->n = n;
    a->prob = (double *)malloc(sizeof(double) * (size_t)n);
    a->alias = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
    a->ids = NULL;
    int32_t *small = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
    int32_t *large = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
    double *sc = (double *)malloc(sizeof(double) * (size_t)n);
    if (!a->prob || !a->alias || !small || !large || !sc) return -1;
    double tot = 0.0;
    for (int32_t i = 0; i < n; i++) tot += w[i];
    int32_t ns = 0, nl = 0;
    for (int32_t i = 0; i < n; i++) {
        sc[i] = w[i] * (double)n / tot;
        if (sc[i] < 1.0) small[ns++] = i; else large[nl++] = i;
    }
    while (ns > 0 && nl > 0) {
        int32_t l = small[--ns], g = large[--nl];
        a->prob[l] = sc[l];
        a->alias[l] = g;
        sc[g] = (sc[g] + sc[l]) - 1.0;
        if (sc[g] < 1.0) small[ns++] = g; else large[nl++] = g;
    }
    while (nl > 0) { int32_t g = large[--nl]; a->prob[g] = 1.0; a->alias[g] = g; }
    while (ns > 0) { int32_t l = small[--ns]; a->prob[l] = 1.0; a->alias[l] = l; }
    free(small); free(large); free(sc);
    if (ids) {
        a->ids = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
        if (!a->ids) return -1;
        memcpy(a->ids, ids, sizeof(int32_t) * (size_t)n);
    }
    return 0;
}

static inline int32_t alias_draw(const alias_t *a, uint64_t *s) {
    uint32_t col = below(s, (uint32_t)a->n);
    double u = u01(s);
    int32_t k = (u < a->prob[col]) ? (int32_t)col : a->alias[col];
    return a->ids ? a->ids[k] : k;
}

static void alias_free(alias_t *a) { free(a->prob); free(a->alias); free(a->ids); }

/* Zipf weights p(r) = r^-s / H, r = 1..V (id = r-1). Writes normalised p. */
int synth_zipf_probs(int32_t V, double s, double *p) {
    if (V < 1) return -1;
    double tot = 0.0;
    for (int32_t i = 0; i < V; i++) { p[i] = pow((double)(i + 1), -s); tot += p[i]; }
    for (int32_t i = 0; i < V; i++) p[i] /= tot;
    return 0;
}

/* The ids owned by topic tau: m distinct ids, partial Fisher-Yates keyed by (seed, tau). */
static void topic_subset(uint64_t seed, int32_t tau, int32_t V, int32_t m, int32_t *perm, int32_t *out) {
    for (int32_t i = 0; i < V; i++) perm[i] = i;
    uint64_t st = mix_key(seed, 0x70C1CULL, (uint64_t)tau);
    for (int32_t i = 0; i < m; i++) {
        int32_t j = i + (int32_t)below(&st, (uint32_t)(V - i));
        int32_t t = perm[i]; perm[i] = perm[j]; perm[j] = t;
        out[i] = perm[i];
    }
}

int synth_topic_subset(uint64_t seed, int32_t tau, int32_t V, int32_t m, int32_t *out) {
    int32_t *perm = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
    if (!perm) return -1;
    topic_subset(seed, tau, V, m, perm, out);
    free(perm);
    return 0;
}

int32_t synth_topic_size(int32_t V, double frac) {
    double m = floor(frac * (double)V + 0.5);
    if (m < 1) m = 1;
    if (m > V) m = V;
    return (int32_t)m;
}

/* Topic of document k. */
int32_t synth_doc_topic(uint64_t seed, int64_t doc, int32_t T) {
    if (T <= 0) return -1;
    uint64_t st = mix_key(seed, 0xD0CULL, (uint64_t)doc);
    return (int32_t)below(&st, (uint32_t)T);
}

/*
 * Fill out[0..n_tokens) with word ids in [0, V).
 * Returns 0 on success, -1 on bad arguments or allocation failure.
 */
int synth_corpus(int64_t n_tokens, int32_t V, double s, int32_t T, double frac, double boost,
                 int32_t doc_len, uint64_t seed, int32_t n_threads, int32_t *out) {
    if (n_tokens < 0 || V < 1 || doc_len < 1 || T < 0 || boost < 1.0) return -1;
    double *p = (double *)malloc(sizeof(double) * (size_t)V);
    if (!p) return -1;
    synth_zipf_probs(V, s, p);
    alias_t base;
    if (alias_build(&base, p, V, NULL)) return -1;

    alias_t *topics = NULL;
    double *pbase = NULL; /* probability of drawing from the base table, per topic */
    if (T > 0) {
        int32_t m = synth_topic_size(V, frac);
        topics = (alias_t *)calloc((size_t)T, sizeof(alias_t));
        pbase = (double *)malloc(sizeof(double) * (size_t)T);
        int32_t *perm = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
        int32_t *sub = (int32_t *)malloc(sizeof(int32_t) * (size_t)m);
        double *w = (double *)malloc(sizeof(double) * (size_t)m);
        if (!topics || !pbase || !perm || !sub || !w) return -1;
        for (int32_t t = 0; t < T; t++) {
            topic_subset(seed, t, V, m, perm, sub);
            double ps = 0.0;
            for (int32_t i = 0; i < m; i++) { w[i] = p[sub[i]]; ps += w[i]; }
            pbase[t] = 1.0 / (1.0 + (boost - 1.0) * ps);
            if (alias_build(&topics[t], w, m, sub)) return -1;
        }
        free(perm); free(sub); free(w);
    }
    int64_t n_docs = (n_tokens + doc_len - 1) / doc_len;
#ifdef _OPENMP
    if (n_threads > 0) omp_set_num_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 64)
#endif
    for (int64_t d = 0; d < n_docs; d++) {
        int64_t lo = d * (int64_t)doc_len;
        int64_t hi = lo + doc_len;
        if (hi > n_tokens) hi = n_tokens;
        uint64_t st = mix_key(seed, 0x70CE5ULL, (uint64_t)d);
        if (T == 0) {
            for (int64_t i = lo; i < hi; i++) out[i] = alias_draw(&base, &st);
        } else {
            int32_t tau = synth_doc_topic(seed, d, T);
            const alias_t *ta = &topics[tau];
            double pb = pbase[tau];
            for (int64_t i = lo; i < hi; i++)
                out[i] = (u01(&st) < pb) ? alias_draw(&base, &st) : alias_draw(ta, &st);
        }
    }
    alias_free(&base);
    if (T > 0) {
        for (int32_t t = 0; t < T; t++) alias_free(&topics[t]);
        free(topics); free(pbase);
    }
    free(p);
    return 0;
}
