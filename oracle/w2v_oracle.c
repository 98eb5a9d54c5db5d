/*
 * CPU oracle for hierarchical-softmax word2vec training, written from
 * Vuurens, Eickhoff, de Vries, "Efficient Parallel Learning of Word2Vec".
 *
 * TEST INFRASTRUCTURE ONLY: plain, slow and single-threaded on purpose, so
 * that each step can be checked against the paper by eye. Only tests, the
 * smoke check and the benchmark's CPU-baseline leg may call it; the GPU
 * library never does. Built with -ffp-contract=off so that every float
 * operation rounds exactly once, as written.
 *
 * Where the paper is silent the readings below are used (each is restated at
 * the function that applies it):
 *   R1  Algorithm 1 walks the Huffman path of the outer word v with the input
 *       vector of the window word w.
 *   R2  The two saxpy scalars inside the node loop of Algorithm 1 are the
 *       computed `gradient` (the printed `1` would leave `gradient` unused).
 *   R3  `hiddenlayer` starts at zero for every (v, w) pair.
 *   R4  Within a node, the hidden-layer update uses the node vector before
 *       that node's own update; vector[w] is updated only after the path.
 *   R5  sigmoid is the exact logistic function (no table, no clipping).
 *   R6  The turn t is the code bit; the target of node n is 1 - t, so
 *       P(v|w) = prod_j sigma((1 - 2 t_j) x_w . y_{n_j}).
 *   R7  Huffman tree: two-queue merge over the vocabulary sorted by (count
 *       desc, id asc); a leaf wins a count tie; the first child taken gets
 *       bit 0; the a-th merge creates inner node a; the root is V-2.
 *   R8  isFrequent(n) holds for the k inner nodes created last (n >= V-1-k),
 *       which are the k inner nodes with the largest counts and form the top
 *       of the tree.
 *   R9  "time to flush cache": after every flush_every centre words.
 *   R10 "time to update alpha": alpha is a step function of the raw stream
 *       position, one step per 10,000 tokens, decaying linearly to 1e-4*alpha0.
 *   R11 downsample: keep probability sqrt(q) + q with q = t*N_t/count, drawn
 *       from Philox4x32-10 keyed by the raw token index.
 *   R12 window: effective half-width W - b with b uniform on {0..W-1}.
 *   R13 documents of doc_len raw tokens; windows never cross them; dropped and
 *       subsampled tokens are removed before windowing.
 *
 * Negative sampling (named in §2 as the alternative to the hierarchical
 * softmax; the opening of §3.2 describes Ji et al.'s mini-batch form of it):
 *   NS1  the noise distribution is the unigram distribution raised to 3/4 (the
 *       choice of Mikolov et al., whom §2 cites), with the weight of a word of
 *       count c taken in integers as isqrt(c * isqrt(c)), so that every
 *       implementation draws the same words.
 *   NS2  noise table of T = 2^L entries: entry i holds the word v whose weight
 *       prefix sums satisfy Q[v] <= floor(i Q / T) < Q[v+1]; a draw r (32 bits)
 *       picks entry r >> (32 - L).
 *   NS3  a centre's K negatives are shared by all of its window words (Ji et
 *       al., §3.2): negative 4h+i is drawn from word i of Philox4x32-10 with
 *       counter (raw index lo, hi, epoch, 1 + h); a negative equal to the centre
 *       word is dropped.
 *   NS4  mini-batch update (§3.2, level-3 BLAS form; §4.3 notes that it does
 *       not use updated vectors within a mini-batch): with X the window words' vectors and Y
 *       the output vectors of the centre (label 1) and its negatives (label 0),
 *       S = X Y^T, G = alpha (labels - sigmoid(S)); X gains G Y and Y gains
 *       G^T X, both from the values at the start of the centre.
 */
#include "w2v_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Vocabulary: count ids, drop those below min_count ("mintf", §4.1), order   */
/* by (count desc, id asc).                                                   */
/* ------------------------------------------------------------------------ */

/* counts[id] = occurrences of id; returns the number of out-of-range tokens. */
int64_t or_count(const int32_t *tokens, int64_t n, int32_t id_space, int64_t *counts) {
    int64_t bad = 0;
    for (int32_t i = 0; i < id_space; i++) counts[i] = 0;
    for (int64_t i = 0; i < n; i++) {
        int32_t t = tokens[i];
        if (t < 0 || t >= id_space) bad++;
        else counts[t]++;
    }
    return bad;
}

static const int64_t *g_sort_counts;
static int cmp_vocab(const void *a, const void *b) {
    int32_t ia = *(const int32_t *)a, ib = *(const int32_t *)b;
    int64_t ca = g_sort_counts[ia], cb = g_sort_counts[ib];
    if (ca != cb) return ca > cb ? -1 : 1;
    return ia < ib ? -1 : (ia > ib ? 1 : 0);
}

/* Returns V (number of kept ids). vocab_ids/vocab_counts hold the first V entries. */
int32_t or_vocab(const int64_t *counts, int32_t id_space, int64_t min_count, int32_t *vocab_ids,
                 int64_t *vocab_counts, int32_t *id_to_vocab, int64_t *train_words) {
    int32_t V = 0;
    for (int32_t i = 0; i < id_space; i++)
        if (counts[i] >= min_count) vocab_ids[V++] = i;
    g_sort_counts = counts;
    qsort(vocab_ids, (size_t)V, sizeof(int32_t), cmp_vocab);
    int64_t tw = 0;
    for (int32_t i = 0; i < id_space; i++) id_to_vocab[i] = -1;
    for (int32_t r = 0; r < V; r++) {
        vocab_counts[r] = counts[vocab_ids[r]];
        id_to_vocab[vocab_ids[r]] = r;
        tw += vocab_counts[r];
    }
    *train_words = tw;
    return V;
}

void or_remap(const int32_t *tokens, int64_t n, const int32_t *id_to_vocab, int32_t *out) {
    for (int64_t i = 0; i < n; i++) out[i] = id_to_vocab[tokens[i]];
}

/* ------------------------------------------------------------------------ */
/* Huffman tree (§2: the output layer is a binary Huffman tree; a word is     */
/* predicted by the left/right turns at the inner nodes on its root path).    */
/* Construction rule R7. Node numbering: leaves 0..V-1 = vocabulary index,    */
/* inner node a = V + a; parent[] holds inner indices a (-1 for the root).    */
/* ------------------------------------------------------------------------ */
int or_huffman(const int64_t *vocab_counts, int32_t V, int32_t *parent, uint8_t *bit, int64_t *node_count) {
    if (V < 2) return -1;
    int32_t nn = 2 * V - 1;
    for (int32_t i = 0; i < nn; i++) { parent[i] = -1; bit[i] = 0; }
    int64_t *icount = node_count + V;        /* counts of inner nodes */
    for (int32_t i = 0; i < V; i++) node_count[i] = vocab_counts[i];
    int32_t leaf = V - 1;    /* queue of leaves in ascending count: V-1, V-2, ..., 0 */
    int32_t ihead = 0;       /* queue of inner nodes in creation order */
    for (int32_t a = 0; a < V - 1; a++) {
        int64_t sum = 0;
        for (int32_t pick = 0; pick < 2; pick++) {
            int use_leaf;
            if (leaf < 0) use_leaf = 0;
            else if (ihead >= a) use_leaf = 1;                       /* no inner node waiting */
            else use_leaf = vocab_counts[leaf] <= icount[ihead];    /* leaf wins a tie */
            int32_t child;
            if (use_leaf) child = leaf--;
            else child = V + ihead++;
            parent[child] = a;
            bit[child] = (uint8_t)pick;
            sum += node_count[child];
        }
        icount[a] = sum;
    }
    return 0;
}

/*
 * Per word v: codelen[v] = depth; points of v, root first, in
 * points[point_off[v] .. point_off[v+1]); bit j of code[v] = turn taken at
 * points[v][j] (the bit of the child on the path). Returns -1 if a code is
 * longer than 64 or points_cap is too small (points may be NULL: size only).
 */
int or_huffman_codes(const int32_t *parent, const uint8_t *bit, int32_t V, uint8_t *codelen, uint64_t *code,
                     int32_t *point_off, int32_t *points, int64_t points_cap) {
    int32_t path[128];
    uint8_t turn[128];
    int64_t off = 0;
    for (int32_t v = 0; v < V; v++) {
        int32_t depth = 0;
        int32_t node = v;
        while (parent[node] >= 0) {
            if (depth >= 64) return -1;
            path[depth] = parent[node];
            turn[depth] = bit[node];
            depth++;
            node = V + parent[node];
        }
        codelen[v] = (uint8_t)depth;
        point_off[v] = (int32_t)off;
        uint64_t c = 0;
        for (int32_t j = 0; j < depth; j++) {
            /* path[] was collected leaf-upwards; position j from the root is depth-1-j */
            int32_t up = depth - 1 - j;
            if (turn[up]) c |= (uint64_t)1 << j;
            if (points) {
                if (off + j >= points_cap) return -1;
                points[off + j] = path[up];
            }
        }
        code[v] = c;
        off += depth;
    }
    point_off[V] = (int32_t)off;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two       */
/* 32x32->64 multiplies with key bumping by the Weyl constants.               */
/* ------------------------------------------------------------------------ */
void or_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; r++) {
        if (r > 0) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
        uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        c0 = hi1 ^ c1 ^ k0;
        c1 = lo1;
        c2 = hi0 ^ c3 ^ k1;
        c3 = lo0;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

static void draw(uint64_t seed, int64_t raw, int32_t epoch, uint32_t r[4]) {
    uint32_t ctr[4] = {(uint32_t)raw, (uint32_t)((uint64_t)raw >> 32), (uint32_t)epoch, 0u};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    or_philox4x32_10(ctr, key, r);
}

/* ------------------------------------------------------------------------ */
/* Tables: keep thresholds (R11) and learning rate (R10).                     */
/* ------------------------------------------------------------------------ */
void or_keep_thresholds(const int64_t *vocab_counts, int32_t V, double sample, int64_t train_words,
                        uint64_t *thr) {
    const uint64_t all = (uint64_t)1 << 32;
    for (int32_t v = 0; v < V; v++) {
        if (!(sample > 0.0)) { thr[v] = all; continue; }
        double tn = sample * (double)train_words;
        double q = tn / (double)vocab_counts[v];
        double pk = sqrt(q) + q;
        thr[v] = (pk >= 1.0) ? all : (uint64_t)floor(pk * 4294967296.0);
    }
}

float or_alpha(float alpha0, int64_t raw_pos, int32_t epoch, int32_t n_epochs, int64_t corpus_tokens) {
    int64_t progress = (int64_t)epoch * corpus_tokens + raw_pos;
    int64_t block = progress / 10000;
    double frac = (double)(block * 10000) / (double)((int64_t)n_epochs * corpus_tokens + 1);
    double a = 1.0 - frac;
    if (a < 1e-4) a = 1e-4;
    return (float)((double)alpha0 * a);
}

/* ------------------------------------------------------------------------ */
/* Sampler: subsampling (R11), documents (R13), window (R12).                 */
/* ------------------------------------------------------------------------ */
typedef struct {
    int32_t n;        /* kept tokens in the document */
    int32_t *vid;     /* vocabulary index */
    int64_t *raw;     /* global raw index */
    int32_t *eff;     /* effective window half-width of this centre */
} doc_t;

/* Kept tokens of the document starting at local index lo (global raw index first_raw + lo). */
static void doc_sample(const int32_t *tokens, int64_t n, const or_params *p, const uint64_t *thr, int64_t lo,
                       doc_t *d, int64_t *in_vocab) {
    int64_t hi = lo + p->doc_len;
    if (hi > n) hi = n;
    d->n = 0;
    for (int64_t i = lo; i < hi; i++) {
        int32_t v = tokens[i];
        if (v < 0) continue;
        (*in_vocab)++;
        int64_t g = p->first_raw_index + i;
        uint32_t r[4];
        draw(p->seed, g, p->epoch, r);
        if ((uint64_t)r[0] >= thr[v]) continue;
        uint32_t b = (uint32_t)(((uint64_t)r[1] * (uint64_t)p->window) >> 32);
        d->vid[d->n] = v;
        d->raw[d->n] = g;
        d->eff[d->n] = p->window - (int32_t)b;
        d->n++;
    }
}

static int doc_alloc(doc_t *d, int32_t doc_len) {
    d->vid = (int32_t *)malloc(sizeof(int32_t) * (size_t)doc_len);
    d->raw = (int64_t *)malloc(sizeof(int64_t) * (size_t)doc_len);
    d->eff = (int32_t *)malloc(sizeof(int32_t) * (size_t)doc_len);
    return (d->vid && d->raw && d->eff) ? 0 : -1;
}
static void doc_free(doc_t *d) { free(d->vid); free(d->raw); free(d->eff); }

/* Window positions of centre j: c in [j-eff, j+eff], c != j, 0 <= c < n, ascending. */
static int32_t window_of(const doc_t *d, int32_t j, int32_t *ctx) {
    int32_t e = d->eff[j], m = 0;
    for (int32_t c = j - e; c <= j + e; c++)
        if (c != j && c >= 0 && c < d->n) ctx[m++] = c;
    return m;
}

static inline uint64_t fmix64(uint64_t k) {
    k ^= k >> 33; k *= 0xFF51AFD7ED558CCDULL;
    k ^= k >> 33; k *= 0xC4CEB9FE1A85EC53ULL;
    k ^= k >> 33;
    return k;
}

/*
 * All (centre, context) pairs in stream order (documents ascending, centres
 * ascending, window positions ascending), as global raw indices. Writes the
 * first `cap` pairs (arrays may be NULL), the keep mask per local token (may
 * be NULL), the number of kept centres and an order-independent checksum.
 * Returns the total number of pairs.
 */
int64_t or_sample_pairs(const int32_t *tokens, int64_t n, const or_params *p, const int64_t *vocab_counts,
                        int64_t *centre_raw, int64_t *context_raw, int64_t cap, uint8_t *keep_mask,
                        int64_t *n_kept, uint64_t *checksum) {
    doc_t d;
    if (doc_alloc(&d, p->doc_len)) return -1;
    uint64_t *thr = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)p->V);
    if (!thr) return -1;
    or_keep_thresholds(vocab_counts, p->V, p->sample, p->train_words, thr);
    int32_t ctx[2 * 1024 + 2];
    int64_t np = 0, nk = 0, inv = 0;
    uint64_t cs = 0;
    if (keep_mask) memset(keep_mask, 0, (size_t)n);
    for (int64_t lo = 0; lo < n; lo += p->doc_len) {
        doc_sample(tokens, n, p, thr, lo, &d, &inv);
        nk += d.n;
        for (int32_t j = 0; j < d.n; j++) {
            if (keep_mask) keep_mask[d.raw[j] - p->first_raw_index] = 1;
            int32_t m = window_of(&d, j, ctx);
            for (int32_t q = 0; q < m; q++) {
                int64_t c = d.raw[j], x = d.raw[ctx[q]];
                if (np < cap) {
                    if (centre_raw) centre_raw[np] = c;
                    if (context_raw) context_raw[np] = x;
                }
                cs += fmix64((uint64_t)c * 0x9E3779B97F4A7C15ULL + (uint64_t)x);
                np++;
            }
        }
    }
    doc_free(&d);
    free(thr);
    if (n_kept) *n_kept = nk;
    if (checksum) *checksum = cs;
    return np;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 1 (Cached Skipgram HS), one worker.                             */
/* ------------------------------------------------------------------------ */

/* sdot: single-precision dot product, accumulated in order (§3.2). */
static float sdot(int32_t n, const float *x, const float *y) {
    float s = 0.0f;
    for (int32_t i = 0; i < n; i++) s += x[i] * y[i];
    return s;
}
/* saxpy: y += a*x. */
static void saxpy(int32_t n, float a, const float *x, float *y) {
    for (int32_t i = 0; i < n; i++) y[i] += a * x[i];
}
/* R5: exact logistic function in single precision. */
static float sigmoidf(float z) { return 1.0f / (1.0f + expf(-z)); }

typedef struct {
    int32_t k, first;        /* cached nodes: first .. first+k-1 (R8) */
    float *cachedweight;     /* [k][dim] */
    float *original;         /* [k][dim] */
    uint8_t *cached;         /* [k] */
} cache_t;

/* The vector used for inner node n (lazy fill of the cache when frequent). */
static float *used_weight(cache_t *c, float *syn1, int32_t dim, int32_t n) {
    if (c->k > 0 && n >= c->first) {               /* isFrequent(n) */
        int32_t s = n - c->first;
        float *cw = c->cachedweight + (size_t)s * dim;
        if (!c->cached[s]) {                       /* first use since the last flush */
            memcpy(cw, syn1 + (size_t)n * dim, sizeof(float) * (size_t)dim);          /* scopy */
            memcpy(c->original + (size_t)s * dim, cw, sizeof(float) * (size_t)dim);   /* scopy */
            c->cached[s] = 1;
        }
        return cw;
    }
    return syn1 + (size_t)n * dim;
}

/* Flush: cached -= original; weight += cached; un-mark (§3.2, Algorithm 1). */
static void flush_cache(cache_t *c, float *syn1, int32_t dim) {
    for (int32_t s = 0; s < c->k; s++) {
        if (!c->cached[s]) continue;
        float *cw = c->cachedweight + (size_t)s * dim;
        saxpy(dim, -1.0f, c->original + (size_t)s * dim, cw);
        saxpy(dim, 1.0f, cw, syn1 + (size_t)(c->first + s) * dim);
        c->cached[s] = 0;
    }
}

/*
 * One (v, w) pair: walk the tree path of `path_word` with input vector x
 * (R1, R3, R4, R6); returns the number of nodes; accumulates into hidden.
 */
static int32_t walk_pair(cache_t *c, float *syn1, int32_t dim, const or_tree *t, int32_t path_word,
                         const float *x, float alpha, float *hidden) {
    int32_t len = t->codelen[path_word];
    const int32_t *pts = t->points + t->point_off[path_word];
    uint64_t code = t->code[path_word];
    for (int32_t j = 0; j < len; j++) {
        int32_t n = pts[j];
        float turn = (float)((code >> j) & 1u);
        float *used = used_weight(c, syn1, dim, n);
        float f = sigmoidf(sdot(dim, x, used));
        float gradient = (1.0f - turn - f) * alpha;
        saxpy(dim, gradient, used, hidden);     /* R2, R4: uses the node before its update */
        saxpy(dim, gradient, x, used);
    }
    return len;
}

static int cache_init(cache_t *c, const or_params *p) {
    c->k = p->cache_k;
    c->first = p->V - 1 - p->cache_k;
    c->cachedweight = c->original = NULL;
    c->cached = NULL;
    if (c->k <= 0) { c->k = 0; return 0; }
    c->cachedweight = (float *)malloc(sizeof(float) * (size_t)c->k * p->dim);
    c->original = (float *)malloc(sizeof(float) * (size_t)c->k * p->dim);
    c->cached = (uint8_t *)calloc((size_t)c->k, 1);
    return (c->cachedweight && c->original && c->cached) ? 0 : -1;
}
static void cache_free(cache_t *c) { free(c->cachedweight); free(c->original); free(c->cached); }

/*
 * One epoch of asynchronous training as one sequential worker.
 * arch 0 (skip-gram): order 0 is Algorithm 1 as printed; order 1 swaps the
 * window and node loops (for each node, all window words in order), which is
 * the same computation whenever no word occurs twice in one window.
 * arch 1 (CBOW): the input is the mean of the window vectors; one path walk
 * per centre; the accumulated hidden-layer gradient is added to every window
 * vector.
 * stats: [raw tokens, in-vocabulary tokens, kept centres, pairs, node updates].
 */
int or_train(float *syn0, float *syn1, const or_tree *t, const int32_t *tokens, int64_t n, const or_params *p,
             int64_t *stats) {
    const int32_t dim = p->dim;
    if (p->V < 2 || p->window < 1 || p->window > 1024 || p->doc_len < 1 || p->flush_every < 1) return -1;
    doc_t d;
    cache_t c;
    if (doc_alloc(&d, p->doc_len) || cache_init(&c, p)) return -1;
    uint64_t *thr = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)p->V);
    int32_t P = 2 * p->window;
    float *hidden = (float *)malloc(sizeof(float) * (size_t)dim * (P + 1));
    float *h = (float *)malloc(sizeof(float) * (size_t)dim);
    int32_t ctx[2 * 1024 + 2];
    if (!thr || !hidden || !h) return -1;
    or_keep_thresholds(t->vocab_counts, p->V, p->sample, p->train_words, thr);

    int64_t raw = 0, inv = 0, kept = 0, pairs = 0, nodes = 0, since_flush = 0;
    int stop = 0;
    for (int64_t lo = 0; lo < n && !stop; lo += p->doc_len) {
        int64_t hi = lo + p->doc_len < n ? lo + p->doc_len : n;
        raw += hi - lo;
        doc_sample(tokens, n, p, thr, lo, &d, &inv);
        for (int32_t j = 0; j < d.n; j++) {
            if (p->max_centres >= 0 && kept >= p->max_centres) { stop = 1; break; }
            int32_t v = d.vid[j];
            float alpha = or_alpha(p->alpha0, d.raw[j], p->epoch, p->n_epochs, p->corpus_tokens);
            int32_t m = window_of(&d, j, ctx);
            kept++;
            if (p->arch == 1) {
                /* CBOW: h = mean of the window vectors; e = sum_j g_j y_j; vector[w] += e for each w. */
                if (m > 0) {
                    memset(h, 0, sizeof(float) * (size_t)dim);
                    for (int32_t q = 0; q < m; q++) saxpy(dim, 1.0f, syn0 + (size_t)d.vid[ctx[q]] * dim, h);
                    for (int32_t i = 0; i < dim; i++) h[i] = h[i] / (float)m;
                    memset(hidden, 0, sizeof(float) * (size_t)dim);
                    nodes += walk_pair(&c, syn1, dim, t, v, h, alpha, hidden);
                    for (int32_t q = 0; q < m; q++) saxpy(dim, 1.0f, hidden, syn0 + (size_t)d.vid[ctx[q]] * dim);
                    pairs += m;
                }
            } else if (p->order == 0 || p->orient == 1) {
                /* Algorithm 1 as printed: for each window word, walk the path, then update vector[w]. */
                for (int32_t q = 0; q < m; q++) {
                    int32_t w = d.vid[ctx[q]];
                    int32_t in_word = p->orient == 0 ? w : v;
                    int32_t path_word = p->orient == 0 ? v : w;
                    float *x = syn0 + (size_t)in_word * dim;
                    memset(hidden, 0, sizeof(float) * (size_t)dim);
                    nodes += walk_pair(&c, syn1, dim, t, path_word, x, alpha, hidden);
                    saxpy(dim, 1.0f, hidden, x);
                    pairs++;
                }
            } else {
                /* Loop interchange: each node row is visited once per centre, all window words in order. */
                int32_t len = t->codelen[v];
                const int32_t *pts = t->points + t->point_off[v];
                uint64_t code = t->code[v];
                memset(hidden, 0, sizeof(float) * (size_t)dim * m);
                for (int32_t jn = 0; jn < len; jn++) {
                    int32_t nn = pts[jn];
                    float turn = (float)((code >> jn) & 1u);
                    float *used = used_weight(&c, syn1, dim, nn);
                    for (int32_t q = 0; q < m; q++) {
                        const float *x = syn0 + (size_t)d.vid[ctx[q]] * dim;
                        float f = sigmoidf(sdot(dim, x, used));
                        float gradient = (1.0f - turn - f) * alpha;
                        saxpy(dim, gradient, used, hidden + (size_t)q * dim);
                        saxpy(dim, gradient, x, used);
                    }
                }
                for (int32_t q = 0; q < m; q++)
                    saxpy(dim, 1.0f, hidden + (size_t)q * dim, syn0 + (size_t)d.vid[ctx[q]] * dim);
                pairs += m;
                nodes += (int64_t)m * len;
            }
            if (c.k > 0 && ++since_flush >= p->flush_every) { flush_cache(&c, syn1, dim); since_flush = 0; }
        }
    }
    if (c.k > 0) flush_cache(&c, syn1, dim);
    if (stats) { stats[0] = raw; stats[1] = inv; stats[2] = kept; stats[3] = pairs; stats[4] = nodes; }
    doc_free(&d);
    cache_free(&c);
    free(thr); free(hidden); free(h);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Synchronous mode: every gradient of a batch of sync_batch consecutive      */
/* kept centres is taken against the model as it was at the start of the     */
/* batch; the summed deltas (fp64) are applied once at the end of the batch:  */
/* row = row + (float)delta. Skip-gram, path of the centre word (R1).         */
/* n_batches < 0: the whole stream.                                           */
/* ------------------------------------------------------------------------ */
typedef struct {
    double *d;         /* [rows][dim] deltas */
    uint8_t *touched;  /* [rows] */
    int32_t *list;
    int32_t n;
} delta_t;

static int delta_init(delta_t *a, int32_t rows, int32_t dim) {
    a->d = (double *)calloc((size_t)rows * dim, sizeof(double));
    a->touched = (uint8_t *)calloc((size_t)rows, 1);
    a->list = (int32_t *)malloc(sizeof(int32_t) * (size_t)rows);
    a->n = 0;
    return (a->d && a->touched && a->list) ? 0 : -1;
}
static void delta_free(delta_t *a) { free(a->d); free(a->touched); free(a->list); }
static double *delta_row(delta_t *a, int32_t r, int32_t dim) {
    if (!a->touched[r]) { a->touched[r] = 1; a->list[a->n++] = r; }
    return a->d + (size_t)r * dim;
}
static void delta_apply(delta_t *a, float *w, int32_t dim) {
    for (int32_t i = 0; i < a->n; i++) {
        int32_t r = a->list[i];
        double *dr = a->d + (size_t)r * dim;
        float *wr = w + (size_t)r * dim;
        for (int32_t k = 0; k < dim; k++) { wr[k] = wr[k] + (float)dr[k]; dr[k] = 0.0; }
        a->touched[r] = 0;
    }
    a->n = 0;
}

int or_train_sync(float *syn0, float *syn1, const or_tree *t, const int32_t *tokens, int64_t n,
                  const or_params *p, int64_t n_batches, int64_t *stats) {
    const int32_t dim = p->dim;
    if (p->V < 2 || p->window < 1 || p->window > 1024 || p->doc_len < 1 || p->sync_batch < 1) return -1;
    doc_t d;
    delta_t d0, d1;
    if (doc_alloc(&d, p->doc_len) || delta_init(&d0, p->V, dim) || delta_init(&d1, p->V - 1, dim)) return -1;
    uint64_t *thr = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)p->V);
    if (!thr) return -1;
    or_keep_thresholds(t->vocab_counts, p->V, p->sample, p->train_words, thr);
    int32_t ctx[2 * 1024 + 2];
    int64_t raw = 0, inv = 0, kept = 0, pairs = 0, nodes = 0, in_batch = 0, batches = 0;
    int stop = 0;
    for (int64_t lo = 0; lo < n && !stop; lo += p->doc_len) {
        int64_t hi = lo + p->doc_len < n ? lo + p->doc_len : n;
        raw += hi - lo;
        doc_sample(tokens, n, p, thr, lo, &d, &inv);
        for (int32_t j = 0; j < d.n; j++) {
            if (n_batches >= 0 && batches >= n_batches) { stop = 1; break; }
            int32_t v = d.vid[j];
            float alpha = or_alpha(p->alpha0, d.raw[j], p->epoch, p->n_epochs, p->corpus_tokens);
            int32_t m = window_of(&d, j, ctx);
            int32_t len = t->codelen[v];
            const int32_t *pts = t->points + t->point_off[v];
            uint64_t code = t->code[v];
            for (int32_t q = 0; q < m; q++) {
                int32_t w = d.vid[ctx[q]];
                const float *x = syn0 + (size_t)w * dim;       /* unchanged until the batch ends */
                double *dx = delta_row(&d0, w, dim);
                for (int32_t jn = 0; jn < len; jn++) {
                    int32_t nn = pts[jn];
                    const float *y = syn1 + (size_t)nn * dim;
                    float turn = (float)((code >> jn) & 1u);
                    float f = sigmoidf(sdot(dim, x, y));
                    float gradient = (1.0f - turn - f) * alpha;
                    double *dy = delta_row(&d1, nn, dim);
                    for (int32_t k = 0; k < dim; k++) {
                        dx[k] += (double)gradient * (double)y[k];
                        dy[k] += (double)gradient * (double)x[k];
                    }
                }
                nodes += len;
            }
            pairs += m;
            kept++;
            if (++in_batch == p->sync_batch) {
                delta_apply(&d0, syn0, dim);
                delta_apply(&d1, syn1, dim);
                in_batch = 0;
                batches++;
            }
        }
    }
    delta_apply(&d0, syn0, dim);
    delta_apply(&d1, syn1, dim);
    if (stats) { stats[0] = raw; stats[1] = inv; stats[2] = kept; stats[3] = pairs; stats[4] = nodes; }
    doc_free(&d);
    delta_free(&d0);
    delta_free(&d1);
    free(thr);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Evaluation: log P(v | x) under the hierarchical softmax (R6), fp64.       */
/* ------------------------------------------------------------------------ */
static double log_sigmoid(double u) {
    /* log(1/(1+exp(-u))), evaluated without overflow */
    return u >= 0.0 ? -log1p(exp(-u)) : u - log1p(exp(u));
}

double or_log_prob_f64(const double *x, const double *syn1, int32_t dim, const or_tree *t, int32_t v) {
    double s = 0.0;
    const int32_t *pts = t->points + t->point_off[v];
    for (int32_t j = 0; j < t->codelen[v]; j++) {
        const double *y = syn1 + (size_t)pts[j] * dim;
        double z = 0.0;
        for (int32_t k = 0; k < dim; k++) z += x[k] * y[k];
        double sign = ((t->code[v] >> j) & 1u) ? -1.0 : 1.0;
        s += log_sigmoid(sign * z);
    }
    return s;
}

double or_log_prob(const float *x, const float *syn1, int32_t dim, const or_tree *t, int32_t v) {
    double s = 0.0;
    const int32_t *pts = t->points + t->point_off[v];
    for (int32_t j = 0; j < t->codelen[v]; j++) {
        const float *y = syn1 + (size_t)pts[j] * dim;
        double z = 0.0;
        for (int32_t k = 0; k < dim; k++) z += (double)x[k] * (double)y[k];
        double sign = ((t->code[v] >> j) & 1u) ? -1.0 : 1.0;
        s += log_sigmoid(sign * z);
    }
    return s;
}

/* log P(v | h) for an fp64 input h and fp32 inner-node vectors. */
static double or_log_prob_mixed(const double *h, const float *syn1, int32_t dim, const or_tree *t, int32_t v) {
    double s = 0.0;
    const int32_t *pts = t->points + t->point_off[v];
    for (int32_t j = 0; j < t->codelen[v]; j++) {
        const float *y = syn1 + (size_t)pts[j] * dim;
        double z = 0.0;
        for (int32_t k = 0; k < dim; k++) z += h[k] * (double)y[k];
        double sign = ((t->code[v] >> j) & 1u) ? -1.0 : 1.0;
        s += log_sigmoid(sign * z);
    }
    return s;
}

/*
 * Held-out objective of the sampler's stream, drawn with p's seed, epoch and
 * sampling settings (R11-R13).
 * arch 0 (skip-gram): the sum over pairs (v, w) of log P(v | vector[w]);
 *   n_pairs counts pairs.
 * arch 1 (CBOW): the sum over centres v with at least one window word of
 *   log P(v | h), h = the mean of the window words' vectors (taken in fp64),
 *   the same hierarchical softmax (§2) with CBOW's input; n_pairs counts those
 *   centres.
 * n_nodes: the tree nodes the terms visit.
 */
int or_loglik(const float *syn0, const float *syn1, const or_tree *t, const int32_t *tokens, int64_t n,
              const or_params *p, double *sum_ll, int64_t *n_pairs, int64_t *n_nodes) {
    doc_t d;
    if (doc_alloc(&d, p->doc_len)) return -1;
    uint64_t *thr = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)p->V);
    if (!thr) return -1;
    or_keep_thresholds(t->vocab_counts, p->V, p->sample, p->train_words, thr);
    int32_t ctx[2 * 1024 + 2];
    double *h = (double *)malloc(sizeof(double) * (size_t)p->dim);
    if (!h) return -1;
    int64_t inv = 0, np = 0, nn = 0;
    double s = 0.0;
    for (int64_t lo = 0; lo < n; lo += p->doc_len) {
        doc_sample(tokens, n, p, thr, lo, &d, &inv);
        for (int32_t j = 0; j < d.n; j++) {
            int32_t m = window_of(&d, j, ctx);
            if (p->arch == 1) {
                if (m == 0) continue;
                for (int32_t k = 0; k < p->dim; k++) {
                    double a = 0.0;
                    for (int32_t q = 0; q < m; q++) a += (double)syn0[(size_t)d.vid[ctx[q]] * p->dim + k];
                    h[k] = a / (double)m;
                }
                s += or_log_prob_mixed(h, syn1, p->dim, t, d.vid[j]);
                np++;
                nn += t->codelen[d.vid[j]];
                continue;
            }
            for (int32_t q = 0; q < m; q++) {
                s += or_log_prob(syn0 + (size_t)d.vid[ctx[q]] * p->dim, syn1, p->dim, t, d.vid[j]);
                np++;
                nn += t->codelen[d.vid[j]];
            }
        }
    }
    *sum_ll = s;
    *n_pairs = np;
    if (n_nodes) *n_nodes = nn;
    doc_free(&d);
    free(thr);
    free(h);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Negative sampling: noise table (NS1, NS2), shared negatives (NS3), mini-batch */
/* updates (NS4), objective.                                                   */
/* ------------------------------------------------------------------------ */

/* floor(sqrt(x)) for x < 2^62, by bisection on integers. */
static uint64_t isqrt_u64(uint64_t x) {
    uint64_t lo = 0, hi = (uint64_t)1 << 31;
    while (lo < hi) {           /* largest m with m*m <= x */
        uint64_t mid = (lo + hi + 1) / 2;
        if (mid * mid <= x) lo = mid; else hi = mid - 1;
    }
    return lo;
}

/* weight[v] = isqrt(c * isqrt(c)), c = count of v (NS1); returns the total. */
int64_t or_noise_weights(const int64_t *vocab_counts, int32_t V, int64_t *weight) {
    int64_t tot = 0;
    for (int32_t v = 0; v < V; v++) {
        uint64_t c = (uint64_t)vocab_counts[v];
        weight[v] = (int64_t)isqrt_u64(c * isqrt_u64(c));
        tot += weight[v];
    }
    return tot;
}

/* table[i] = v with Q[v] <= floor(i * Q / 2^L) < Q[v+1] (NS2). Returns -1 on bad input. */
int or_noise_table(const int64_t *vocab_counts, int32_t V, int32_t log2_size, int32_t *table) {
    if (V < 1 || log2_size < 1 || log2_size > 30) return -1;
    int64_t *wt = (int64_t *)malloc(sizeof(int64_t) * (size_t)V);
    if (!wt) return -1;
    int64_t tot = or_noise_weights(vocab_counts, V, wt);
    if (tot <= 0 || tot >= ((int64_t)1 << (63 - log2_size))) { free(wt); return -1; }   /* i * Q < 2^63 */
    int64_t T = (int64_t)1 << log2_size;
    int32_t v = 0;
    int64_t q_hi = wt[0];       /* Q[v+1] */
    for (int64_t i = 0; i < T; i++) {
        int64_t u = (int64_t)(((uint64_t)i * (uint64_t)tot) >> log2_size);
        while (u >= q_hi) { v++; q_hi += wt[v]; }
        table[i] = v;
    }
    free(wt);
    return 0;
}

/* The K shared negatives of the centre at global raw index raw (NS3); -1 where dropped. */
static void draw_negatives(uint64_t seed, int64_t raw, int32_t epoch, int32_t K, const int32_t *table,
                           int32_t log2_size, int32_t centre, int32_t *neg) {
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    for (int32_t h = 0; 4 * h < K; h++) {
        uint32_t ctr[4] = {(uint32_t)raw, (uint32_t)((uint64_t)raw >> 32), (uint32_t)epoch, 1u + (uint32_t)h};
        uint32_t r[4];
        or_philox4x32_10(ctr, key, r);
        for (int32_t i = 0; i < 4 && 4 * h + i < K; i++) {
            int32_t t = table[r[i] >> (32 - log2_size)];
            neg[4 * h + i] = (t == centre) ? -1 : t;
        }
    }
}

/*
 * The negatives of every kept centre in stream order: the first cap centres'
 * K values go to negatives[cap][K] (may be NULL); checksum = sum over all
 * kept centres and k of fmix64(raw * 0x9E3779B97F4A7C15 + k * 2^32 + (neg + 1)).
 * Returns the number of kept centres.
 */
int64_t or_sample_negatives(const int32_t *tokens, int64_t n, const or_params *p, const int64_t *vocab_counts,
                            const int32_t *table, int32_t log2_size, int32_t *negatives, int64_t cap,
                            int64_t *n_kept, uint64_t *checksum) {
    if (p->negative < 1 || p->negative > 64) return -1;
    doc_t d;
    if (doc_alloc(&d, p->doc_len)) return -1;
    uint64_t *thr = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)p->V);
    if (!thr) return -1;
    or_keep_thresholds(vocab_counts, p->V, p->sample, p->train_words, thr);
    int32_t neg[64];
    int64_t nk = 0, inv = 0;
    uint64_t cs = 0;
    for (int64_t lo = 0; lo < n; lo += p->doc_len) {
        doc_sample(tokens, n, p, thr, lo, &d, &inv);
        for (int32_t j = 0; j < d.n; j++) {
            draw_negatives(p->seed, d.raw[j], p->epoch, p->negative, table, log2_size, d.vid[j], neg);
            for (int32_t k = 0; k < p->negative; k++) {
                if (negatives && nk < cap) negatives[nk * p->negative + k] = neg[k];
                cs += fmix64((uint64_t)d.raw[j] * 0x9E3779B97F4A7C15ULL + ((uint64_t)k << 32) +
                             (uint64_t)(int64_t)(neg[k] + 1));
            }
            nk++;
        }
    }
    doc_free(&d);
    free(thr);
    if (n_kept) *n_kept = nk;
    if (checksum) *checksum = cs;
    return nk;
}

/*
 * One epoch of skip-gram with shared negatives, one sequential worker (NS3,
 * NS4). Per kept centre v with window words w_1..w_m and targets
 * t_0 = v (label 1), t_1..t_K its negatives (label 0, dropped ones skipped):
 *   s_qk = vector[w_q] . out[t_k],  g_qk = alpha (label_k - sigmoid(s_qk))
 *   dx_q = sum_k g_qk out[t_k],     dy_k = sum_q g_qk vector[w_q]
 * all from the values at the start of the centre; then vector[w_q] += dx_q
 * (q ascending) and out[t_k] += dy_k (k ascending).
 * stats: [raw, in-vocabulary, kept centres, pairs, pair-target updates].
 */
int or_train_ns(float *syn0, float *syn1, const int64_t *vocab_counts, const int32_t *table, int32_t log2_size,
                const int32_t *tokens, int64_t n, const or_params *p, int64_t *stats) {
    const int32_t dim = p->dim, K = p->negative;
    if (p->V < 2 || p->window < 1 || p->window > 1024 || p->doc_len < 1 || K < 1 || K > 64) return -1;
    doc_t d;
    if (doc_alloc(&d, p->doc_len)) return -1;
    uint64_t *thr = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)p->V);
    int32_t M = 2 * p->window;
    float *dx = (float *)malloc(sizeof(float) * (size_t)dim * M);
    float *dy = (float *)malloc(sizeof(float) * (size_t)dim * (K + 1));
    float *g = (float *)malloc(sizeof(float) * (size_t)M * (K + 1));
    int32_t ctx[2 * 1024 + 2], tgt[65];
    if (!thr || !dx || !dy || !g) return -1;
    or_keep_thresholds(vocab_counts, p->V, p->sample, p->train_words, thr);

    int64_t raw = 0, inv = 0, kept = 0, pairs = 0, updates = 0;
    for (int64_t lo = 0; lo < n; lo += p->doc_len) {
        int64_t hi = lo + p->doc_len < n ? lo + p->doc_len : n;
        raw += hi - lo;
        doc_sample(tokens, n, p, thr, lo, &d, &inv);
        for (int32_t j = 0; j < d.n; j++) {
            if (p->max_centres >= 0 && kept >= p->max_centres) break;
            kept++;
            int32_t m = window_of(&d, j, ctx);
            if (m == 0) continue;
            float alpha = or_alpha(p->alpha0, d.raw[j], p->epoch, p->n_epochs, p->corpus_tokens);
            tgt[0] = d.vid[j];
            draw_negatives(p->seed, d.raw[j], p->epoch, K, table, log2_size, d.vid[j], tgt + 1);
            /* gradients at the snapshot */
            for (int32_t q = 0; q < m; q++) {
                const float *x = syn0 + (size_t)d.vid[ctx[q]] * dim;
                for (int32_t k = 0; k <= K; k++) {
                    if (tgt[k] < 0) { g[q * (K + 1) + k] = 0.0f; continue; }
                    float f = sigmoidf(sdot(dim, x, syn1 + (size_t)tgt[k] * dim));
                    g[q * (K + 1) + k] = ((k == 0 ? 1.0f : 0.0f) - f) * alpha;
                    updates++;
                }
            }
            for (int32_t q = 0; q < m; q++) {
                float *e = dx + (size_t)q * dim;
                memset(e, 0, sizeof(float) * (size_t)dim);
                for (int32_t k = 0; k <= K; k++)
                    if (tgt[k] >= 0) saxpy(dim, g[q * (K + 1) + k], syn1 + (size_t)tgt[k] * dim, e);
            }
            for (int32_t k = 0; k <= K; k++) {
                float *e = dy + (size_t)k * dim;
                memset(e, 0, sizeof(float) * (size_t)dim);
                if (tgt[k] < 0) continue;
                for (int32_t q = 0; q < m; q++)
                    saxpy(dim, g[q * (K + 1) + k], syn0 + (size_t)d.vid[ctx[q]] * dim, e);
            }
            /* apply */
            for (int32_t q = 0; q < m; q++) saxpy(dim, 1.0f, dx + (size_t)q * dim, syn0 + (size_t)d.vid[ctx[q]] * dim);
            for (int32_t k = 0; k <= K; k++)
                if (tgt[k] >= 0) saxpy(dim, 1.0f, dy + (size_t)k * dim, syn1 + (size_t)tgt[k] * dim);
            pairs += m;
        }
    }
    if (stats) { stats[0] = raw; stats[1] = inv; stats[2] = kept; stats[3] = pairs; stats[4] = updates; }
    doc_free(&d);
    free(thr); free(dx); free(dy); free(g);
    return 0;
}

/*
 * Negative-sampling objective over the sampler's pairs (fp64 sums): for pair
 * (v, w) with the centre's negatives n_k (drawn with p's seed and epoch),
 * log sigmoid(x_w . y_v) + sum over kept k of log sigmoid(-x_w . y_{n_k}).
 */
int or_ns_objective(const float *syn0, const float *syn1, const int64_t *vocab_counts, const int32_t *table,
                    int32_t log2_size, const int32_t *tokens, int64_t n, const or_params *p, double *sum,
                    int64_t *n_pairs, int64_t *n_terms) {
    const int32_t dim = p->dim, K = p->negative;
    if (K < 1 || K > 64) return -1;
    doc_t d;
    if (doc_alloc(&d, p->doc_len)) return -1;
    uint64_t *thr = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)p->V);
    if (!thr) return -1;
    or_keep_thresholds(vocab_counts, p->V, p->sample, p->train_words, thr);
    int32_t ctx[2 * 1024 + 2], tgt[65];
    int64_t inv = 0, np = 0, nt = 0;
    double s = 0.0;
    for (int64_t lo = 0; lo < n; lo += p->doc_len) {
        doc_sample(tokens, n, p, thr, lo, &d, &inv);
        for (int32_t j = 0; j < d.n; j++) {
            int32_t m = window_of(&d, j, ctx);
            if (m == 0) continue;
            tgt[0] = d.vid[j];
            draw_negatives(p->seed, d.raw[j], p->epoch, K, table, log2_size, d.vid[j], tgt + 1);
            for (int32_t q = 0; q < m; q++) {
                const float *x = syn0 + (size_t)d.vid[ctx[q]] * dim;
                for (int32_t k = 0; k <= K; k++) {
                    if (tgt[k] < 0) continue;
                    const float *y = syn1 + (size_t)tgt[k] * dim;
                    double z = 0.0;
                    for (int32_t i = 0; i < dim; i++) z += (double)x[i] * (double)y[i];
                    s += log_sigmoid(k == 0 ? z : -z);
                    nt++;
                }
                np++;
            }
        }
    }
    *sum = s;
    *n_pairs = np;
    if (n_terms) *n_terms = nt;
    doc_free(&d);
    free(thr);
    return 0;
}
