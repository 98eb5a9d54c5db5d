/*
 * CPU oracle for hierarchical-softmax word2vec (Vuurens, Eickhoff, de Vries,
 * "Efficient Parallel Learning of Word2Vec", ICML 2016 workshop).
 *
 * TEST INFRASTRUCTURE ONLY. This is a plain, slow, single-threaded C
 * implementation written from the paper; it exists to check the GPU library.
 * Only tests, the smoke check and the benchmark's CPU-baseline leg may load
 * it. It shares no source with the GPU library.
 *
 * Model state is fp32, as in the paper, whose implementation works through
 * single-precision level-1 BLAS (scopy/sdot/saxpy, §3.2). Evaluation sums
 * (log-likelihood, synchronous-mode deltas) are fp64.
 *
 * Arrays are dense row-major: syn0 = vector[V][dim] (input word vectors),
 * syn1 = weight[V-1][dim] (inner-node vectors of the Huffman tree).
 */
#ifndef W2V_ORACLE_H
#define W2V_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- vocabulary ---- */
int64_t or_count(const int32_t *tokens, int64_t n, int32_t id_space, int64_t *counts);
int32_t or_vocab(const int64_t *counts, int32_t id_space, int64_t min_count, int32_t *vocab_ids,
                 int64_t *vocab_counts, int32_t *id_to_vocab, int64_t *train_words);
void or_remap(const int32_t *tokens, int64_t n, const int32_t *id_to_vocab, int32_t *out);

/* ---- Huffman tree ---- */
int or_huffman(const int64_t *vocab_counts, int32_t V, int32_t *parent, uint8_t *bit, int64_t *node_count);
int or_huffman_codes(const int32_t *parent, const uint8_t *bit, int32_t V, uint8_t *codelen, uint64_t *code,
                     int32_t *point_off, int32_t *points, int64_t points_cap);

/* ---- counter-based RNG ---- */
void or_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* ---- sampling tables ---- */
void or_keep_thresholds(const int64_t *vocab_counts, int32_t V, double sample, int64_t train_words,
                        uint64_t *thr);
float or_alpha(float alpha0, int64_t raw_pos, int32_t epoch, int32_t n_epochs, int64_t corpus_tokens);

typedef struct {
    int32_t V, dim;
    int32_t window, doc_len;
    double sample;
    float alpha0;
    int32_t epoch, n_epochs;
    int64_t train_words;      /* N_t: sum of in-vocabulary counts (for the keep probability) */
    int64_t corpus_tokens;    /* N_raw of one epoch (for the learning-rate schedule) */
    int64_t first_raw_index;  /* global raw index of tokens[0]; a multiple of doc_len */
    uint64_t seed;
    int32_t cache_k;          /* number of top inner nodes cached (0 = none) */
    int32_t flush_every;      /* flush the cache after this many centre words */
    int32_t order;            /* 0 = as printed (pair-major), 1 = centre-major interchange */
    int32_t orient;           /* 0 = path of the centre word v, input vector[w]; 1 = reverse */
    int32_t arch;             /* 0 = skip-gram, 1 = CBOW */
    int32_t sync_batch;       /* synchronous mode: centres per batch */
    int64_t max_centres;      /* stop after this many kept centres (-1 = all) */
    int32_t negative;         /* negative sampling: negatives shared by a centre's window (NS3) */
    int32_t reserved;
} or_params;

typedef struct {
    const int64_t *vocab_counts; /* [V], descending (for the keep thresholds) */
    const uint8_t *codelen;
    const uint64_t *code;
    const int32_t *point_off;
    const int32_t *points;
} or_tree;

/* ---- sampler: (centre, context) pairs in stream order ---- */
int64_t or_sample_pairs(const int32_t *tokens, int64_t n, const or_params *p, const int64_t *vocab_counts,
                        int64_t *centre_raw, int64_t *context_raw, int64_t cap, uint8_t *keep_mask,
                        int64_t *n_kept, uint64_t *checksum);

/* ---- training ---- */
int or_train(float *syn0, float *syn1, const or_tree *t, const int32_t *tokens, int64_t n, const or_params *p,
             int64_t *stats);
int or_train_sync(float *syn0, float *syn1, const or_tree *t, const int32_t *tokens, int64_t n,
                  const or_params *p, int64_t n_batches, int64_t *stats);

/* ---- evaluation ---- */
double or_log_prob(const float *x, const float *syn1, int32_t dim, const or_tree *t, int32_t v);
double or_log_prob_f64(const double *x, const double *syn1, int32_t dim, const or_tree *t, int32_t v);
/* p->arch 0: sum of log P(v | vector[w]) over the sampled pairs; p->arch 1 (CBOW): sum of log P(v | h)
   over the sampled centres with a window, h = the mean of the window vectors. n_pairs counts the terms. */
int or_loglik(const float *syn0, const float *syn1, const or_tree *t, const int32_t *tokens, int64_t n,
              const or_params *p, double *sum_ll, int64_t *n_pairs, int64_t *n_nodes);

/* ---- negative sampling (the alternative objective named in §2; Ji et al.'s shared-negative
        mini-batch, §3.2): syn1 is then the [V][dim] output vectors of the words ---- */
int64_t or_noise_weights(const int64_t *vocab_counts, int32_t V, int64_t *weight);
int or_noise_table(const int64_t *vocab_counts, int32_t V, int32_t log2_size, int32_t *table);
int64_t or_sample_negatives(const int32_t *tokens, int64_t n, const or_params *p, const int64_t *vocab_counts,
                            const int32_t *table, int32_t log2_size, int32_t *negatives, int64_t cap,
                            int64_t *n_kept, uint64_t *checksum);
int or_train_ns(float *syn0, float *syn1, const int64_t *vocab_counts, const int32_t *table, int32_t log2_size,
                const int32_t *tokens, int64_t n, const or_params *p, int64_t *stats);
int or_ns_objective(const float *syn0, const float *syn1, const int64_t *vocab_counts, const int32_t *table,
                    int32_t log2_size, const int32_t *tokens, int64_t n, const or_params *p, double *sum,
                    int64_t *n_pairs, int64_t *n_terms);

#ifdef __cplusplus
}
#endif
#endif
