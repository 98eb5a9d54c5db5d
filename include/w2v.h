/*
 * w2v.h — C ABI of the MI355X (gfx950) hierarchical-softmax word2vec library.
 *
 * The library trains skip-gram (and CBOW) word vectors against a hierarchical
 * softmax, as in Vuurens, Eickhoff and de Vries, "Efficient Parallel Learning
 * of Word2Vec" (Algorithm 1, Cached Skipgram HS), including the paper's
 * remedy for update collisions: the vectors of the top inner nodes of the
 * Huffman tree are cached per worker and their change is written back
 * periodically (§3.2). On the GPU the cache owner is a workgroup and the
 * cache lives in LDS.
 *
 * Conventions (all entry points):
 *   - Every pointer is a DEVICE pointer unless its name ends in _host.
 *   - The caller owns all memory; the library never allocates device memory.
 *     Scratch space comes in through (workspace, workspace_bytes); each call
 *     has a *_workspace_bytes() query.
 *   - Work is stream-ordered on hip_stream (a hipStream_t; NULL = the null
 *     stream). Calls that write *_host outputs synchronise that stream before
 *     returning; the others return without synchronising.
 *   - Return value: W2V_OK or a negative w2v_status. Arguments are checked
 *     before anything is launched; on W2V_E_ARG / W2V_E_RANGE /
 *     W2V_E_WORKSPACE no output has been touched. On W2V_E_DEVICE outputs are
 *     undefined. w2v_last_error() gives a message for the calling thread.
 *   - Calls on different streams with disjoint buffers may run concurrently;
 *     the only global state is the per-thread error message and a per-device
 *     cache of device properties and timing events.
 */
#ifndef W2V_H
#define W2V_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    W2V_OK = 0,
    W2V_E_ARG = -1,        /* a null pointer, a size out of range, an inconsistent setting */
    W2V_E_RANGE = -2,      /* data out of range: a token id outside [0, id_space), a code longer than 64 */
    W2V_E_WORKSPACE = -3,  /* workspace_bytes below what the *_workspace_bytes query returns */
    W2V_E_DEVICE = -4      /* a HIP runtime error (launch failure, fault surfaced at a synchronisation) */
} w2v_status;

/* Message for the calling thread's last non-OK return ("" if none). */
const char *w2v_last_error(void);

/* ------------------------------------------------------------------------
 * Vocabulary (the "mintf" setting of §4.1; Algorithm 1 iterates over word
 * ids of the text).
 *
 * Counts every id in tokens[0..n_tokens), keeps the ids whose count is at
 * least min_count and orders them by (count descending, id ascending); the
 * position in that order is the vocabulary index 0..V-1.
 *   tokens        int32[n_tokens], ids in [0, id_space)
 *   counts_by_id  int64[id_space]  out: occurrences of each id
 *   vocab_ids     int32[id_space]  out: id of vocabulary index r (r < V); -1 beyond V
 *   vocab_counts  int64[id_space]  out: count of vocabulary index r (r < V); 0 beyond V
 *   id_to_vocab   int32[id_space]  out: vocabulary index of each id, -1 if dropped
 *   tokens_out    int32[n_tokens]  out, may be NULL: tokens mapped to vocabulary
 *                                  indices (-1 = dropped); may not alias tokens
 *   V_host, train_words_host       out: V and the sum of kept counts
 * Errors: W2V_E_RANGE if a token lies outside [0, id_space) (outputs are then
 * written but invalid); W2V_E_ARG if id_space < 1, n_tokens < 0 or
 * min_count < 0. Synchronises the stream.
 * ---------------------------------------------------------------------- */
size_t w2v_build_vocab_workspace_bytes(int32_t id_space);
int w2v_build_vocab(const int32_t *tokens, int64_t n_tokens, int32_t id_space, int64_t min_count,
                    int64_t *counts_by_id, int32_t *vocab_ids, int64_t *vocab_counts, int32_t *id_to_vocab,
                    int32_t *tokens_out, int32_t *V_host, int64_t *train_words_host, void *workspace,
                    size_t workspace_bytes, void *hip_stream);

/* ------------------------------------------------------------------------
 * Huffman tree (§2: the output layer is a binary Huffman tree; a word is
 * predicted by the turns at the inner nodes on its path from the root).
 *
 * Built from vocab_counts[0..V) (descending) by the two-queue merge: leaves in
 * ascending count (vocabulary index V-1 first), inner nodes in creation order;
 * each merge takes the smaller front twice, a leaf winning a count tie; the
 * first child taken gets bit 0; merge a creates inner node a; the root is V-2.
 *   codelen    uint8[V]     out: depth of each word
 *   code       uint64[V]    out: bit j = turn at the j-th inner node from the root
 *   point_off  int32[V+1]   out: word v's inner nodes are points[point_off[v] ..
 *                           point_off[v+1]), root first
 *   points     int32[points_cap] out; NULL = size query (only codelen, code,
 *                           point_off and the host outputs are written)
 *   points_len_host, max_len_host  out: sum of code lengths, longest code
 * Errors: W2V_E_ARG if V < 2, vocab_counts is not in descending order, or
 * points_cap < sum of lengths (points given); W2V_E_RANGE if a code would be
 * longer than 64. Synchronises the stream.
 * ---------------------------------------------------------------------- */
size_t w2v_build_huffman_workspace_bytes(int32_t V);
int w2v_build_huffman(const int64_t *vocab_counts, int32_t V, uint8_t *codelen, uint64_t *code,
                      int32_t *point_off, int32_t *points, int64_t points_cap, int64_t *points_len_host,
                      int32_t *max_len_host, void *workspace, size_t workspace_bytes, void *hip_stream);

/* ------------------------------------------------------------------------
 * Model and training settings.
 *
 * syn0 ("vector[w]" of Algorithm 1) is float[V][row_stride], syn1
 * ("weight[n]", the inner-node vectors) is float[V-1][row_stride]; only the
 * first dim floats of a row are used. row_stride >= dim, a multiple of 4;
 * both arrays 16-byte aligned. Training may write zeros into a row's padding
 * columns (dim .. row_stride-1); their contents are otherwise ignored.
 * ---------------------------------------------------------------------- */
typedef struct {
    float *syn0;
    float *syn1;
    int32_t V, dim, row_stride;
    int32_t reserved0;
    const int64_t *vocab_counts;  /* int64[V] from w2v_build_vocab (keep probabilities) */
    int64_t train_words;          /* sum of vocab_counts (N_t) */
    const uint8_t *codelen;       /* from w2v_build_huffman */
    const uint64_t *code;
    const int32_t *point_off;
    const int32_t *points;
} w2v_model;

typedef struct {
    int32_t arch;            /* 0 = skip-gram (Algorithm 1), 1 = CBOW (mean of the window as input),
                                2 = skip-gram with the reversed orientation: for each window word w in order
                                the path of w is walked with the centre's vector as input, which gains that
                                pair's hidden-layer gradient before the next pair (asynchronous mode only) */
    int32_t mode;            /* 0 = asynchronous (lock-free, top-k cache in LDS), 1 = synchronous batches
                                (skip-gram, arch 0, only) */
    int32_t window;          /* W ("windowsize", §4.1), 1..10; effective half-width uniform on 1..W */
    int32_t doc_len;         /* documents of doc_len raw tokens (1..65535); windows never cross them */
    double sample;           /* subsampling threshold t ("downsample", §4.1); 0 = keep all */
    float alpha0;            /* initial learning rate */
    int32_t epoch, n_epochs; /* this epoch and the total, for the learning-rate schedule */
    int32_t reserved1;
    int64_t corpus_tokens;   /* raw tokens of one epoch (the whole corpus, for the schedule) */
    int64_t first_raw_index; /* global raw index of tokens[0]; a multiple of doc_len */
    uint64_t seed;           /* Philox4x32-10 key for subsampling and window draws */
    int32_t cache_k;         /* inner nodes cached per workgroup ("isFrequent"): the k created last */
    int32_t flush_every;     /* write the cache back after this many centre words per workgroup (>= 1) */
    int32_t sync_batch;      /* synchronous mode: kept centres per batch (>= 1) */
    int32_t workers;         /* wavefronts that take documents; 0 = fill the GPU; 1 = one sequential worker */
    int32_t write_policy;    /* bit 0: uncached inner-node rows are stored (lock-free, concurrent updates may be
                                overwritten, as in Hogwild) instead of atomically adding their change;
                                bit 1: the same for the word vectors syn0 (a word repeated within a window
                                stores at its first position and adds the change of the others);
                                bit 2: the same for the cached rows in the workgroup's LDS copy;
                                bit 3 (needs bit 1): word rows kept across centres -- a wavefront
                                holds the rows of the kept words within `window` positions of its centre in
                                registers while it walks a document's centres in order, loading a row when it
                                enters that span and storing it when it leaves or becomes the centre (one read
                                and write per word and span instead of one per pair). Applies to rows of 129 to
                                512 floats with window <= 5: CBOW always, skip-gram on the store-only walk
                                (bit 0; bit 2 when cache_k > 0; hot_k 0; cache_mode 0) and with window <= 2
                                above 320 floats; elsewhere the bit is ignored; w2v_train_word_span reports
                                which */
    int32_t flush_policy;    /* cache write-back: 0 = add the change (cached - original), the write-back of
                                §3.2 as printed (stable at a few hundred wavefronts; at full occupancy the
                                top rows' summed stale changes diverge); 1 = add the change divided by the
                                number of workgroups, so that their progress on the cached rows is averaged
                                (local SGD on those rows) -- a departure from §3.2, and the default */
    int32_t hot_k;           /* with write_policy bit 0: the hot_k inner nodes created just before the cached
                                ones (on most paths, so the most contended rows) still take atomic adds of
                                their change; >= 0 */
    int32_t negative;        /* negative sampling (w2v_train_ns_epoch, w2v_ns_objective): negatives per centre,
                                shared by its window words; 1..11 (1..7 above 320 columns); ignored elsewhere */
    int32_t cache_mode;      /* asynchronous mode's cache: 0 = each workgroup holds a copy of the cached rows and
                                their values at the last write-back, whose difference it writes back (§3.2);
                                1 = delta-only: it holds just its change since the last write-back, reads a
                                cached row as the HBM row plus that change and adds its updates to the change
                                with LDS atomics (write_policy bit 2 does not apply); half the LDS per row */
    int32_t span_refresh;    /* with write_policy bit 3 in effect: the words of vocabulary index below this
                                (the most frequent) are written back, if changed, and read again after every
                                centre while they stay in the span, so that other wavefronts' updates to them
                                are lost for one centre at most, as without bit 3; 0 = off; >= 0 */
    int32_t span_stash;      /* with write_policy bit 3 in effect: 1 = the row of the word that
                                becomes the next centre waits in a per-wavefront LDS row while that word is the
                                centre, and re-enters the span from there instead of from memory (one row read
                                less per centre when the row fits beside the cache), so other wavefronts'
                                updates to it during that centre are lost when it is stored again (for the
                                frequent words, with many wavefronts, this lowers the held-out log-likelihood
                                and widens its run-to-run spread: see stash_from); 0 = off (the default) or 1 */
    int32_t stash_from;      /* with span_stash 1: only words of vocabulary index >= stash_from (the less
                                frequent ones, whose rows few other wavefronts update meanwhile) re-enter from
                                the stash; the more frequent ones are read again from memory (10000 at V = 1M
                                keeps the log-likelihood of the run without the stash); >= 0 */
} w2v_params;

/* stats int64[5]: raw tokens, in-vocabulary tokens, kept centre words, (centre, context) pairs,
   node updates (pair-node updates for skip-gram, centre-node updates for CBOW). */
#define W2V_N_STATS 5

/* ------------------------------------------------------------------------
 * One training pass over tokens[0..n_tokens) (vocabulary indices, -1 =
 * dropped), updating m->syn0 and m->syn1 in place.
 *
 * Per kept centre word v (subsampling: keep with probability
 * min(1, sqrt(q) + q), q = t N_t / count(v), drawn from Philox4x32-10 keyed
 * by (seed; raw index, epoch)), with window words w_1..w_P (the kept words of
 * the same document within the effective half-width), the path of v is
 * walked once; at each inner node n with turn t and every window word in
 * order: f = sigmoid(syn0[w].syn1[n]), g = (1 - t - f) alpha, the
 * hidden-layer gradient of w gains g syn1[n] and syn1[n] gains g syn0[w];
 * afterwards each syn0[w] gains its hidden-layer gradient (Algorithm 1 with
 * the window and node loops swapped, which is the same computation whenever
 * a window holds no repeated word). alpha decays linearly with the raw stream
 * position in steps of 10,000 tokens down to 1e-4 alpha0.
 *
 * mode 0: segments of up to 128 kept centres of a document are claimed by
 * wavefronts from a queue (in stream order); the top cache_k
 * inner-node vectors live in each workgroup's LDS and are written back as a
 * change (cached - original) every flush_every centres (§3.2); other rows are
 * updated in HBM, by atomic adds of their change or, as write_policy selects,
 * by stores of the new row. Lock-free: results vary with scheduling, as in
 * the paper's Hogwild setting, except with workers=1.
 * mode 1: every gradient of a batch of sync_batch consecutive kept centres
 * uses the model at the start of the batch; the sums (exact int64 fixed
 * point, 40 fraction bits) are applied at its end. Deterministic. A row's
 * change within one batch must stay below 2^23 in magnitude (the fixed
 * point's range); a batch that large has diverged (e.g. batches of hundreds
 * of centres over a vocabulary of a few dozen words). Synchronises the
 * stream once (to read the number of kept centres).
 * stats: int64[W2V_N_STATS] device buffer, overwritten (may be NULL).
 * Errors: W2V_E_ARG for a bad model/params (V < 2, dim not in 1..1024,
 * window not in 1..10, cache_mode not 0 or 1, LDS budget exceeded: 2 cache_k
 * rows (1 with the delta-only cache) of 4-byte floats,
 * a row being dim rounded up to 64, 128, 256, 320 or 512 for dim <= 512 and
 * dim above, plus, for dim <= 512, 2 KiB of centre records per wavefront of
 * a workgroup (16 wavefronts for dim <= 64, 12 for dim <= 320, 8 above), ...).
 * ---------------------------------------------------------------------- */
size_t w2v_train_workspace_bytes(const w2v_model *m, int64_t n_tokens, const w2v_params *p);
int w2v_train_hs_epoch(const w2v_model *m, const int32_t *tokens, int64_t n_tokens, const w2v_params *p,
                       int64_t *stats, void *workspace, size_t workspace_bytes, void *hip_stream);

/* Half-width of the word-row span that w2v_train_hs_epoch keeps in registers
   for these arguments (write_policy bit 3): the rows of the kept words within
   that many positions of the centre stay in registers across centres; 0 when
   every centre reads and writes its window rows itself. Host-side, no launch;
   returns -1 for a NULL pointer or an invalid model or parameter block
   (w2v_last_error says which). */
int32_t w2v_train_word_span(const w2v_model *m, const w2v_params *p);

/* Duration in milliseconds of the main training kernel of the last
   w2v_train_hs_epoch call on the calling thread's current device (HIP events
   recorded on that call's stream). Waits for that kernel to finish. */
int w2v_last_train_kernel_ms(float *ms_host);

/* Launch shape of the main training kernel of the last asynchronous
   w2v_train_hs_epoch call on the calling thread's current device: workgroups
   (cache owners) and wavefronts that took documents. Host-side, no wait. */
int w2v_last_train_launch(int32_t *workgroups_host, int32_t *wavefronts_host);

/* Resources of that same launch (the last asynchronous hierarchical-softmax
   or negative-sampling training kernel on the calling thread's current
   device): LDS bytes per workgroup (static centre records plus the dynamic
   cache rows), vector registers per lane as the HIP runtime reports them,
   and resident wavefronts per SIMD at that LDS size (occupancy). All three
   are 0 before the first launch. Host-side, no wait. Errors: W2V_E_ARG for a
   NULL pointer. */
int w2v_last_train_resources(int32_t *lds_bytes_host, int32_t *vgprs_host, int32_t *waves_per_simd_host);

/* ------------------------------------------------------------------------
 * Hierarchical-softmax log-likelihood (evaluation, §2's objective): over the
 * (centre, context) pairs that the sampler draws from tokens with p's seed,
 * epoch, window and sample settings, sum_ll = sum of log P(v | syn0[w]) with
 * P(v|x) = prod_j sigmoid((1 - 2 t_j) x . syn1[n_j]) over v's path, and
 * n_pairs = the number of pairs (p->arch 0 or 2).
 * p->arch 1 (CBOW): the same softmax with CBOW's input, one term per sampled
 * centre v that has at least one window word: sum_ll = sum of log P(v | h),
 * h = the mean of the window words' syn0 rows; n_pairs = the number of such
 * centres. n_nodes (may be NULL): the path nodes the terms visit.
 * Skip-gram: dot products in fp32; CBOW: h and its dot products in fp64;
 * logarithms and sums in fp64, summed in a fixed order (deterministic).
 * Read-only on the model. Synchronises the stream. Errors: W2V_E_ARG for a
 * bad model, params (arch outside 0..2) or NULL required pointer,
 * W2V_E_WORKSPACE for a short workspace, W2V_E_DEVICE for a HIP failure.
 * ---------------------------------------------------------------------- */
size_t w2v_hs_loglik_workspace_bytes(const w2v_model *m, int64_t n_tokens, const w2v_params *p);
int w2v_hs_loglik(const w2v_model *m, const int32_t *tokens, int64_t n_tokens, const w2v_params *p,
                  double *sum_ll_host, int64_t *n_pairs_host, int64_t *n_nodes_host, void *workspace,
                  size_t workspace_bytes, void *hip_stream);

/* ------------------------------------------------------------------------
 * w2v_hs_loglik on the library's own scratch memory, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Same arguments, results and errors as
 * w2v_hs_loglik without the workspace: the workspace is a static device
 * array of w2v_noalloc_scratch_bytes() bytes (64 MiB) that every GPU the
 * library runs on holds until the process ends. The call itself allocates
 * nothing; its first call on a device looks up that device's copy of the
 * array. Evaluations whose w2v_hs_loglik_workspace_bytes exceed the scratch
 * return W2V_E_RANGE before anything is launched (about 11 bytes per token
 * with 1,000-token documents, plus 8 bytes per vocabulary word: e.g. V = 1M
 * with up to about 5.3M tokens). Every call on a device shares that device's
 * scratch, which keeps the last call's contents: calls that overlap on one
 * device (other streams or threads) race on it and must not be issued
 * concurrently. Synchronises the stream.
 * ---------------------------------------------------------------------- */
size_t w2v_noalloc_scratch_bytes(void);
int w2v_hs_loglik_noalloc(const w2v_model *m, const int32_t *tokens, int64_t n_tokens, const w2v_params *p,
                          double *sum_ll_host, int64_t *n_pairs_host, int64_t *n_nodes_host, void *hip_stream);

/* ------------------------------------------------------------------------
 * Negative sampling: the alternative objective to the hierarchical softmax
 * that §2 names, trained in the mini-batch form of Ji et al. that the opening
 * of §3.2 describes (every window word of a centre trains against the same
 * targets, all gradients of the centre taken before any of its updates).
 * For these calls m->syn1 holds the output vectors of the words,
 * float[V][row_stride]; the Huffman arrays of m are not used (may be NULL).
 *
 * w2v_build_noise_table: the noise distribution, unigram counts raised to
 * 3/4, with the weight of count c taken in integers as isqrt(c * isqrt(c)),
 * laid out in table int32[2^log2_size]: entry i holds the vocabulary index
 * v with Q[v] <= floor(i Q / 2^log2_size) < Q[v+1] (Q[v] = weight of the
 * indices below v, Q = total). log2_size in 1..30; total_weight_host gets Q.
 * Errors: W2V_E_ARG for bad sizes or NULL pointers; W2V_E_RANGE if Q is not
 * in [1, 2^(63 - log2_size)). Synchronises the stream.
 * ---------------------------------------------------------------------- */
size_t w2v_noise_table_workspace_bytes(int32_t V);
int w2v_build_noise_table(const int64_t *vocab_counts, int32_t V, int32_t log2_size, int32_t *table,
                          int64_t *total_weight_host, void *workspace, size_t workspace_bytes, void *hip_stream);

/* ------------------------------------------------------------------------
 * One pass of skip-gram with shared negatives over tokens (vocabulary
 * indices, -1 = dropped): the same subsampling, documents, window draws and
 * learning-rate schedule as w2v_train_hs_epoch. Per kept centre v with
 * window words w_1..w_P, its targets are v (label 1) and p->negative
 * negatives (label 0): negative 4h+i is table[r_i >> (32 - log2_size)], r =
 * Philox4x32-10(counter (raw index lo, raw index hi, epoch, 1 + h), key =
 * seed); one equal to v is dropped. With S_qk = syn0[w_q] . syn1[t_k] and
 * g_qk = alpha (label_k - sigmoid(S_qk)), syn0[w_q] gains sum_k g_qk
 * syn1[t_k] and syn1[t_k] gains sum_q g_qk syn0[w_q], all from the values
 * before the centre. Write-back (p->write_policy): bit 0 set, a target row is
 * stored as its value before the centre plus its change (lock-free, as in
 * Hogwild: concurrent changes can be overwritten); bit 1 set, a word row is
 * re-read and stored with its change; otherwise, and for a word or negative
 * repeated within the centre, the change is added atomically. Centres run
 * concurrently, so results vary with scheduling except with workers = 1. stats int64[W2V_N_STATS]: raw tokens, in-vocabulary tokens,
 * kept centres, pairs, pair-target updates. Asynchronous (mode 0) skip-gram
 * only; dim <= 512. Errors as w2v_train_hs_epoch, and W2V_E_ARG for a NULL
 * table, log2_size outside 1..30 or negative out of range.
 * ---------------------------------------------------------------------- */
size_t w2v_train_ns_workspace_bytes(const w2v_model *m, int64_t n_tokens, const w2v_params *p);
int w2v_train_ns_epoch(const w2v_model *m, const int32_t *noise_table, int32_t log2_size, const int32_t *tokens,
                       int64_t n_tokens, const w2v_params *p, int64_t *stats, void *workspace, size_t workspace_bytes,
                       void *hip_stream);

/* Negative-sampling objective (evaluation) over the sampler's pairs drawn
   with p's seed and epoch, each pair with its centre's negatives: sum_host =
   sum over pairs (v, w) of log sigmoid(syn0[w] . syn1[v]) + sum over kept
   negatives n of log sigmoid(-syn0[w] . syn1[n]). Dot products in fp32, logs
   and sums in fp64, in a fixed order (deterministic). n_terms_host (may be
   NULL) = number of log-sigmoid terms. Read-only. Synchronises the stream. */
size_t w2v_ns_objective_workspace_bytes(const w2v_model *m, int64_t n_tokens, const w2v_params *p);
int w2v_ns_objective(const w2v_model *m, const int32_t *noise_table, int32_t log2_size, const int32_t *tokens,
                     int64_t n_tokens, const w2v_params *p, double *sum_host, int64_t *n_pairs_host,
                     int64_t *n_terms_host, void *workspace, size_t workspace_bytes, void *hip_stream);

/* ------------------------------------------------------------------------
 * Test hooks (not part of the training contract).
 *
 * w2v_sample_pairs: the (centre, context) pairs of the sampler in stream
 * order (documents, then centres, then window positions ascending), as global
 * raw indices; the first pair_cap are written (centre_raw/context_raw may be
 * NULL); keep_mask uint8[n_tokens] (may be NULL) marks kept centres;
 * checksum_host = sum over all pairs of fmix64(centre * 0x9E3779B97F4A7C15 +
 * context) mod 2^64 (MurmurHash3 finaliser). Synchronises the stream.
 *
 * w2v_keep_thresholds: thr[v] = 2^32 if the keep probability is >= 1, else
 * floor(p_keep 2^32); a token is kept iff its first Philox word < thr.
 *
 * w2v_sample_negatives: the p->negative negatives of every kept centre in
 * stream order (-1 where dropped), the first negatives_cap centres written to
 * negatives int32[cap][negative] (may be NULL); checksum_host = sum over kept
 * centres and k of fmix64(raw * 0x9E3779B97F4A7C15 + k * 2^32 + (negative + 1))
 * mod 2^64. Synchronises the stream.
 * ---------------------------------------------------------------------- */
size_t w2v_sample_pairs_workspace_bytes(int32_t V, int64_t n_tokens, const w2v_params *p);
int w2v_sample_pairs(const int32_t *tokens, int64_t n_tokens, int32_t V, const int64_t *vocab_counts,
                     int64_t train_words, const w2v_params *p, int64_t *centre_raw, int64_t *context_raw,
                     int64_t pair_cap, uint8_t *keep_mask, int64_t *n_pairs_host, int64_t *n_kept_host,
                     uint64_t *checksum_host, void *workspace, size_t workspace_bytes, void *hip_stream);
int w2v_keep_thresholds(const int64_t *vocab_counts, int32_t V, double sample, int64_t train_words, uint64_t *thr,
                        void *hip_stream);
size_t w2v_sample_negatives_workspace_bytes(int32_t V, int64_t n_tokens, const w2v_params *p);
int w2v_sample_negatives(const int32_t *tokens, int64_t n_tokens, int32_t V, const int64_t *vocab_counts,
                         int64_t train_words, const w2v_params *p, const int32_t *noise_table, int32_t log2_size,
                         int32_t *negatives, int64_t negatives_cap, int64_t *n_kept_host, uint64_t *checksum_host,
                         void *workspace, size_t workspace_bytes, void *hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* W2V_H */
