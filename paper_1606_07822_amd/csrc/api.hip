// C ABI entry points: argument checks, workspace carving, launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <string>

#include "w2v_internal.h"

namespace w2v {

// defined in the kernel translation units
size_t vocab_workspace_bytes(int32_t id_space);
int run_build_vocab(const int32_t *, int64_t, int32_t, int64_t, int64_t *, int32_t *, int64_t *, int32_t *, int32_t *,
                    int32_t *, int64_t *, void *, hipStream_t);
size_t huffman_workspace_bytes(int32_t V);
int run_build_huffman(const int64_t *, int32_t, uint8_t *, uint64_t *, int32_t *, int32_t *, int64_t, int64_t *,
                      int32_t *, void *, hipStream_t);
size_t pairs_workspace_bytes(int32_t V, int64_t n_tokens, int32_t doc_len);
int run_sample_pairs(const int32_t *, int64_t, int32_t, const int64_t *, int64_t, const w2v_params *, int64_t *,
                     int64_t *, int64_t, uint8_t *, int64_t *, int64_t *, uint64_t *, void *, hipStream_t);
size_t train_lds_bytes(int32_t cache_k, int32_t dim, bool delta);
int train_launch_shape(int arch, int dim, int cache_k, bool delta, bool buf, int workers, int64_t n_units, int *grid,
                       int *waves,
                       bool slide = false, bool stash = false);
int64_t train_egrad_floats(int arch, int dim, bool buf, int stride, int window, int waves);
int train_word_span(int arch, int dim, bool buf, int write_policy, int window);
int launch_train_async(TrainArgs a, int arch, int window, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s,
                       int64_t *stats_out, const int64_t *totals);
size_t sync_extra_bytes(int32_t V, int32_t dim, int64_t n_docs);
int run_train_sync(const w2v_model *m, const w2v_params *p, const SampleBufs &b, int64_t n_tokens, Carve &c,
                   const float *alpha_tab, int64_t blk0, unsigned long long *tstats, hipStream_t s);
size_t noise_workspace_bytes(int32_t V);
int run_noise_table(const int64_t *vocab_counts, int32_t V, int32_t log2_size, int32_t *table, int64_t *total_host,
                    void *workspace, hipStream_t s);
size_t ns_train_extra_bytes();
int launch_train_ns(const w2v_model *m, const int32_t *table, int32_t log2_size, const w2v_params *p,
                    const SampleBufs &b, int64_t n_tokens, const float *alpha_tab, int64_t blk0, Carve &c,
                    hipEvent_t ev0, hipEvent_t ev1, int64_t *stats, hipStream_t s);
size_t ns_objective_extra_bytes(int64_t n_docs, int32_t doc_len);
int run_ns_objective(const w2v_model *m, const int32_t *table, int32_t log2_size, const w2v_params *p,
                     const SampleBufs &b, int64_t n_tokens, Carve &c, double *sum_host, int64_t *n_pairs_host,
                     int64_t *n_terms_host, hipStream_t s);
size_t ns_negatives_extra_bytes(int64_t n_docs);
int run_ns_negatives(const w2v_params *p, const int32_t *table, int32_t log2_size, const SampleBufs &b,
                     int64_t n_tokens, Carve &c, int32_t *out, int64_t cap, int64_t *n_kept_host,
                     uint64_t *checksum_host, hipStream_t s);
int64_t loglik_units(int64_t n_tokens, int32_t doc_len);
size_t loglik_extra_bytes(int64_t n_units);
int run_loglik(const w2v_model *m, const w2v_params *p, const SampleBufs &b, int64_t n_tokens, Carve &c,
               double *sum_ll_host, int64_t *n_pairs_host, int64_t *n_nodes_host, hipStream_t s);

// ---------------------------------------------------------------- errors
static thread_local std::string g_err;
void set_error(const std::string &msg) { g_err = msg; }
int fail(int code, const std::string &msg) {
    g_err = msg;
    return code;
}
int hip_fail(hipError_t e, const char *what) {
    g_err = std::string(what) + ": " + hipGetErrorName(e) + " (" + hipGetErrorString(e) + ")";
    return W2V_E_DEVICE;
}

// ------------------------------------------------------- device properties
struct DevInfo {
    int cus = 0;
    size_t lds = 0;
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
    bool have_timing = false;
    int last_groups = 0, last_waves = 0;
    int last_lds = 0, last_vgprs = 0, last_waves_per_simd = 0;
};
std::mutex g_mu;
DevInfo g_dev[64];

DevInfo &dev_info() {
    int d = 0;
    (void)hipGetDevice(&d);
    if (d < 0 || d >= 64) d = 0;
    std::lock_guard<std::mutex> lk(g_mu);
    DevInfo &di = g_dev[d];
    if (di.cus == 0) {
        hipDeviceProp_t prop;
        if (hipGetDeviceProperties(&prop, d) == hipSuccess) {
            di.cus = prop.multiProcessorCount;
            di.lds = prop.maxSharedMemoryPerMultiProcessor ? prop.maxSharedMemoryPerMultiProcessor
                                                           : prop.sharedMemPerBlock;
        } else {
            di.cus = 256;
            di.lds = 160 * 1024;
        }
    }
    return di;
}

int device_cu_count() { return dev_info().cus; }
void record_train_launch(int groups, int waves, const void *fn, int block, size_t dyn_lds) {
    hipFuncAttributes fa{};
    int lds = 0, vgprs = 0, per_cu = 0;
    if (hipFuncGetAttributes(&fa, fn) == hipSuccess) {
        lds = static_cast<int>(fa.sharedSizeBytes + dyn_lds);
        vgprs = fa.numRegs;
    }
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, block, dyn_lds) != hipSuccess) per_cu = 0;
    DevInfo &di = dev_info();
    std::lock_guard<std::mutex> lk(g_mu);
    di.last_groups = groups;
    di.last_waves = waves;
    di.last_lds = lds;
    di.last_vgprs = vgprs;
    di.last_waves_per_simd = per_cu * (block / kWave) / 4;   // 4 SIMDs per compute unit
}
size_t device_max_lds() { return dev_info().lds; }

}  // namespace w2v

using namespace w2v;

namespace {

hipStream_t as_stream(void *s) { return static_cast<hipStream_t>(s); }

int check_ws(void *ws, size_t have, size_t need) {
    if (have < need)
        return fail(W2V_E_WORKSPACE, "workspace_bytes " + std::to_string(have) + " < required " + std::to_string(need));
    if (need > 0 && !ws) return fail(W2V_E_ARG, "workspace is NULL");
    return W2V_OK;
}

int check_params(const w2v_params *p, bool training) {
    if (!p) return fail(W2V_E_ARG, "params is NULL");
    if (p->window < 1 || p->window > 10) return fail(W2V_E_ARG, "window must be in 1..10");
    if (p->doc_len < 1 || p->doc_len > 65535) return fail(W2V_E_ARG, "doc_len must be in 1..65535");
    if (!(p->sample >= 0.0) || p->sample >= 1.0) return fail(W2V_E_ARG, "sample must be in [0, 1)");
    if (p->first_raw_index < 0 || p->first_raw_index % p->doc_len != 0)
        return fail(W2V_E_ARG, "first_raw_index must be a non-negative multiple of doc_len");
    if (training) {
        if (p->arch < 0 || p->arch > 2)
            return fail(W2V_E_ARG, "arch must be 0 (skip-gram), 1 (CBOW) or 2 (skip-gram, reversed orientation)");
        if (p->mode != 0 && p->mode != 1) return fail(W2V_E_ARG, "mode must be 0 (async) or 1 (sync)");
        if (p->mode == 1 && p->arch != 0) return fail(W2V_E_ARG, "synchronous mode is skip-gram only");
        if (p->n_epochs < 1 || p->epoch < 0 || p->epoch >= p->n_epochs)
            return fail(W2V_E_ARG, "need 0 <= epoch < n_epochs");
        if (p->corpus_tokens < 1) return fail(W2V_E_ARG, "corpus_tokens must be >= 1");
        if (!(p->alpha0 > 0.0f)) return fail(W2V_E_ARG, "alpha0 must be > 0");
        if (p->cache_k < 0) return fail(W2V_E_ARG, "cache_k must be >= 0");
        if (p->flush_every < 1) return fail(W2V_E_ARG, "flush_every must be >= 1");
        if (p->mode == 1 && p->sync_batch < 1) return fail(W2V_E_ARG, "sync_batch must be >= 1");
        if (p->workers < 0) return fail(W2V_E_ARG, "workers must be >= 0");
        if (p->write_policy < 0 || p->write_policy > 15) return fail(W2V_E_ARG, "write_policy must be in 0..15");
        if ((p->write_policy & 8) && !(p->write_policy & 2))
            return fail(W2V_E_ARG, "write_policy bit 3 (word rows kept across centres) needs bit 1 (word rows stored)");
        if (p->flush_policy != 0 && p->flush_policy != 1) return fail(W2V_E_ARG, "flush_policy must be 0 or 1");
        if (p->cache_mode != 0 && p->cache_mode != 1) return fail(W2V_E_ARG, "cache_mode must be 0 or 1");
        if (p->hot_k < 0) return fail(W2V_E_ARG, "hot_k must be >= 0");
        if (p->span_refresh < 0) return fail(W2V_E_ARG, "span_refresh must be >= 0");
        if (p->span_stash != 0 && p->span_stash != 1) return fail(W2V_E_ARG, "span_stash must be 0 or 1");
        if (p->stash_from < 0) return fail(W2V_E_ARG, "stash_from must be >= 0");
    }
    return W2V_OK;
}

int check_model(const w2v_model *m, bool need_tree) {
    if (!m) return fail(W2V_E_ARG, "model is NULL");
    if (m->V < 2) return fail(W2V_E_ARG, "V must be >= 2");
    if (m->dim < 1 || m->dim > 1024) return fail(W2V_E_ARG, "dim must be in 1..1024");
    if (m->row_stride < m->dim || m->row_stride % 4 != 0)
        return fail(W2V_E_ARG, "row_stride must be >= dim and a multiple of 4");
    if (!m->syn0 || !m->syn1) return fail(W2V_E_ARG, "syn0/syn1 is NULL");
    if ((reinterpret_cast<uintptr_t>(m->syn0) | reinterpret_cast<uintptr_t>(m->syn1)) & 15)
        return fail(W2V_E_ARG, "syn0/syn1 must be 16-byte aligned");
    if (!m->vocab_counts) return fail(W2V_E_ARG, "vocab_counts is NULL");
    if (m->train_words < 1) return fail(W2V_E_ARG, "train_words must be >= 1");
    if (need_tree && (!m->codelen || !m->code || !m->point_off || !m->points))
        return fail(W2V_E_ARG, "Huffman arrays are NULL");
    return W2V_OK;
}

// negative sampling: the noise table and the number of negatives (dim bounds the register tiles)
int check_ns(const w2v_model *m, const int32_t *table, int32_t log2_size, const w2v_params *p) {
    if (!table) return fail(W2V_E_ARG, "noise_table is NULL");
    if (log2_size < 1 || log2_size > 30) return fail(W2V_E_ARG, "log2_size must be in 1..30");
    if (m && m->dim > 512) return fail(W2V_E_ARG, "negative sampling needs dim <= 512");
    const int kmax = (m && m->dim > 320) ? 7 : 11;
    if (p->negative < 1 || p->negative > kmax)
        return fail(W2V_E_ARG, "negative must be in 1.." + std::to_string(kmax));
    return W2V_OK;
}

int timing_events(hipEvent_t *e0, hipEvent_t *e1) {
    int d = 0;
    W2V_HIP(hipGetDevice(&d));
    if (d < 0 || d >= 64) return fail(W2V_E_ARG, "device index out of range");
    std::lock_guard<std::mutex> lk(g_mu);
    DevInfo &di = g_dev[d];
    if (!di.have_timing) {
        W2V_HIP(hipEventCreate(&di.ev0));
        W2V_HIP(hipEventCreate(&di.ev1));
        di.have_timing = true;
    }
    *e0 = di.ev0;
    *e1 = di.ev1;
    return W2V_OK;
}

__global__ void k_zero_stats(unsigned long long *p) {
    if (threadIdx.x < 4) p[threadIdx.x] = 0;
}

// Parked hidden-layer gradients of the asynchronous kernel (skip-gram windows
// wider than one register group): floats, 0 when none are needed.
// The write policy the training kernel applies: the delta-only cache updates cached rows by LDS adds.
int32_t kernel_write_policy(const w2v_params *p) {
    return (p->cache_mode == 1 && p->cache_k > 0) ? (p->write_policy & ~4) : p->write_policy;
}

int64_t egrad_floats(const w2v_model *m, int64_t n_tokens, const w2v_params *p) {
    if (p->mode != 0) return 0;
    int grid = 0, waves = 0;
    const int64_t n_docs = n_tokens > 0 ? ceil_div(n_tokens, static_cast<int64_t>(p->doc_len)) : 0;
    const bool buf = train_stores_only(kernel_write_policy(p), p->cache_k, p->hot_k, m->dim);
    const bool delta = p->cache_mode == 1 && p->cache_k > 0;
    if (train_launch_shape(p->arch, m->dim, p->cache_k, delta, buf, p->workers, n_docs * segs_per_doc(p->doc_len),
                           &grid, &waves))
        return 0;
    return train_egrad_floats(p->arch, m->dim, buf, m->row_stride, p->window, waves);
}

size_t train_bytes(const w2v_model *m, int64_t n_tokens, const w2v_params *p) {
    Carve c;
    sample_bufs_carve(c, m->V, n_tokens, p->doc_len);
    const int64_t span = std::max<int64_t>(1, n_tokens);
    c.take<float>(static_cast<size_t>(span / 10000 + 3));   // alpha blocks
    c.take<int32_t>(4);                                     // queue
    c.take<unsigned long long>(4);                          // kernel stats
    c.take<float>(static_cast<size_t>(egrad_floats(m, n_tokens, p)));
    size_t b = c.used();
    if (p->mode == 1) b += sync_extra_bytes(m->V, m->dim, std::max<int64_t>(1, ceil_div(n_tokens, p->doc_len)));
    return b;
}

}  // namespace

namespace w2v {

int check_loglik_args(const w2v_model *m, const int32_t *tokens, int64_t n_tokens, const w2v_params *p,
                      const double *sum_ll_host, const int64_t *n_pairs_host) {
    if (int rc = check_model(m, true)) return rc;
    if (int rc = check_params(p, false)) return rc;
    if (p->arch < 0 || p->arch > 2)
        return fail(W2V_E_ARG, "arch must be 0 or 2 (pairs' objective) or 1 (CBOW's objective)");
    if (n_tokens < 0 || (n_tokens > 0 && !tokens)) return fail(W2V_E_ARG, "bad tokens / n_tokens");
    if (!sum_ll_host || !n_pairs_host) return fail(W2V_E_ARG, "a required pointer is NULL");
    return W2V_OK;
}

int loglik_run(const w2v_model *m, const int32_t *tokens, int64_t n_tokens, const w2v_params *p, double *sum_ll_host,
               int64_t *n_pairs_host, int64_t *n_nodes_host, void *workspace, hipStream_t s) {
    Carve c(workspace);
    SampleBufs b = sample_bufs_carve(c, m->V, n_tokens, p->doc_len);
    if (int rc = launch_sampling(tokens, n_tokens, m->V, m->vocab_counts, m->train_words, p, b, nullptr, s)) return rc;
    return run_loglik(m, p, b, n_tokens, c, sum_ll_host, n_pairs_host, n_nodes_host, s);
}

}  // namespace w2v

extern "C" {

const char *w2v_last_error(void) { return g_err.c_str(); }

size_t w2v_build_vocab_workspace_bytes(int32_t id_space) {
    return id_space < 1 ? 0 : vocab_workspace_bytes(id_space);
}

int w2v_build_vocab(const int32_t *tokens, int64_t n_tokens, int32_t id_space, int64_t min_count,
                    int64_t *counts_by_id, int32_t *vocab_ids, int64_t *vocab_counts, int32_t *id_to_vocab,
                    int32_t *tokens_out, int32_t *V_host, int64_t *train_words_host, void *workspace,
                    size_t workspace_bytes, void *hip_stream) {
    g_err.clear();
    if (id_space < 1 || id_space > (1 << 30)) return fail(W2V_E_ARG, "id_space must be in 1..2^30");
    if (n_tokens < 0) return fail(W2V_E_ARG, "n_tokens must be >= 0");
    if (min_count < 0) return fail(W2V_E_ARG, "min_count must be >= 0");
    if ((n_tokens > 0 && !tokens) || !counts_by_id || !vocab_ids || !vocab_counts || !id_to_vocab || !V_host ||
        !train_words_host)
        return fail(W2V_E_ARG, "a required pointer is NULL");
    if (tokens_out && tokens_out == tokens) return fail(W2V_E_ARG, "tokens_out may not alias tokens");
    if (int rc = check_ws(workspace, workspace_bytes, vocab_workspace_bytes(id_space))) return rc;
    return run_build_vocab(tokens, n_tokens, id_space, min_count, counts_by_id, vocab_ids, vocab_counts, id_to_vocab,
                           tokens_out, V_host, train_words_host, workspace, as_stream(hip_stream));
}

size_t w2v_build_huffman_workspace_bytes(int32_t V) { return V < 2 ? 0 : huffman_workspace_bytes(V); }

int w2v_build_huffman(const int64_t *vocab_counts, int32_t V, uint8_t *codelen, uint64_t *code, int32_t *point_off,
                      int32_t *points, int64_t points_cap, int64_t *points_len_host, int32_t *max_len_host,
                      void *workspace, size_t workspace_bytes, void *hip_stream) {
    g_err.clear();
    if (V < 2 || V > (1 << 26)) return fail(W2V_E_ARG, "V must be in 2..2^26");
    if (!vocab_counts || !codelen || !code || !point_off || !points_len_host || !max_len_host)
        return fail(W2V_E_ARG, "a required pointer is NULL");
    if (points && points_cap < 0) return fail(W2V_E_ARG, "points_cap must be >= 0");
    if (int rc = check_ws(workspace, workspace_bytes, huffman_workspace_bytes(V))) return rc;
    return run_build_huffman(vocab_counts, V, codelen, code, point_off, points, points_cap, points_len_host,
                             max_len_host, workspace, as_stream(hip_stream));
}

size_t w2v_train_workspace_bytes(const w2v_model *m, int64_t n_tokens, const w2v_params *p) {
    if (!m || !p || p->doc_len < 1 || m->V < 2) return 0;
    return train_bytes(m, n_tokens, p);
}

int w2v_train_hs_epoch(const w2v_model *m, const int32_t *tokens, int64_t n_tokens, const w2v_params *p,
                       int64_t *stats, void *workspace, size_t workspace_bytes, void *hip_stream) {
    g_err.clear();
    if (int rc = check_model(m, true)) return rc;
    if (int rc = check_params(p, true)) return rc;
    if (n_tokens < 0 || (n_tokens > 0 && !tokens)) return fail(W2V_E_ARG, "bad tokens / n_tokens");
    if (p->cache_k > m->V - 1) return fail(W2V_E_ARG, "cache_k must be <= V-1");
    const size_t lds = train_lds_bytes(p->cache_k, m->dim, p->cache_mode == 1);
    if (lds + 1024 > device_max_lds())
        return fail(W2V_E_ARG, "cache does not fit LDS: the cache_k rows and the centre records take " +
                                    std::to_string(lds) + " bytes");
    if (int rc = check_ws(workspace, workspace_bytes, train_bytes(m, n_tokens, p))) return rc;
    if (ceil_div(std::max<int64_t>(0, n_tokens), p->doc_len) * segs_per_doc(p->doc_len) > INT32_MAX)
        return fail(W2V_E_ARG, "too many documents for one call: split the stream (first_raw_index)");
    hipStream_t s = as_stream(hip_stream);
    Carve c(workspace);
    SampleBufs b = sample_bufs_carve(c, m->V, n_tokens, p->doc_len);
    const int64_t span = std::max<int64_t>(1, n_tokens);
    float *alpha_tab = c.take<float>(static_cast<size_t>(span / 10000 + 3));
    int32_t *queue = c.take<int32_t>(4);
    unsigned long long *tstats = c.take<unsigned long long>(4);
    const int64_t n_egrad = egrad_floats(m, n_tokens, p);
    float *egrad = c.take<float>(static_cast<size_t>(n_egrad));

    if (int rc = launch_sampling(tokens, n_tokens, m->V, m->vocab_counts, m->train_words, p, b, nullptr, s)) return rc;
    const int64_t eb = static_cast<int64_t>(p->epoch) * p->corpus_tokens;
    const int64_t blk0 = (eb + p->first_raw_index) / 10000;
    const int64_t blk1 = (eb + p->first_raw_index + span - 1) / 10000;
    if (int rc = launch_alpha_table(p, blk0, blk1 - blk0 + 1, alpha_tab, s)) return rc;

    if (p->mode == 1) {
        k_zero_stats<<<1, 64, 0, s>>>(tstats);
        W2V_LAUNCH_CHECK("k_zero_stats");
        if (int rc = run_train_sync(m, p, b, n_tokens, c, alpha_tab, blk0, tstats, s)) return rc;
        if (stats) {
            // raw and in-vocabulary counts from the sampler, the rest from the gradient kernel
            W2V_HIP(hipMemcpyAsync(stats, b.totals, 2 * sizeof(int64_t), hipMemcpyDeviceToDevice, s));
            W2V_HIP(hipMemcpyAsync(stats + 2, tstats, 3 * sizeof(int64_t), hipMemcpyDeviceToDevice, s));
        }
        return W2V_OK;
    }
    TrainArgs a{};
    a.syn0 = m->syn0;
    a.syn1 = m->syn1;
    a.V = m->V;
    a.dim = m->dim;
    a.stride = m->row_stride;
    a.codelen = m->codelen;
    a.code = m->code;
    a.point_off = m->point_off;
    a.points = m->points;
    a.kept_vid = b.kept_vid;
    a.kept_meta = b.kept_meta;
    a.doc_kept = b.doc_kept;
    a.n_docs = n_tokens > 0 ? ceil_div(n_tokens, p->doc_len) : 0;
    a.doc_len = p->doc_len;
    a.seg_len = kSegLen;
    a.segs_per_doc = segs_per_doc(p->doc_len);
    a.n_units = a.n_docs * a.segs_per_doc;
    a.first_raw = p->first_raw_index;
    a.epoch_base = eb;
    a.alpha_tab = alpha_tab;
    a.blk0 = blk0;
    a.cache_k = p->cache_k;
    a.cache_first = m->V - 1 - p->cache_k;
    a.atomic_first = static_cast<int32_t>(std::max<int64_t>(0, static_cast<int64_t>(a.cache_first) - p->hot_k));
    a.flush_every = p->flush_every;
    a.workers = p->workers;
    a.cache_delta = (p->cache_mode == 1 && p->cache_k > 0) ? 1 : 0;
    a.span_refresh = p->span_refresh;
    a.span_stash = p->span_stash;
    a.stash_from = p->stash_from;
    a.write_policy = kernel_write_policy(p);
    a.stores_only = train_stores_only(a.write_policy, p->cache_k, p->hot_k, m->dim) ? 1 : 0;
    a.flush_scale = p->flush_policy == 1 ? 0.0f : 1.0f;   // 0: set to 1 / workgroups at launch
    a.queue = queue;
    a.stats = tstats;
    a.egrad = n_egrad > 0 ? egrad : nullptr;
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
    if (int rc = timing_events(&ev0, &ev1)) return rc;
    return launch_train_async(a, p->arch, p->window, ev0, ev1, s, stats, b.totals);
}

int32_t w2v_train_word_span(const w2v_model *m, const w2v_params *p) {
    g_err.clear();
    if (!m || !p) {
        fail(W2V_E_ARG, "a required pointer is NULL");
        return -1;
    }
    if (check_model(m, false) != W2V_OK || check_params(p, true) != W2V_OK) return -1;
    if (p->mode != 0) return 0;
    const int32_t wp = kernel_write_policy(p);
    return train_word_span(p->arch, m->dim, train_stores_only(wp, p->cache_k, p->hot_k, m->dim), wp, p->window);
}

int w2v_last_train_kernel_ms(float *ms_host) {
    g_err.clear();
    if (!ms_host) return fail(W2V_E_ARG, "ms_host is NULL");
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
    if (int rc = timing_events(&ev0, &ev1)) return rc;
    W2V_HIP(hipEventSynchronize(ev1));
    W2V_HIP(hipEventElapsedTime(ms_host, ev0, ev1));
    return W2V_OK;
}

int w2v_last_train_launch(int32_t *workgroups_host, int32_t *wavefronts_host) {
    g_err.clear();
    if (!workgroups_host || !wavefronts_host) return fail(W2V_E_ARG, "a required pointer is NULL");
    DevInfo &di = dev_info();
    std::lock_guard<std::mutex> lk(g_mu);
    *workgroups_host = di.last_groups;
    *wavefronts_host = di.last_waves;
    return W2V_OK;
}

int w2v_last_train_resources(int32_t *lds_bytes_host, int32_t *vgprs_host, int32_t *waves_per_simd_host) {
    g_err.clear();
    if (!lds_bytes_host || !vgprs_host || !waves_per_simd_host) return fail(W2V_E_ARG, "a required pointer is NULL");
    DevInfo &di = dev_info();
    std::lock_guard<std::mutex> lk(g_mu);
    *lds_bytes_host = di.last_lds;
    *vgprs_host = di.last_vgprs;
    *waves_per_simd_host = di.last_waves_per_simd;
    return W2V_OK;
}

size_t w2v_hs_loglik_workspace_bytes(const w2v_model *m, int64_t n_tokens, const w2v_params *p) {
    if (!m || !p || p->doc_len < 1 || m->V < 2) return 0;
    Carve c;
    sample_bufs_carve(c, m->V, n_tokens, p->doc_len);
    return c.used() + loglik_extra_bytes(loglik_units(n_tokens, p->doc_len));
}

int w2v_hs_loglik(const w2v_model *m, const int32_t *tokens, int64_t n_tokens, const w2v_params *p,
                  double *sum_ll_host, int64_t *n_pairs_host, int64_t *n_nodes_host, void *workspace,
                  size_t workspace_bytes, void *hip_stream) {
    g_err.clear();
    if (int rc = check_loglik_args(m, tokens, n_tokens, p, sum_ll_host, n_pairs_host)) return rc;
    if (int rc = check_ws(workspace, workspace_bytes, w2v_hs_loglik_workspace_bytes(m, n_tokens, p))) return rc;
    return loglik_run(m, tokens, n_tokens, p, sum_ll_host, n_pairs_host, n_nodes_host, workspace,
                      as_stream(hip_stream));
}

size_t w2v_noise_table_workspace_bytes(int32_t V) { return V < 1 ? 0 : noise_workspace_bytes(V); }

int w2v_build_noise_table(const int64_t *vocab_counts, int32_t V, int32_t log2_size, int32_t *table,
                          int64_t *total_weight_host, void *workspace, size_t workspace_bytes, void *hip_stream) {
    g_err.clear();
    if (V < 1 || V > (1 << 30)) return fail(W2V_E_ARG, "V must be in 1..2^30");
    if (log2_size < 1 || log2_size > 30) return fail(W2V_E_ARG, "log2_size must be in 1..30");
    if (!vocab_counts || !table || !total_weight_host) return fail(W2V_E_ARG, "a required pointer is NULL");
    if (int rc = check_ws(workspace, workspace_bytes, noise_workspace_bytes(V))) return rc;
    return run_noise_table(vocab_counts, V, log2_size, table, total_weight_host, workspace, as_stream(hip_stream));
}

size_t w2v_train_ns_workspace_bytes(const w2v_model *m, int64_t n_tokens, const w2v_params *p) {
    if (!m || !p || p->doc_len < 1 || m->V < 2) return 0;
    Carve c;
    sample_bufs_carve(c, m->V, n_tokens, p->doc_len);
    c.take<float>(static_cast<size_t>(std::max<int64_t>(1, n_tokens) / 10000 + 3));   // alpha blocks
    return c.used() + ns_train_extra_bytes();
}

int w2v_train_ns_epoch(const w2v_model *m, const int32_t *noise_table, int32_t log2_size, const int32_t *tokens,
                       int64_t n_tokens, const w2v_params *p, int64_t *stats, void *workspace, size_t workspace_bytes,
                       void *hip_stream) {
    g_err.clear();
    if (int rc = check_model(m, false)) return rc;
    if (int rc = check_params(p, true)) return rc;
    if (p->arch != 0 || p->mode != 0) return fail(W2V_E_ARG, "negative sampling trains skip-gram, mode 0, only");
    if (int rc = check_ns(m, noise_table, log2_size, p)) return rc;
    if (n_tokens < 0 || (n_tokens > 0 && !tokens)) return fail(W2V_E_ARG, "bad tokens / n_tokens");
    if (int rc = check_ws(workspace, workspace_bytes, w2v_train_ns_workspace_bytes(m, n_tokens, p))) return rc;
    if (ceil_div(std::max<int64_t>(0, n_tokens), p->doc_len) * segs_per_doc(p->doc_len) > INT32_MAX)
        return fail(W2V_E_ARG, "too many documents for one call: split the stream (first_raw_index)");
    hipStream_t s = as_stream(hip_stream);
    Carve c(workspace);
    SampleBufs b = sample_bufs_carve(c, m->V, n_tokens, p->doc_len);
    const int64_t span = std::max<int64_t>(1, n_tokens);
    float *alpha_tab = c.take<float>(static_cast<size_t>(span / 10000 + 3));
    if (int rc = launch_sampling(tokens, n_tokens, m->V, m->vocab_counts, m->train_words, p, b, nullptr, s)) return rc;
    const int64_t eb = static_cast<int64_t>(p->epoch) * p->corpus_tokens;
    const int64_t blk0 = (eb + p->first_raw_index) / 10000;
    const int64_t blk1 = (eb + p->first_raw_index + span - 1) / 10000;
    if (int rc = launch_alpha_table(p, blk0, blk1 - blk0 + 1, alpha_tab, s)) return rc;
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
    if (int rc = timing_events(&ev0, &ev1)) return rc;
    return launch_train_ns(m, noise_table, log2_size, p, b, n_tokens, alpha_tab, blk0, c, ev0, ev1, stats, s);
}

size_t w2v_ns_objective_workspace_bytes(const w2v_model *m, int64_t n_tokens, const w2v_params *p) {
    if (!m || !p || p->doc_len < 1 || m->V < 2) return 0;
    Carve c;
    sample_bufs_carve(c, m->V, n_tokens, p->doc_len);
    return c.used() + ns_objective_extra_bytes(std::max<int64_t>(1, ceil_div(n_tokens, p->doc_len)), p->doc_len);
}

int w2v_ns_objective(const w2v_model *m, const int32_t *noise_table, int32_t log2_size, const int32_t *tokens,
                     int64_t n_tokens, const w2v_params *p, double *sum_host, int64_t *n_pairs_host,
                     int64_t *n_terms_host, void *workspace, size_t workspace_bytes, void *hip_stream) {
    g_err.clear();
    if (int rc = check_model(m, false)) return rc;
    if (int rc = check_params(p, false)) return rc;
    if (int rc = check_ns(m, noise_table, log2_size, p)) return rc;
    if (n_tokens < 0 || (n_tokens > 0 && !tokens)) return fail(W2V_E_ARG, "bad tokens / n_tokens");
    if (!sum_host || !n_pairs_host) return fail(W2V_E_ARG, "a required pointer is NULL");
    if (int rc = check_ws(workspace, workspace_bytes, w2v_ns_objective_workspace_bytes(m, n_tokens, p))) return rc;
    hipStream_t s = as_stream(hip_stream);
    Carve c(workspace);
    SampleBufs b = sample_bufs_carve(c, m->V, n_tokens, p->doc_len);
    if (int rc = launch_sampling(tokens, n_tokens, m->V, m->vocab_counts, m->train_words, p, b, nullptr, s)) return rc;
    return run_ns_objective(m, noise_table, log2_size, p, b, n_tokens, c, sum_host, n_pairs_host, n_terms_host, s);
}

size_t w2v_sample_negatives_workspace_bytes(int32_t V, int64_t n_tokens, const w2v_params *p) {
    if (!p || p->doc_len < 1 || V < 1) return 0;
    Carve c;
    sample_bufs_carve(c, V, n_tokens, p->doc_len);
    return c.used() + ns_negatives_extra_bytes(std::max<int64_t>(1, ceil_div(n_tokens, p->doc_len)));
}

int w2v_sample_negatives(const int32_t *tokens, int64_t n_tokens, int32_t V, const int64_t *vocab_counts,
                         int64_t train_words, const w2v_params *p, const int32_t *noise_table, int32_t log2_size,
                         int32_t *negatives, int64_t negatives_cap, int64_t *n_kept_host, uint64_t *checksum_host,
                         void *workspace, size_t workspace_bytes, void *hip_stream) {
    g_err.clear();
    if (int rc = check_params(p, false)) return rc;
    if (int rc = check_ns(nullptr, noise_table, log2_size, p)) return rc;
    if (V < 1) return fail(W2V_E_ARG, "V must be >= 1");
    if (n_tokens < 0 || (n_tokens > 0 && !tokens) || !vocab_counts) return fail(W2V_E_ARG, "bad tokens / counts");
    if (!n_kept_host || !checksum_host) return fail(W2V_E_ARG, "a required pointer is NULL");
    if (negatives_cap < 0) return fail(W2V_E_ARG, "negatives_cap must be >= 0");
    if (p->sample > 0.0 && train_words < 1) return fail(W2V_E_ARG, "train_words must be >= 1 when sample > 0");
    if (int rc = check_ws(workspace, workspace_bytes, w2v_sample_negatives_workspace_bytes(V, n_tokens, p))) return rc;
    hipStream_t s = as_stream(hip_stream);
    Carve c(workspace);
    SampleBufs b = sample_bufs_carve(c, V, n_tokens, p->doc_len);
    if (int rc = launch_sampling(tokens, n_tokens, V, vocab_counts, train_words, p, b, nullptr, s)) return rc;
    return run_ns_negatives(p, noise_table, log2_size, b, n_tokens, c, negatives, negatives_cap, n_kept_host,
                            checksum_host, s);
}

size_t w2v_sample_pairs_workspace_bytes(int32_t V, int64_t n_tokens, const w2v_params *p) {
    if (!p || p->doc_len < 1 || V < 1) return 0;
    return pairs_workspace_bytes(V, n_tokens, p->doc_len);
}

int w2v_sample_pairs(const int32_t *tokens, int64_t n_tokens, int32_t V, const int64_t *vocab_counts,
                     int64_t train_words, const w2v_params *p, int64_t *centre_raw, int64_t *context_raw,
                     int64_t pair_cap, uint8_t *keep_mask, int64_t *n_pairs_host, int64_t *n_kept_host,
                     uint64_t *checksum_host, void *workspace, size_t workspace_bytes, void *hip_stream) {
    g_err.clear();
    if (int rc = check_params(p, false)) return rc;
    if (V < 1) return fail(W2V_E_ARG, "V must be >= 1");
    if (n_tokens < 0 || (n_tokens > 0 && !tokens) || !vocab_counts) return fail(W2V_E_ARG, "bad tokens / counts");
    if (!n_pairs_host || !n_kept_host || !checksum_host) return fail(W2V_E_ARG, "a required pointer is NULL");
    if (pair_cap < 0) return fail(W2V_E_ARG, "pair_cap must be >= 0");
    if (p->sample > 0.0 && train_words < 1) return fail(W2V_E_ARG, "train_words must be >= 1 when sample > 0");
    if (int rc = check_ws(workspace, workspace_bytes, pairs_workspace_bytes(V, n_tokens, p->doc_len))) return rc;
    return run_sample_pairs(tokens, n_tokens, V, vocab_counts, train_words, p, centre_raw, context_raw, pair_cap,
                            keep_mask, n_pairs_host, n_kept_host, checksum_host, workspace, as_stream(hip_stream));
}

int w2v_keep_thresholds(const int64_t *vocab_counts, int32_t V, double sample, int64_t train_words, uint64_t *thr,
                        void *hip_stream) {
    g_err.clear();
    if (V < 1 || !vocab_counts || !thr) return fail(W2V_E_ARG, "bad arguments");
    if (!(sample >= 0.0) || sample >= 1.0) return fail(W2V_E_ARG, "sample must be in [0, 1)");
    return launch_thresholds(vocab_counts, V, sample, train_words, thr, as_stream(hip_stream));
}

}  // extern "C"

