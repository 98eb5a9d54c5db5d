// Subsampling ("downsample", §4.1), documents, window draws ("each wordid w
// within window of v", Algorithm 1) and the learning-rate table ("update
// alpha", Algorithm 1).
//
// Every raw token at global index g draws Philox4x32-10 with counter
// (g_lo, g_hi, epoch, 0) and key = seed: word 0 decides the keep
// (keep iff in vocabulary and word0 < thr[v]); word 1 the window
// (half-width W - floor(word1 W / 2^32)). Being keyed by position, the draws do
// not depend on the order in which the GPU visits documents.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "w2v_internal.h"
#include "w2v_scan.h"

namespace w2v {
namespace {

// thr[v] = 2^32 if p_keep >= 1 else floor(p_keep 2^32), p_keep = sqrt(q) + q, q = t N_t / count(v).
// Explicit round-to-nearest operations: no contraction, so the table is exact and reproducible.
__global__ void k_thresholds(const int64_t *__restrict__ counts, int32_t V, double sample, int64_t train_words,
                             uint64_t *__restrict__ thr) {
    const int32_t v = blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= V) return;
    const uint64_t all = 1ull << 32;
    if (!(sample > 0.0)) {
        thr[v] = all;
        return;
    }
    const double tn = __dmul_rn(sample, static_cast<double>(train_words));
    const double q = __ddiv_rn(tn, static_cast<double>(counts[v]));
    const double pk = __dadd_rn(__dsqrt_rn(q), q);
    thr[v] = (pk >= 1.0) ? all : static_cast<uint64_t>(floor(__dmul_rn(pk, 4294967296.0)));
}

// alpha of the 10,000-token block b of the run (blocks counted over epoch * N_raw + raw index):
// alpha0 * max(1e-4, 1 - 10^4 b / (E N_raw + 1)).
__global__ void k_alpha(float alpha0, int64_t blk0, int64_t nblk, int32_t n_epochs, int64_t corpus_tokens,
                        float *__restrict__ tab) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= nblk) return;
    const int64_t b = blk0 + i;
    const double frac = __ddiv_rn(static_cast<double>(b * 10000),
                                  static_cast<double>(static_cast<int64_t>(n_epochs) * corpus_tokens + 1));
    double a = __dsub_rn(1.0, frac);
    if (a < 1e-4) a = 1e-4;
    tab[i] = static_cast<float>(__dmul_rn(static_cast<double>(alpha0), a));
}

__global__ void k_zero_i64(int64_t *p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

// One wavefront per document: keep mask, compaction in raw order, window draw,
// pair count. Writes kept_vid / kept_meta in the document's slots.
constexpr int kSampleThreads = 256;
__global__ __launch_bounds__(kSampleThreads) void k_subsample(const int32_t *__restrict__ tok, int64_t n, int32_t V,
                                                              int32_t doc_len, int64_t first_raw, int32_t epoch,
                                                              uint64_t seed, int32_t window,
                                                              const uint64_t *__restrict__ thr,
                                                              int32_t *__restrict__ kept_vid,
                                                              uint32_t *__restrict__ kept_meta,
                                                              int32_t *__restrict__ doc_kept,
                                                              int64_t *__restrict__ doc_pairs,
                                                              uint8_t *__restrict__ keep_mask,
                                                              int64_t *__restrict__ totals) {
    const int lane = lane_id();
    const int64_t n_docs = ceil_div(n, doc_len);
    const int64_t wave0 = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * blockDim.x / kWave;
    int64_t my_raw = 0, my_inv = 0, my_kept = 0, my_pairs = 0;
    for (int64_t d = wave0; d < n_docs; d += nwaves) {
        const int64_t lo = d * doc_len;
        const int32_t len = static_cast<int32_t>(min<int64_t>(doc_len, n - lo));
        int32_t nk = 0;
        for (int32_t b = 0; b < len; b += kWave) {
            const int32_t off = b + lane;
            bool keep = false;
            int32_t v = -1;
            uint32_t eff = 0;
            if (off < len) {
                v = tok[lo + off];
                if (v >= V) v = -1;   // not a vocabulary index: treated as dropped
                if (v >= 0) {
                    ++my_inv;
                    const U4 r = token_draw(seed, first_raw + lo + off, epoch);
                    keep = static_cast<uint64_t>(r.x) < thr[v];
                    const uint32_t bw = static_cast<uint32_t>((static_cast<uint64_t>(r.y) * window) >> 32);
                    eff = static_cast<uint32_t>(window) - bw;
                }
                if (keep_mask) keep_mask[lo + off] = keep ? 1 : 0;
            }
            const uint64_t m = __ballot(keep);
            const int32_t pos = nk + static_cast<int32_t>(__popcll(m & ((1ull << lane) - 1)));
            if (keep) {
                kept_vid[lo + pos] = v;
                kept_meta[lo + pos] = static_cast<uint32_t>(off) | (eff << 16);
            }
            nk += static_cast<int32_t>(__popcll(m));
        }
        // pairs of each kept centre: min(eff, j) + min(eff, nk - 1 - j)
        int64_t pc = 0;
        for (int32_t j = lane; j < nk; j += kWave) {
            const int32_t e = static_cast<int32_t>(kept_meta[lo + j] >> 16);
            pc += min(e, j) + min(e, nk - 1 - j);
        }
        pc = wave_sum(pc);
        if (lane == 0) {
            doc_kept[d] = nk;
            doc_pairs[d] = pc;
        }
        my_raw += len;
        my_kept += nk;
        my_pairs += pc;
    }
    my_inv = wave_sum(my_inv);
    if (lane == 0) {
        atomicAdd(reinterpret_cast<unsigned long long *>(&totals[0]), static_cast<unsigned long long>(my_raw));
        atomicAdd(reinterpret_cast<unsigned long long *>(&totals[1]), static_cast<unsigned long long>(my_inv));
        atomicAdd(reinterpret_cast<unsigned long long *>(&totals[2]), static_cast<unsigned long long>(my_kept));
        atomicAdd(reinterpret_cast<unsigned long long *>(&totals[3]), static_cast<unsigned long long>(my_pairs));
    }
}

}  // namespace

size_t sample_bufs_bytes(int32_t V, int64_t n_tokens, int32_t doc_len) {
    Carve c;
    sample_bufs_carve(c, V, n_tokens, doc_len);
    return c.used();
}

SampleBufs sample_bufs_carve(Carve &c, int32_t V, int64_t n_tokens, int32_t doc_len) {
    const int64_t n_docs = std::max<int64_t>(1, ceil_div(n_tokens, doc_len));
    SampleBufs b;
    b.kept_vid = c.take<int32_t>(static_cast<size_t>(n_docs) * doc_len);
    b.kept_meta = c.take<uint32_t>(static_cast<size_t>(n_docs) * doc_len);
    b.doc_kept = c.take<int32_t>(static_cast<size_t>(n_docs));
    b.doc_pairs = c.take<int64_t>(static_cast<size_t>(n_docs));
    b.thr = c.take<uint64_t>(static_cast<size_t>(V));
    b.totals = c.take<int64_t>(4);
    return b;
}

int launch_thresholds(const int64_t *vocab_counts, int32_t V, double sample, int64_t train_words, uint64_t *thr,
                      hipStream_t s) {
    k_thresholds<<<static_cast<unsigned>(ceil_div(V, 256)), 256, 0, s>>>(vocab_counts, V, sample, train_words, thr);
    W2V_LAUNCH_CHECK("k_thresholds");
    return W2V_OK;
}

int launch_sampling(const int32_t *tokens, int64_t n_tokens, int32_t V, const int64_t *vocab_counts,
                    int64_t train_words, const w2v_params *p, const SampleBufs &b, uint8_t *keep_mask,
                    hipStream_t s) {
    int rc = launch_thresholds(vocab_counts, V, p->sample, train_words, b.thr, s);
    if (rc) return rc;
    k_zero_i64<<<1, 64, 0, s>>>(b.totals, 4);
    W2V_LAUNCH_CHECK("k_zero_i64");
    if (n_tokens <= 0) return W2V_OK;
    const int64_t n_docs = ceil_div(n_tokens, p->doc_len);
    const int64_t want = ceil_div(n_docs, kSampleThreads / kWave);
    const unsigned grid = static_cast<unsigned>(std::min<int64_t>(want, 16LL * device_cu_count()));
    k_subsample<<<grid, kSampleThreads, 0, s>>>(tokens, n_tokens, V, p->doc_len, p->first_raw_index, p->epoch, p->seed,
                                                p->window, b.thr, b.kept_vid, b.kept_meta, b.doc_kept, b.doc_pairs,
                                                keep_mask, b.totals);
    W2V_LAUNCH_CHECK("k_subsample");
    return W2V_OK;
}

int launch_alpha_table(const w2v_params *p, int64_t blk0, int64_t nblk, float *tab, hipStream_t s) {
    if (nblk <= 0) return W2V_OK;
    k_alpha<<<static_cast<unsigned>(ceil_div(nblk, 256)), 256, 0, s>>>(p->alpha0, blk0, nblk, p->n_epochs,
                                                                       p->corpus_tokens, tab);
    W2V_LAUNCH_CHECK("k_alpha");
    return W2V_OK;
}

// ------------------------------------------------------------ pair listing
namespace {

// exclusive scan of doc_pairs (int64) over n_docs (one workgroup)
__global__ __launch_bounds__(kScanThreads) void k_scan_i64(const int64_t *__restrict__ in, int64_t n,
                                                           int64_t *__restrict__ out) {
    block_exclusive_scan(in, n, out);
}

// one wave per document: write its pairs at the document's offset; checksum of all pairs
__global__ __launch_bounds__(256) void k_pairs(int64_t n, int32_t doc_len, int64_t first_raw,
                                               const uint32_t *__restrict__ kept_meta,
                                               const int32_t *__restrict__ doc_kept,
                                               const int64_t *__restrict__ doc_off, int64_t *__restrict__ c_out,
                                               int64_t *__restrict__ x_out, int64_t cap,
                                               unsigned long long *__restrict__ checksum) {
    const int lane = lane_id();
    const int64_t n_docs = ceil_div(n, doc_len);
    const int64_t wave0 = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * blockDim.x / kWave;
    uint64_t cs = 0;
    for (int64_t d = wave0; d < n_docs; d += nwaves) {
        const int64_t lo = d * doc_len;
        const int32_t nk = doc_kept[d];
        int64_t base = doc_off[d];
        for (int32_t j0 = 0; j0 < nk; j0 += kWave) {
            const int32_t j = j0 + lane;
            int32_t cnt = 0, e = 0;
            if (j < nk) {
                e = static_cast<int32_t>(kept_meta[lo + j] >> 16);
                cnt = min(e, j) + min(e, nk - 1 - j);
            }
            int32_t inc = cnt;
#pragma unroll
            for (int dd = 1; dd < 64; dd <<= 1) {
                const int32_t y = __shfl_up(inc, dd, 64);
                if (lane >= dd) inc += y;
            }
            const int64_t at = base + inc - cnt;
            if (j < nk) {
                const int64_t gc = first_raw + lo + (kept_meta[lo + j] & 0xFFFFu);
                int64_t k = at;
                for (int32_t c = max(0, j - e); c <= min(nk - 1, j + e); ++c) {
                    if (c == j) continue;
                    const int64_t gx = first_raw + lo + (kept_meta[lo + c] & 0xFFFFu);
                    if (k < cap) {
                        if (c_out) c_out[k] = gc;
                        if (x_out) x_out[k] = gx;
                    }
                    cs += fmix64(static_cast<uint64_t>(gc) * 0x9E3779B97F4A7C15ull + static_cast<uint64_t>(gx));
                    ++k;
                }
            }
            base += __shfl(inc, 63, 64);
        }
    }
    // wrap-around sum across the wave, then one atomic
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) cs += __shfl_xor(cs, m, kWave);
    if (lane == 0) atomicAdd(checksum, static_cast<unsigned long long>(cs));
}

__global__ void k_zero_u64s(unsigned long long *p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

}  // namespace

size_t pairs_workspace_bytes(int32_t V, int64_t n_tokens, int32_t doc_len) {
    Carve c;
    sample_bufs_carve(c, V, n_tokens, doc_len);
    c.take<int64_t>(static_cast<size_t>(std::max<int64_t>(1, ceil_div(n_tokens, doc_len))));
    c.take<unsigned long long>(2);
    return c.used();
}

int run_sample_pairs(const int32_t *tokens, int64_t n_tokens, int32_t V, const int64_t *vocab_counts,
                     int64_t train_words, const w2v_params *p, int64_t *centre_raw, int64_t *context_raw,
                     int64_t pair_cap, uint8_t *keep_mask, int64_t *n_pairs_host, int64_t *n_kept_host,
                     uint64_t *checksum_host, void *workspace, hipStream_t s) {
    Carve c(workspace);
    SampleBufs b = sample_bufs_carve(c, V, n_tokens, p->doc_len);
    const int64_t n_docs = std::max<int64_t>(1, ceil_div(n_tokens, p->doc_len));
    int64_t *doc_off = c.take<int64_t>(static_cast<size_t>(n_docs));
    unsigned long long *cs = c.take<unsigned long long>(2);
    int rc = launch_sampling(tokens, n_tokens, V, vocab_counts, train_words, p, b, keep_mask, s);
    if (rc) return rc;
    k_zero_u64s<<<1, 64, 0, s>>>(cs, 2);
    W2V_LAUNCH_CHECK("k_zero_u64s");
    if (n_tokens > 0) {
        k_scan_i64<<<1, kScanThreads, 0, s>>>(b.doc_pairs, ceil_div(n_tokens, p->doc_len), doc_off);
        W2V_LAUNCH_CHECK("k_scan_i64");
        const unsigned grid = static_cast<unsigned>(
            std::min<int64_t>(ceil_div(ceil_div(n_tokens, p->doc_len), 4), 16LL * device_cu_count()));
        k_pairs<<<grid, 256, 0, s>>>(n_tokens, p->doc_len, p->first_raw_index, b.kept_meta, b.doc_kept, doc_off,
                                     centre_raw, context_raw, pair_cap, cs);
        W2V_LAUNCH_CHECK("k_pairs");
    }
    int64_t tot[4];
    unsigned long long hcs = 0;
    W2V_HIP(hipMemcpyAsync(tot, b.totals, sizeof(tot), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipMemcpyAsync(&hcs, cs, sizeof(hcs), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipStreamSynchronize(s));
    *n_pairs_host = tot[3];
    *n_kept_host = tot[2];
    *checksum_host = hcs;
    return W2V_OK;
}

}  // namespace w2v
