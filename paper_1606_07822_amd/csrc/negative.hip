// Negative sampling, the alternative objective to the hierarchical softmax
// that §2 names, in the mini-batch form of Ji et al. that the opening of §3.2
// describes: all window words of a centre train against the same targets --
// the centre word (label 1) and K negatives shared by the window (label 0) --
// and every gradient of the centre is taken from the vectors as they were
// before it (the level-3 form, which does not use updated vectors within a
// mini-batch, §4.3).
//
// Noise distribution: unigram counts raised to 3/4, with the weight of a
// count c computed in integers as isqrt(c * isqrt(c)) and laid out in a table
// of T = 2^L entries (entry i holds the word whose weight interval contains
// floor(i Q / T), Q = total weight), so that a 32-bit random word picks a
// negative with one load. Negative 4h+i of the centre at raw index g is
// table[r_i >> (32 - L)], r = Philox4x32-10(counter (g lo, g hi, epoch, 1+h),
// key = seed); one equal to the centre word is dropped.
//
// GPU form (one wavefront per centre, 128-centre document segments from a queue): the
// target rows Y are loaded once per centre and held in registers; the window
// rows X stream through, each once: its dot products with the targets are
// reduced four at a time (row j of the reduction holds target 4c+j), the
// gradients go to LDS and their outer product with x accumulates the targets'
// change in registers. A second pass over the window forms each word's change
// from the gradients in LDS and the unchanged targets. Target rows are
// written back as stores of their value before the centre plus the change
// (lock-free; the frequent words are negatives of many centres at once and
// atomic adds to them were the kernel's main cost); word rows take atomic
// adds of their change (or a re-read and store); a negative drawn twice or a
// word twice in the window adds its second change atomically, so one worker
// reproduces the sequential result. No MFMA: at P <= 20 window words
// and K + 1 <= 12 targets the products are far too small for matrix tiles,
// and the work is bound by the row traffic.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "w2v_internal.h"
#include "w2v_scan.h"

namespace w2v {
namespace {

constexpr int kNsWaves = 4;      // wavefronts per workgroup (one per SIMD: occupancy in steps of one wave)
constexpr int kMaxWindow = 20;   // window words per centre (2 * window, window <= 10)

// ------------------------------------------------------------ noise table
// floor(sqrt(x)) for x < 2^62: a double estimate corrected in integers.
__device__ __forceinline__ uint64_t isqrt_exact(uint64_t x) {
    uint64_t s = static_cast<uint64_t>(sqrt(static_cast<double>(x)));
    while (s * s > x) --s;
    while ((s + 1) * (s + 1) <= x) ++s;
    return s;
}

__global__ void k_noise_weights(const int64_t *__restrict__ counts, int32_t V, int64_t *__restrict__ w) {
    for (int64_t v = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; v < V;
         v += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const uint64_t c = static_cast<uint64_t>(counts[v]);
        w[v] = static_cast<int64_t>(isqrt_exact(c * isqrt_exact(c)));
    }
}

// exclusive scan of n int64 (one workgroup); out[n] = total
__global__ __launch_bounds__(kScanThreads) void k_scan_weights(const int64_t *__restrict__ in, int64_t n,
                                                               int64_t *__restrict__ out) {
    const int64_t total = block_exclusive_scan(in, n, out);
    if (threadIdx.x == 0) out[n] = total;
}

// word v fills entries [ceil(Q[v] T / Q), ceil(Q[v+1] T / Q)): exactly the i with
// Q[v] <= floor(i Q / T) < Q[v+1]. One wavefront per word, lanes along its entries.
__global__ __launch_bounds__(256) void k_noise_fill(const int64_t *__restrict__ pre, int32_t V, int32_t log2_size,
                                                    int32_t *__restrict__ table) {
    const int lane = lane_id();
    const uint64_t tot = static_cast<uint64_t>(pre[V]);
    const int64_t wave0 = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * blockDim.x / kWave;
    for (int64_t v = wave0; v < V; v += nwaves) {
        const uint64_t lo = ((static_cast<uint64_t>(pre[v]) << log2_size) + tot - 1) / tot;
        const uint64_t hi = ((static_cast<uint64_t>(pre[v + 1]) << log2_size) + tot - 1) / tot;
        for (uint64_t i = lo + lane; i < hi; i += kWave) table[i] = static_cast<int32_t>(v);
    }
}

// ------------------------------------------------------------ negatives
// Target slot t of a centre: 0 = the centre word, 1..K = its negatives, -1 = dropped or past K.
__device__ __forceinline__ int target_of(int t, int v, int K, uint64_t seed, int64_t raw, int32_t epoch,
                                         const int32_t *__restrict__ table, int log2_size) {
    if (t == 0) return v;
    if (t > K) return -1;
    const int k = t - 1;
    const U4 r = philox4x32_10(static_cast<uint32_t>(raw), static_cast<uint32_t>(static_cast<uint64_t>(raw) >> 32),
                               static_cast<uint32_t>(epoch), 1u + static_cast<uint32_t>(k >> 2),
                               static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32));
    const int i = k & 3;
    const uint32_t w = i == 0 ? r.x : i == 1 ? r.y : i == 2 ? r.z : r.w;
    const int n = table[w >> (32 - log2_size)];
    return n == v ? -1 : n;
}

template <int NE>
__device__ __forceinline__ void load_row(float (&r)[NE], const float *__restrict__ p, int lane, int dim) {
#pragma unroll
    for (int i = 0; i < NE; ++i) {
        const int col = lane + i * kWave;
        r[i] = (col < dim) ? p[col] : 0.0f;
    }
}

template <int NE>
__device__ __forceinline__ void atomic_add_row(float *p, const float (&r)[NE], int lane, int dim) {
#pragma unroll
    for (int i = 0; i < NE; ++i)
        if (lane + i * kWave < dim) atomicAdd(p + lane + i * kWave, r[i]);
}

template <int NE>
__device__ __forceinline__ void store_row(float *p, const float (&r)[NE], int lane, int dim) {
#pragma unroll
    for (int i = 0; i < NE; ++i)
        if (lane + i * kWave < dim) p[lane + i * kWave] = r[i];
}

// Partial dot product with target slot t, zero for the padding slots of the last group of four.
template <int NE, int NT>
__device__ __forceinline__ float dot_slot(const float (&x)[NE], const float (&y)[NT][NE], int t) {
    if (t < NT) return dot_partial<NE>(x, y[t]);
    return 0.0f;
}

__device__ __forceinline__ float bcast(float v, int lane) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}

// log sigmoid(u) = min(u, 0) - log(1 + exp(-|u|)): the same operations as the two one-sided forms, without
// a branch (lanes of both signs would run both sides)
__device__ __forceinline__ double log_sigmoid(double u) {
    return fmin(u, 0.0) - log1p(exp(-fabs(u)));
}

// Held-out objective work units: kObjSeg kept centres (short units keep the read-only walk's latency spread
// over many wavefronts, as in the hierarchical-softmax evaluation).
constexpr int kObjSeg = 8;
inline int32_t obj_segs_per_doc(int32_t doc_len) { return static_cast<int32_t>(ceil_div(doc_len, kObjSeg)); }

// ------------------------------------------------------------ training
struct NsArgs {
    float *syn0;
    float *syn1;
    int32_t dim, stride;
    const int32_t *kept_vid;
    const uint32_t *kept_meta;
    const int32_t *doc_kept;
    int64_t n_docs;
    int32_t doc_len;
    int32_t segs_per_doc;    // work unit: kSegLen consecutive kept centres of one document
    int64_t n_units;
    int64_t first_raw;
    int64_t epoch_base;
    int32_t epoch;
    uint64_t seed;
    const float *alpha_tab;
    int64_t blk0;
    const int32_t *table;
    int32_t log2_size, negative;
    int32_t workers;
    int32_t write_policy;    // bit 0: target rows stored, bit 1: word rows stored (else atomic adds)
    int32_t *queue;
    unsigned long long *stats;   // [3]: kept, pairs, pair-target updates
    // objective: units of kObjSeg consecutive kept centres of one document, one wavefront each
    int32_t obj_segs_per_doc;
    int64_t obj_units;
    double *doc_sum;     // per objective unit
    int64_t *doc_terms;
};

// NT target slots (K + 1 <= NT), rows of NE elements per lane.
template <int NE, int NT>
__global__ __launch_bounds__(kNsWaves *kWave) void k_train_ns(NsArgs a) {
    constexpr int XR = NE <= 5 ? 3 : 2;   // window rows reloaded together in pass 2
    __shared__ float s_g[kNsWaves][kMaxWindow * NT];
    const int lane = lane_id();
    const int wid = static_cast<int>(threadIdx.x / kWave);
    float *G = s_g[wid];
    const int gw = blockIdx.x * kNsWaves + wid;
    if (gw >= a.workers) return;
    uint64_t n_kept = 0, n_pairs = 0, n_upd = 0;
    while (true) {
        int unit = 0;
        if (lane == 0) unit = atomicAdd(a.queue, 1);
        unit = __builtin_amdgcn_readfirstlane(unit);
        if (unit >= a.n_units) break;
        const int doc = unit / a.segs_per_doc;
        const int nk = a.doc_kept[doc];
        const int j0 = (unit - doc * a.segs_per_doc) * kSegLen;
        if (j0 >= nk) continue;
        const int j1 = min(nk, j0 + kSegLen);
        const int64_t base = static_cast<int64_t>(doc) * a.doc_len;
        const int32_t *kv = a.kept_vid + base;
        const uint32_t *km = a.kept_meta + base;
        for (int j = j0; j < j1; ++j) {
            const uint32_t meta = km[j];
            const int v = kv[j];
            const int eff = static_cast<int>(meta >> 16);
            const int lo = max(0, j - eff), hi = min(nk - 1, j + eff);
            const int P = hi - lo;
            ++n_kept;
            if (P <= 0) continue;
            const int64_t raw = a.first_raw + base + static_cast<int64_t>(meta & 0xFFFFu);
            const float alpha = a.alpha_tab[(a.epoch_base + raw) / 10000 - a.blk0];
            int wv = 0;
            if (lane < P) wv = kv[lo + lane + ((lo + lane >= j) ? 1 : 0)];
            const int tg = (lane < NT) ? target_of(lane, v, a.negative, a.seed, raw, a.epoch, a.table, a.log2_size)
                                       : -1;
            const uint64_t tmask = __ballot(lane < NT && tg >= 0);
            // targets (snapshot) and their accumulated change
            float y[NT][NE], dy[NT][NE];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int n = __builtin_amdgcn_readlane(tg, t);
                buf_load_row<NE>(y[t], row_rsrc(a.syn1, n >= 0 ? n : 0, a.stride, n >= 0 ? a.dim * 4 : 0), lane);
#pragma unroll
                for (int i = 0; i < NE; ++i) dy[t][i] = 0.0f;
            }
            // pass 1: gradients of every (window word, target), the targets' change. Window rows alternate
            // between two register sets, each loaded one row ahead of its use (empty ranges past the
            // window), so that a row's load is in flight while the row before it is used.
            const int row = lane >> 4;
            auto step = [&](const float(&x)[NE], int p) {
#pragma unroll
                for (int c = 0; c < (NT + 3) / 4; ++c) {
                    const float z = reduce4(dot_slot<NE, NT>(x, y, 4 * c), dot_slot<NE, NT>(x, y, 4 * c + 1),
                                            dot_slot<NE, NT>(x, y, 4 * c + 2), dot_slot<NE, NT>(x, y, 4 * c + 3));
                    const int t = 4 * c + row;
                    const float label = (t == 0) ? 1.0f : 0.0f;
                    const float f = __builtin_amdgcn_rcpf(1.0f + __expf(-z));
                    const float g = ((tmask >> t) & 1ull) ? (label - f) * alpha : 0.0f;
                    if ((lane & 15) == 0 && t < NT) G[p * NT + t] = g;
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj) {
                        if (4 * c + jj < NT) {
                            const float gj = bcast(g, 16 * jj);
#pragma unroll
                            for (int i = 0; i < NE; ++i) dy[4 * c + jj][i] = fmaf(gj, x[i], dy[4 * c + jj][i]);
                        }
                    }
                }
            };
            auto window_row = [&](int p) {
                const bool in = p < P;
                const int w = __builtin_amdgcn_readlane(wv, min(p, kWave - 1));
                return row_rsrc(a.syn0, in ? w : 0, a.stride, in ? a.dim * 4 : 0);
            };
            float xa[NE], xb[NE];
            buf_load_row<NE>(xa, window_row(0), lane);
            for (int p = 0; p < P; p += 2) {
                buf_load_row<NE>(xb, window_row(p + 1), lane);
                step(xa, p);
                buf_load_row<NE>(xa, window_row(p + 2), lane);
                if (p + 1 < P) step(xb, p + 1);
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            // pass 2: each window word's change from the gradients and the unchanged targets. With
            // write_policy bit 1 the first occurrence of a word stores its row plus the change (a reload,
            // XR rows at a time), later occurrences in the same window add theirs atomically.
            for (int p0 = 0; p0 < P; p0 += XR) {
                float cur[XR][NE], dx[XR][NE];
                bool st[XR];
#pragma unroll
                for (int r = 0; r < XR; ++r) {
                    const int p = p0 + r;
                    st[r] = false;
                    if (p < P) {
                        const int w = __builtin_amdgcn_readlane(wv, p);
                        const bool dup = __ballot(lane < p && wv == w) != 0ull;
                        st[r] = (a.write_policy & 2) && !dup;
                        if (st[r]) load_row<NE>(cur[r], a.syn0 + static_cast<int64_t>(w) * a.stride, lane, a.dim);
                    }
                }
#pragma unroll
                for (int r = 0; r < XR; ++r) {
                    const int p = p0 + r;
                    if (p < P) {
#pragma unroll
                        for (int i = 0; i < NE; ++i) dx[r][i] = 0.0f;
#pragma unroll
                        for (int t = 0; t < NT; ++t) {
                            const float g = G[p * NT + t];
#pragma unroll
                            for (int i = 0; i < NE; ++i) dx[r][i] = fmaf(g, y[t][i], dx[r][i]);
                        }
                        float *row_p = a.syn0 + static_cast<int64_t>(__builtin_amdgcn_readlane(wv, p)) * a.stride;
                        if (st[r]) {
#pragma unroll
                            for (int i = 0; i < NE; ++i) cur[r][i] += dx[r][i];
                            store_row<NE>(row_p, cur[r], lane, a.dim);
                        } else {
                            atomic_add_row<NE>(row_p, dx[r], lane, a.dim);
                        }
                    }
                }
            }
            // targets: with write_policy bit 0 the first slot of a word stores the snapshot plus its change
            // (no reload), a repeated negative adds its change atomically
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int n = __builtin_amdgcn_readlane(tg, t);
                if (n >= 0) {
                    float *row_n = a.syn1 + static_cast<int64_t>(n) * a.stride;
                    const bool dup = __ballot(lane < t && tg == n) != 0ull;
                    if ((a.write_policy & 1) && !dup) {
#pragma unroll
                        for (int i = 0; i < NE; ++i) y[t][i] += dy[t][i];
                        store_row<NE>(row_n, y[t], lane, a.dim);
                    } else {
                        atomic_add_row<NE>(row_n, dy[t], lane, a.dim);
                    }
                }
            }
            __builtin_amdgcn_wave_barrier();
            n_pairs += P;
            n_upd += static_cast<uint64_t>(P) * __popcll(tmask);
        }
    }
    if (lane == 0 && n_kept) {
        atomicAdd(&a.stats[0], static_cast<unsigned long long>(n_kept));
        atomicAdd(&a.stats[1], static_cast<unsigned long long>(n_pairs));
        atomicAdd(&a.stats[2], static_cast<unsigned long long>(n_upd));
    }
}

// Objective over the sampler's pairs: one wavefront per document, per-document sums.
template <int NE, int NT>
__global__ __launch_bounds__(256) void k_ns_objective(NsArgs a) {
    const int lane = lane_id();
    const int64_t wave0 = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * blockDim.x / kWave;
    for (int64_t u = wave0; u < a.obj_units; u += nwaves) {
        const int64_t d = u / a.obj_segs_per_doc;
        const int nk = a.doc_kept[d];
        const int j0 = static_cast<int>(u - d * a.obj_segs_per_doc) * kObjSeg;
        const int j1 = min(nk, j0 + kObjSeg);
        const int64_t base = d * a.doc_len;
        double acc = 0.0;
        int64_t terms = 0;
        for (int j = j0; j < j1; ++j) {
            const uint32_t meta = a.kept_meta[base + j];
            const int v = a.kept_vid[base + j];
            const int eff = static_cast<int>(meta >> 16);
            const int lo = max(0, j - eff), hi = min(nk - 1, j + eff);
            const int P = hi - lo;
            if (P <= 0) continue;
            const int64_t raw = a.first_raw + base + static_cast<int64_t>(meta & 0xFFFFu);
            const int tg = (lane < NT) ? target_of(lane, v, a.negative, a.seed, raw, a.epoch, a.table, a.log2_size)
                                       : -1;
            const uint64_t tmask = __ballot(lane < NT && tg >= 0);
            float y[NT][NE];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int n = __builtin_amdgcn_readlane(tg, t);
                if (n >= 0) load_row<NE>(y[t], a.syn1 + static_cast<int64_t>(n) * a.stride, lane, a.dim);
                else {
#pragma unroll
                    for (int i = 0; i < NE; ++i) y[t][i] = 0.0f;
                }
            }
            const int row = lane >> 4;
            for (int p = 0; p < P; ++p) {
                const int w = a.kept_vid[base + lo + p + ((lo + p >= j) ? 1 : 0)];
                float x[NE];
                load_row<NE>(x, a.syn0 + static_cast<int64_t>(w) * a.stride, lane, a.dim);
#pragma unroll
                for (int c = 0; c < (NT + 3) / 4; ++c) {
                    const float z = reduce4(dot_slot<NE, NT>(x, y, 4 * c), dot_slot<NE, NT>(x, y, 4 * c + 1),
                                            dot_slot<NE, NT>(x, y, 4 * c + 2), dot_slot<NE, NT>(x, y, 4 * c + 3));
                    const int t = 4 * c + row;
                    if ((lane & 15) == 0 && t < NT && ((tmask >> t) & 1ull)) {
                        const double u = t == 0 ? static_cast<double>(z) : -static_cast<double>(z);
                        acc += log_sigmoid(u);
                    }
                }
            }
            terms += static_cast<int64_t>(P) * __popcll(tmask);
        }
        acc = wave_sum(acc);
        if (lane == 0) {
            a.doc_sum[u] = acc;
            a.doc_terms[u] = terms;
        }
    }
}

__global__ __launch_bounds__(1024) void k_sum_docs_ns(const double *__restrict__ s, const int64_t *__restrict__ t,
                                                      int64_t n, double *__restrict__ out_s,
                                                      int64_t *__restrict__ out_t) {
    __shared__ double ss[1024];
    __shared__ int64_t st[1024];
    double x = 0.0;
    int64_t y = 0;
    for (int64_t i = threadIdx.x; i < n; i += 1024) {
        x += s[i];
        y += t[i];
    }
    ss[threadIdx.x] = x;
    st[threadIdx.x] = y;
    __syncthreads();
    for (int k = 512; k > 0; k >>= 1) {
        if (threadIdx.x < k) {
            ss[threadIdx.x] += ss[threadIdx.x + k];
            st[threadIdx.x] += st[threadIdx.x + k];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        *out_s = ss[0];
        *out_t = st[0];
    }
}

// exclusive scan of per-document kept counts (int32) into int64 offsets (one workgroup)
__global__ __launch_bounds__(kScanThreads) void k_scan_kept_ns(const int32_t *__restrict__ in, int64_t n,
                                                               int64_t *__restrict__ out) {
    block_exclusive_scan(in, n, out);
}

// Test hook: every kept centre's negatives (stream order) and their checksum.
__global__ __launch_bounds__(256) void k_ns_negatives(NsArgs a, const int64_t *__restrict__ doc_off,
                                                      int32_t *__restrict__ out, int64_t cap,
                                                      unsigned long long *__restrict__ checksum) {
    const int lane = lane_id();
    const int64_t wave0 = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * blockDim.x / kWave;
    const int K = a.negative;
    uint64_t cs = 0;
    for (int64_t d = wave0; d < a.n_docs; d += nwaves) {
        const int nk = a.doc_kept[d];
        const int64_t base = d * a.doc_len;
        for (int j = 0; j < nk; ++j) {
            const uint32_t meta = a.kept_meta[base + j];
            const int v = a.kept_vid[base + j];
            const int64_t raw = a.first_raw + base + static_cast<int64_t>(meta & 0xFFFFu);
            if (lane < K) {
                const int n = target_of(lane + 1, v, K, a.seed, raw, a.epoch, a.table, a.log2_size);
                const int64_t c = doc_off[d] + j;
                if (c < cap) out[c * K + lane] = n;
                cs += fmix64(static_cast<uint64_t>(raw) * 0x9E3779B97F4A7C15ull +
                             (static_cast<uint64_t>(lane) << 32) + static_cast<uint64_t>(static_cast<int64_t>(n) + 1));
            }
        }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) cs += __shfl_xor(cs, m, kWave);
    if (lane == 0) atomicAdd(checksum, static_cast<unsigned long long>(cs));
}

__global__ void k_zero_ns(int32_t *queue, unsigned long long *stats) {
    if (threadIdx.x == 0 && queue) *queue = 0;
    if (threadIdx.x < 4) stats[threadIdx.x] = 0;
}

__global__ void k_write_ns_stats(const int64_t *totals, const unsigned long long *tstats, int64_t *out) {
    if (threadIdx.x == 0) {
        out[0] = totals[0];
        out[1] = totals[1];
        out[2] = static_cast<int64_t>(tstats[0]);
        out[3] = static_cast<int64_t>(tstats[1]);
        out[4] = static_cast<int64_t>(tstats[2]);
    }
}

using NsFn = void (*)(NsArgs);

template <int NT>
NsFn pick_by_ne(int ne, bool objective) {
    if (ne <= 1) return objective ? k_ns_objective<1, NT> : k_train_ns<1, NT>;
    if (ne <= 2) return objective ? k_ns_objective<2, NT> : k_train_ns<2, NT>;
    if (ne <= 4) return objective ? k_ns_objective<4, NT> : k_train_ns<4, NT>;
    if (ne <= 5) return objective ? k_ns_objective<5, NT> : k_train_ns<5, NT>;
    if constexpr (NT <= 8) return objective ? k_ns_objective<8, NT> : k_train_ns<8, NT>;
    return nullptr;   // more than 7 negatives above 320 columns: refused by the caller's checks
}

// dim <= 512; negative <= 11, and <= 7 above 320 columns (checked by the caller)
NsFn pick_ns(int dim, int negative, bool objective) {
    const int ne = (dim + kWave - 1) / kWave;
    if (negative + 1 <= 4) return pick_by_ne<4>(ne, objective);
    if (negative + 1 <= 6) return pick_by_ne<6>(ne, objective);
    if (negative + 1 <= 8) return pick_by_ne<8>(ne, objective);
    return pick_by_ne<12>(ne, objective);
}

NsArgs ns_args(const w2v_model *m, const int32_t *table, int32_t log2_size, const w2v_params *p,
               const SampleBufs &b, int64_t n_tokens) {
    NsArgs a{};
    a.syn0 = m->syn0;
    a.syn1 = m->syn1;
    a.dim = m->dim;
    a.stride = m->row_stride;
    a.kept_vid = b.kept_vid;
    a.kept_meta = b.kept_meta;
    a.doc_kept = b.doc_kept;
    a.n_docs = n_tokens > 0 ? ceil_div(n_tokens, p->doc_len) : 0;
    a.doc_len = p->doc_len;
    a.segs_per_doc = segs_per_doc(p->doc_len);
    a.n_units = a.n_docs * a.segs_per_doc;
    a.first_raw = p->first_raw_index;
    a.epoch_base = static_cast<int64_t>(p->epoch) * p->corpus_tokens;
    a.epoch = p->epoch;
    a.seed = p->seed;
    a.table = table;
    a.log2_size = log2_size;
    a.negative = p->negative;
    a.write_policy = p->write_policy;
    return a;
}

}  // namespace

// ------------------------------------------------------------------ host side
size_t noise_workspace_bytes(int32_t V) {
    Carve c;
    c.take<int64_t>(static_cast<size_t>(V) + 1);
    c.take<int64_t>(static_cast<size_t>(V) + 1);
    return c.used();
}

int run_noise_table(const int64_t *vocab_counts, int32_t V, int32_t log2_size, int32_t *table,
                    int64_t *total_host, void *workspace, hipStream_t s) {
    Carve c(workspace);
    int64_t *w = c.take<int64_t>(static_cast<size_t>(V) + 1);
    int64_t *pre = c.take<int64_t>(static_cast<size_t>(V) + 1);
    const unsigned g = static_cast<unsigned>(std::min<int64_t>(ceil_div(V, 256), 4096));
    k_noise_weights<<<g, 256, 0, s>>>(vocab_counts, V, w);
    W2V_LAUNCH_CHECK("k_noise_weights");
    k_scan_weights<<<1, kScanThreads, 0, s>>>(w, V, pre);
    W2V_LAUNCH_CHECK("k_scan_weights");
    int64_t tot = 0;
    W2V_HIP(hipMemcpyAsync(&tot, pre + V, sizeof(tot), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipStreamSynchronize(s));
    *total_host = tot;
    if (tot < 1 || tot >= (int64_t(1) << (63 - log2_size)))   // entry arithmetic Q[v] 2^L stays below 2^63
        return fail(W2V_E_RANGE, "total noise weight " + std::to_string(tot) + " outside [1, 2^(63 - log2_size))");
    const unsigned gf = static_cast<unsigned>(std::min<int64_t>(ceil_div(V, 4), 16LL * device_cu_count()));
    k_noise_fill<<<gf, 256, 0, s>>>(pre, V, log2_size, table);
    W2V_LAUNCH_CHECK("k_noise_fill");
    return W2V_OK;
}

size_t ns_train_extra_bytes() {
    Carve c;
    c.take<int32_t>(4);
    c.take<unsigned long long>(4);
    return c.used();
}

int launch_train_ns(const w2v_model *m, const int32_t *table, int32_t log2_size, const w2v_params *p,
                    const SampleBufs &b, int64_t n_tokens, const float *alpha_tab, int64_t blk0, Carve &c,
                    hipEvent_t ev0, hipEvent_t ev1, int64_t *stats, hipStream_t s) {
    NsArgs a = ns_args(m, table, log2_size, p, b, n_tokens);
    a.alpha_tab = alpha_tab;
    a.blk0 = blk0;
    a.queue = c.take<int32_t>(4);
    a.stats = c.take<unsigned long long>(4);
    NsFn fn = pick_ns(m->dim, p->negative, false);
    if (!fn) return fail(W2V_E_ARG, "no kernel variant for this dim and number of negatives");
    int per_cu = 0;
    W2V_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(fn),
                                                         kNsWaves * kWave, 0));
    int64_t grid = static_cast<int64_t>(device_cu_count()) * std::max(1, per_cu);
    if (p->workers > 0) grid = ceil_div(p->workers, kNsWaves);
    // at least kMinUnits work units per wavefront
    constexpr int kMinUnits = 8;
    grid = std::max<int64_t>(1, std::min<int64_t>(grid, ceil_div(a.n_units, int64_t(kNsWaves) * kMinUnits)));
    a.workers = p->workers > 0 ? p->workers : static_cast<int32_t>(grid * kNsWaves);
    record_train_launch(static_cast<int>(grid), a.workers, reinterpret_cast<const void *>(fn), kNsWaves * kWave, 0);
    k_zero_ns<<<1, 64, 0, s>>>(a.queue, a.stats);
    W2V_LAUNCH_CHECK("k_zero_ns");
    if (ev0) W2V_HIP(hipEventRecord(ev0, s));
    hipLaunchKernelGGL(fn, dim3(static_cast<unsigned>(grid)), dim3(kNsWaves * kWave), 0, s, a);
    W2V_LAUNCH_CHECK("k_train_ns");
    if (ev1) W2V_HIP(hipEventRecord(ev1, s));
    if (stats) {
        k_write_ns_stats<<<1, 64, 0, s>>>(b.totals, a.stats, stats);
        W2V_LAUNCH_CHECK("k_write_ns_stats");
    }
    return W2V_OK;
}

size_t ns_objective_extra_bytes(int64_t n_docs, int32_t doc_len) {
    const int64_t units = n_docs * obj_segs_per_doc(doc_len);
    Carve c;
    c.take<double>(static_cast<size_t>(units));
    c.take<int64_t>(static_cast<size_t>(units));
    c.take<double>(1);
    c.take<int64_t>(1);
    return c.used();
}

int run_ns_objective(const w2v_model *m, const int32_t *table, int32_t log2_size, const w2v_params *p,
                     const SampleBufs &b, int64_t n_tokens, Carve &c, double *sum_host, int64_t *n_pairs_host,
                     int64_t *n_terms_host, hipStream_t s) {
    NsArgs a = ns_args(m, table, log2_size, p, b, n_tokens);
    const int64_t n_docs = std::max<int64_t>(1, ceil_div(n_tokens, p->doc_len));
    a.obj_segs_per_doc = obj_segs_per_doc(p->doc_len);
    a.obj_units = a.n_docs * a.obj_segs_per_doc;
    const int64_t units_cap = n_docs * a.obj_segs_per_doc;
    a.doc_sum = c.take<double>(static_cast<size_t>(units_cap));
    a.doc_terms = c.take<int64_t>(static_cast<size_t>(units_cap));
    double *out = c.take<double>(1);
    int64_t *out_t = c.take<int64_t>(1);
    if (a.n_docs > 0) {
        // one unit per wavefront: the hardware hands out workgroups as others finish
        const unsigned grid = static_cast<unsigned>(std::min<int64_t>(ceil_div(a.obj_units, 4), INT32_MAX));
        NsFn fn = pick_ns(m->dim, p->negative, true);
        if (!fn) return fail(W2V_E_ARG, "no kernel variant for this dim and number of negatives");
        hipLaunchKernelGGL(fn, dim3(grid), dim3(256), 0, s, a);
        W2V_LAUNCH_CHECK("k_ns_objective");
        k_sum_docs_ns<<<1, 1024, 0, s>>>(a.doc_sum, a.doc_terms, a.obj_units, out, out_t);
        W2V_LAUNCH_CHECK("k_sum_docs_ns");
    }
    double hs = 0.0;
    int64_t ht = 0;
    int64_t tot[4] = {0, 0, 0, 0};
    if (a.n_docs > 0) {
        W2V_HIP(hipMemcpyAsync(&hs, out, sizeof(hs), hipMemcpyDeviceToHost, s));
        W2V_HIP(hipMemcpyAsync(&ht, out_t, sizeof(ht), hipMemcpyDeviceToHost, s));
    }
    W2V_HIP(hipMemcpyAsync(tot, b.totals, sizeof(tot), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipStreamSynchronize(s));
    *sum_host = hs;
    *n_pairs_host = tot[3];
    if (n_terms_host) *n_terms_host = ht;
    return W2V_OK;
}

size_t ns_negatives_extra_bytes(int64_t n_docs) {
    Carve c;
    c.take<int64_t>(static_cast<size_t>(n_docs));
    c.take<unsigned long long>(2);
    return c.used();
}

int run_ns_negatives(const w2v_params *p, const int32_t *table, int32_t log2_size, const SampleBufs &b,
                     int64_t n_tokens, Carve &c, int32_t *out, int64_t cap, int64_t *n_kept_host,
                     uint64_t *checksum_host, hipStream_t s) {
    w2v_model dummy{};
    NsArgs a = ns_args(&dummy, table, log2_size, p, b, n_tokens);
    const int64_t n_docs = std::max<int64_t>(1, ceil_div(n_tokens, p->doc_len));
    int64_t *doc_off = c.take<int64_t>(static_cast<size_t>(n_docs));
    unsigned long long *cs = c.take<unsigned long long>(2);
    k_zero_ns<<<1, 64, 0, s>>>(nullptr, cs);
    W2V_LAUNCH_CHECK("k_zero_ns");
    if (a.n_docs > 0) {
        k_scan_kept_ns<<<1, kScanThreads, 0, s>>>(b.doc_kept, a.n_docs, doc_off);
        W2V_LAUNCH_CHECK("k_scan_kept_ns");
        const unsigned grid =
            static_cast<unsigned>(std::min<int64_t>(ceil_div(a.n_docs, 4), 16LL * device_cu_count()));
        k_ns_negatives<<<grid, 256, 0, s>>>(a, doc_off, out, out ? cap : 0, cs);
        W2V_LAUNCH_CHECK("k_ns_negatives");
    }
    int64_t tot[4];
    unsigned long long hcs = 0;
    W2V_HIP(hipMemcpyAsync(tot, b.totals, sizeof(tot), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipMemcpyAsync(&hcs, cs, sizeof(hcs), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipStreamSynchronize(s));
    *n_kept_host = tot[2];
    *checksum_host = hcs;
    return W2V_OK;
}

}  // namespace w2v
