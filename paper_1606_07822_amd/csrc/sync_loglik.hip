// Deterministic synchronous training mode and the HS log-likelihood evaluator.
//
// Synchronous mode: every gradient of a batch of B consecutive kept centres is
// taken against the model as it stood at the start of the batch; the changes
// are summed exactly as int64 fixed point (value * 2^kFrac, integer atomics
// commute, so the sums do not depend on scheduling) and applied after the
// batch: row = row + (float)(sum * 2^-kFrac).
//
// Log-likelihood: sum over the sampler's pairs (v, w) of
// log P(v | syn0[w]) = sum_j log sigmoid((1 - 2 t_j) syn0[w] . syn1[n_j]);
// dot products in fp32, logarithms and all sums in fp64, in a fixed order.
// CBOW's objective: the same hierarchical softmax (§2) with the mean h of the
// window words' vectors as input, one term log P(v | h) per centre that has a
// window; h and its dot products in fp64.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "w2v_internal.h"
#include "w2v_scan.h"

namespace w2v {

constexpr int kFrac = 40;   // fixed-point fraction bits of the synchronous-mode sums

struct SyncArgs {
    const float *syn0;
    const float *syn1;
    int32_t V, dim, stride;
    const uint8_t *codelen;
    const uint64_t *code;
    const int32_t *point_off;
    const int32_t *points;
    const int32_t *kept_vid;
    const uint32_t *kept_meta;
    const int32_t *doc_kept;
    const int64_t *kept_off;   // exclusive prefix of doc_kept
    int64_t n_docs;
    int32_t doc_len;
    int64_t first_raw, epoch_base;
    const float *alpha_tab;
    int64_t blk0;
    int64_t c_lo, c_hi;        // global kept indices of this batch
    unsigned long long *d0;    // [V][dim] fixed-point deltas of syn0
    unsigned long long *d1;    // [V-1][dim] of syn1
    int32_t *flag0, *flag1;    // touched rows
    int32_t *list0, *list1;
    int32_t *cnt;              // [2] list lengths
    unsigned long long *stats; // kept, pairs, nodes
};

namespace {

__device__ __forceinline__ unsigned long long to_fixed(double v) {
    return static_cast<unsigned long long>(__double2ll_rn(ldexp(v, kFrac)));
}

__device__ __forceinline__ void touch(int32_t *flag, int32_t *list, int32_t *cnt, int32_t r) {
    if (atomicExch(&flag[r], 1) == 0) list[atomicAdd(cnt, 1)] = r;
}

template <int NE>
__global__ __launch_bounds__(256) void k_sync_grad(SyncArgs a) {
    const int lane = lane_id();
    const int64_t gi = a.c_lo + (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    if (gi >= a.c_hi) return;
    // document of kept centre gi: last d with kept_off[d] <= gi
    int64_t lo = 0, hi = a.n_docs - 1;
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) >> 1;
        if (a.kept_off[mid] <= gi) lo = mid; else hi = mid - 1;
    }
    const int64_t d = lo;
    const int j = static_cast<int>(gi - a.kept_off[d]);
    const int nk = a.doc_kept[d];
    const int64_t base = d * a.doc_len;
    const uint32_t meta = a.kept_meta[base + j];
    const int v = a.kept_vid[base + j];
    const int eff = static_cast<int>(meta >> 16);
    const int clo = max(0, j - eff), chi = min(nk - 1, j + eff);
    const int P = chi - clo;
    const int len = a.codelen[v];
    if (lane == 0) {
        atomicAdd(&a.stats[0], 1ull);
        atomicAdd(&a.stats[1], static_cast<unsigned long long>(P));
        atomicAdd(&a.stats[2], static_cast<unsigned long long>(P) * len);
    }
    if (P == 0) return;
    const int64_t g = a.epoch_base + a.first_raw + base + static_cast<int64_t>(meta & 0xFFFFu);
    const float alpha = a.alpha_tab[g / 10000 - a.blk0];
    const uint64_t code = a.code[v];
    const int my_pt = (lane < len) ? a.points[a.point_off[v] + lane] : 0;
    for (int p = 0; p < P; ++p) {
        const int c = clo + p + ((clo + p >= j) ? 1 : 0);
        const int w = a.kept_vid[base + c];
        float x[NE];
#pragma unroll
        for (int i = 0; i < NE; ++i) {
            const int col = lane + i * kWave;
            x[i] = col < a.dim ? a.syn0[static_cast<int64_t>(w) * a.stride + col] : 0.0f;
        }
        for (int jn = 0; jn < len; ++jn) {
            const int n = __builtin_amdgcn_readlane(my_pt, jn);
            const float t = static_cast<float>((code >> jn) & 1ull);
            float y[NE];
            float s = 0.0f;
#pragma unroll
            for (int i = 0; i < NE; ++i) {
                const int col = lane + i * kWave;
                y[i] = col < a.dim ? a.syn1[static_cast<int64_t>(n) * a.stride + col] : 0.0f;
                s = fmaf(x[i], y[i], s);
            }
            const float z = wave_sum(s);
            const float f = 1.0f / (1.0f + expf(-z));
            const float gr = (1.0f - t - f) * alpha;
            if (lane == 0) touch(a.flag1, a.list1, a.cnt + 1, n);
#pragma unroll
            for (int i = 0; i < NE; ++i) {
                const int col = lane + i * kWave;
                if (col < a.dim) {
                    atomicAdd(&a.d1[static_cast<int64_t>(n) * a.dim + col],
                              to_fixed(static_cast<double>(gr) * static_cast<double>(x[i])));
                    atomicAdd(&a.d0[static_cast<int64_t>(w) * a.dim + col],
                              to_fixed(static_cast<double>(gr) * static_cast<double>(y[i])));
                }
            }
        }
        if (lane == 0) touch(a.flag0, a.list0, a.cnt, w);
    }
}

// one wave per touched row: row += (float)(delta 2^-40); clear delta and flag
__global__ __launch_bounds__(256) void k_sync_apply(float *w, int32_t stride, int32_t dim, unsigned long long *dl,
                                                    int32_t *flag, const int32_t *list, const int32_t *cnt) {
    const int lane = lane_id();
    const int n = *cnt;
    const int nw = gridDim.x * blockDim.x / kWave;
    for (int k = (blockIdx.x * blockDim.x + threadIdx.x) / kWave; k < n; k += nw) {
        const int r = list[k];
        for (int col = lane; col < dim; col += kWave) {
            unsigned long long *q = &dl[static_cast<int64_t>(r) * dim + col];
            const double dv = ldexp(static_cast<double>(static_cast<long long>(*q)), -kFrac);
            float *x = &w[static_cast<int64_t>(r) * stride + col];
            *x = *x + static_cast<float>(dv);
            *q = 0ull;
        }
        if (lane == 0) flag[r] = 0;
    }
}

__global__ void k_reset_counts(int32_t *cnt) {
    if (threadIdx.x < 2) cnt[threadIdx.x] = 0;
}

__global__ void k_zero_u64_range(unsigned long long *p, int64_t n) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0;
}
__global__ void k_zero_i32_range(int32_t *p, int64_t n) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0;
}

// exclusive scan of per-document kept counts (int32) into int64 offsets
__global__ __launch_bounds__(kScanThreads) void k_scan_kept(const int32_t *__restrict__ in, int64_t n,
                                                            int64_t *__restrict__ out) {
    block_exclusive_scan(in, n, out);
}

using SyncFn = void (*)(SyncArgs);
SyncFn pick_sync(int dim) {
    const int ne = (dim + kWave - 1) / kWave;
    if (ne <= 1) return k_sync_grad<1>;
    if (ne <= 2) return k_sync_grad<2>;
    if (ne <= 4) return k_sync_grad<4>;
    if (ne <= 5) return k_sync_grad<5>;
    if (ne <= 8) return k_sync_grad<8>;
    return k_sync_grad<16>;
}

}  // namespace

size_t sync_extra_bytes(int32_t V, int32_t dim, int64_t n_docs) {
    Carve c;
    c.take<int64_t>(static_cast<size_t>(n_docs));                        // kept_off
    c.take<unsigned long long>(static_cast<size_t>(V) * dim);            // d0
    c.take<unsigned long long>(static_cast<size_t>(V) * dim);            // d1
    c.take<int32_t>(static_cast<size_t>(V) * 4);                         // flags, lists
    c.take<int32_t>(2);
    return c.used();
}

int run_train_sync(const w2v_model *m, const w2v_params *p, const SampleBufs &b, int64_t n_tokens, Carve &c,
                   const float *alpha_tab, int64_t blk0, unsigned long long *tstats, hipStream_t s) {
    const int64_t n_docs = std::max<int64_t>(1, ceil_div(n_tokens, p->doc_len));
    SyncArgs a{};
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
    int64_t *kept_off = c.take<int64_t>(static_cast<size_t>(n_docs));
    a.kept_off = kept_off;
    a.n_docs = ceil_div(n_tokens, p->doc_len);
    a.doc_len = p->doc_len;
    a.first_raw = p->first_raw_index;
    a.epoch_base = static_cast<int64_t>(p->epoch) * p->corpus_tokens;
    a.alpha_tab = alpha_tab;
    a.blk0 = blk0;
    a.d0 = c.take<unsigned long long>(static_cast<size_t>(m->V) * m->dim);
    a.d1 = c.take<unsigned long long>(static_cast<size_t>(m->V) * m->dim);
    int32_t *fl = c.take<int32_t>(static_cast<size_t>(m->V) * 4);
    a.flag0 = fl;
    a.flag1 = fl + m->V;
    a.list0 = fl + 2 * static_cast<size_t>(m->V);
    a.list1 = fl + 3 * static_cast<size_t>(m->V);
    a.cnt = c.take<int32_t>(2);
    a.stats = tstats;
    const unsigned zg = static_cast<unsigned>(std::min<int64_t>(8192, ceil_div(static_cast<int64_t>(m->V) * m->dim, 256)));
    k_zero_u64_range<<<zg, 256, 0, s>>>(a.d0, static_cast<int64_t>(m->V) * m->dim);
    k_zero_u64_range<<<zg, 256, 0, s>>>(a.d1, static_cast<int64_t>(m->V) * m->dim);
    k_zero_i32_range<<<static_cast<unsigned>(ceil_div(2LL * m->V, 256)), 256, 0, s>>>(fl, 2LL * m->V);
    k_reset_counts<<<1, 64, 0, s>>>(a.cnt);
    if (n_tokens <= 0) return W2V_OK;
    k_scan_kept<<<1, kScanThreads, 0, s>>>(b.doc_kept, a.n_docs, kept_off);
    W2V_LAUNCH_CHECK("sync setup");
    int64_t tot[4];
    W2V_HIP(hipMemcpyAsync(tot, b.totals, sizeof(tot), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipStreamSynchronize(s));
    const int64_t kept = tot[2];
    SyncFn fn = pick_sync(m->dim);
    const unsigned ag = static_cast<unsigned>(std::max(1, device_cu_count() * 4));
    for (int64_t lo = 0; lo < kept; lo += p->sync_batch) {
        a.c_lo = lo;
        a.c_hi = std::min<int64_t>(kept, lo + p->sync_batch);
        const unsigned g = static_cast<unsigned>(ceil_div(a.c_hi - a.c_lo, 4));
        hipLaunchKernelGGL(fn, dim3(g), dim3(256), 0, s, a);
        k_sync_apply<<<ag, 256, 0, s>>>(m->syn0, m->row_stride, m->dim, a.d0, a.flag0, a.list0, a.cnt);
        k_sync_apply<<<ag, 256, 0, s>>>(m->syn1, m->row_stride, m->dim, a.d1, a.flag1, a.list1, a.cnt + 1);
        k_reset_counts<<<1, 64, 0, s>>>(a.cnt);
        W2V_LAUNCH_CHECK("sync batch");
    }
    return W2V_OK;
}

// ------------------------------------------------------------- log-likelihood
namespace {

// log sigmoid(u) = min(u, 0) - log(1 + exp(-|u|)): the same operations as the two one-sided forms, without
// a branch (lanes of both signs would run both sides)
__device__ __forceinline__ double log_sigmoid(double u) {
    return fmin(u, 0.0) - log1p(exp(-fabs(u)));
}

// Held-out evaluation work units: kLLSeg consecutive kept centres of a document, one wavefront each.
// Short units keep the read-only walk's latency spread over many wavefronts (8: 4.2 ms for the 1e6-token
// held-out corpus at V = 1M, d = 300; the training kernel's 128-centre units: 8.4 ms).
constexpr int kLLSeg = 8;
inline int32_t ll_segs_per_doc(int32_t doc_len) { return static_cast<int32_t>(ceil_div(doc_len, kLLSeg)); }

struct LLArgs {
    const float *syn0;
    const float *syn1;
    int32_t dim, stride;
    const uint8_t *codelen;
    const uint64_t *code;
    const int32_t *point_off;
    const int32_t *points;
    const int32_t *kept_vid;
    const uint32_t *kept_meta;
    const int32_t *doc_kept;
    int64_t n_units;        // work units: kLLSeg consecutive kept centres of one document
    int32_t segs_per_doc;
    int32_t doc_len;
    double *unit_ll;
    int64_t *unit_nodes;
    int64_t *unit_terms;    // CBOW: centres with a window, per unit
};

// One wavefront per work unit (a fixed assignment, so the sums are the same from run to run).
// Per centre the path is walked once for a group of up to G window words: four node rows at a
// time (the next four loaded while the current ones are used), the G x 4 dot products reduced
// four at a time; lane n collects the dot products of path node n, and takes the log-sigmoids
// of its node for every pair of the group in fp64.
template <int NE, int G>
__global__ __launch_bounds__(256) void k_loglik(LLArgs a) {
    const int lane = lane_id();
    const int64_t wave0 = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * blockDim.x / kWave;
    for (int64_t u = wave0; u < a.n_units; u += nwaves) {
        const int64_t d = u / a.segs_per_doc;
        const int nk = a.doc_kept[d];
        const int j0 = static_cast<int>(u - d * a.segs_per_doc) * kLLSeg;
        const int j1 = min(nk, j0 + kLLSeg);
        const int64_t base = d * a.doc_len;
        double acc = 0.0;
        int64_t nodes = 0;
        for (int j = j0; j < j1; ++j) {
            const int v = a.kept_vid[base + j];
            const int eff = static_cast<int>(a.kept_meta[base + j] >> 16);
            const int clo = max(0, j - eff), chi = min(nk - 1, j + eff);
            const int P = chi - clo;
            const int len = a.codelen[v];
            const uint64_t code = a.code[v];
            const int my_pt = (lane < len) ? a.points[a.point_off[v] + lane] : 0;
            // lane q: the q-th window word (centre excluded)
            const int cq = clo + lane + ((clo + lane >= j) ? 1 : 0);
            const int my_w = (lane < P) ? a.kept_vid[base + cq] : 0;
            const double sign = ((code >> min(lane, 63)) & 1ull) ? -1.0 : 1.0;
            for (int g0 = 0; g0 < P; g0 += G) {
                const int nx = min(G, P - g0);
                float x[G][NE], mine[G];
#pragma unroll
                for (int p = 0; p < G; ++p) {
                    const int w = __builtin_amdgcn_readlane(my_w, min(g0 + p, kWave - 1));
                    buf_load_row<NE>(x[p], row_rsrc(const_cast<float *>(a.syn0), p < nx ? w : 0, a.stride,
                                                    p < nx ? a.dim * 4 : 0), lane);
                    mine[p] = 0.0f;
                }
                float y[4][NE], yn[4][NE];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int n = __builtin_amdgcn_readlane(my_pt, min(r, kWave - 1));
                    buf_load_row<NE>(y[r], row_rsrc(const_cast<float *>(a.syn1), r < len ? n : 0, a.stride,
                                                    r < len ? a.dim * 4 : 0), lane);
                }
                for (int c0 = 0; c0 < len; c0 += 4) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int c = c0 + 4 + r;
                        const int n = __builtin_amdgcn_readlane(my_pt, min(c, kWave - 1));
                        buf_load_row<NE>(yn[r], row_rsrc(const_cast<float *>(a.syn1), c < len ? n : 0, a.stride,
                                                         c < len ? a.dim * 4 : 0), lane);
                    }
#pragma unroll
                    for (int p = 0; p < G; ++p) {
                        if (p < nx) {
                            const float z = reduce4(dot_partial<NE>(x[p], y[0]), dot_partial<NE>(x[p], y[1]),
                                                    dot_partial<NE>(x[p], y[2]), dot_partial<NE>(x[p], y[3]));
#pragma unroll
                            for (int r = 0; r < 4; ++r) {
                                const float zr = __builtin_bit_cast(
                                    float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, z), 16 * r));
                                mine[p] = (lane == c0 + r) ? zr : mine[p];
                            }
                        }
                    }
#pragma unroll
                    for (int r = 0; r < 4; ++r)
#pragma unroll
                        for (int i = 0; i < NE; ++i) y[r][i] = yn[r][i];
                }
#pragma unroll
                for (int p = 0; p < G; ++p)
                    if (p < nx && lane < len) acc += log_sigmoid(sign * static_cast<double>(mine[p]));
            }
            nodes += static_cast<int64_t>(P) * len;
        }
        acc = wave_sum(acc);
        if (lane == 0) {
            a.unit_ll[u] = acc;
            a.unit_nodes[u] = nodes;
        }
    }
}

// CBOW: one wavefront per work unit; per centre with a window, h = (sum of the window rows in
// ascending window order, fp64) / P, then one walk of the centre's path with fp64 dot products
// (lane n keeps the dot product of path node n and takes its log-sigmoid).
template <int NE>
__global__ __launch_bounds__(256) void k_loglik_cbow(LLArgs a) {
    const int lane = lane_id();
    const int64_t wave0 = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * blockDim.x / kWave;
    for (int64_t u = wave0; u < a.n_units; u += nwaves) {
        const int64_t d = u / a.segs_per_doc;
        const int nk = a.doc_kept[d];
        const int j0 = static_cast<int>(u - d * a.segs_per_doc) * kLLSeg;
        const int j1 = min(nk, j0 + kLLSeg);
        const int64_t base = d * a.doc_len;
        double acc = 0.0;
        int64_t nodes = 0, terms = 0;
        for (int j = j0; j < j1; ++j) {
            const int v = a.kept_vid[base + j];
            const int eff = static_cast<int>(a.kept_meta[base + j] >> 16);
            const int clo = max(0, j - eff), chi = min(nk - 1, j + eff);
            const int P = chi - clo;
            if (P == 0) continue;
            const int len = a.codelen[v];
            const uint64_t code = a.code[v];
            const int my_pt = (lane < len) ? a.points[a.point_off[v] + lane] : 0;
            const int cq = clo + lane + ((clo + lane >= j) ? 1 : 0);
            const int my_w = (lane < P) ? a.kept_vid[base + cq] : 0;
            double h[NE];
#pragma unroll
            for (int i = 0; i < NE; ++i) h[i] = 0.0;
            for (int q = 0; q < P; ++q) {
                float x[NE];
                buf_load_row<NE>(x, row_rsrc(const_cast<float *>(a.syn0), __builtin_amdgcn_readlane(my_w, q),
                                             a.stride, a.dim * 4), lane);
#pragma unroll
                for (int i = 0; i < NE; ++i) h[i] += static_cast<double>(x[i]);
            }
#pragma unroll
            for (int i = 0; i < NE; ++i) h[i] = h[i] / static_cast<double>(P);
            double mine = 0.0;
            for (int c = 0; c < len; ++c) {
                float y[NE];
                buf_load_row<NE>(y, row_rsrc(const_cast<float *>(a.syn1), __builtin_amdgcn_readlane(my_pt, c),
                                             a.stride, a.dim * 4), lane);
                double z = 0.0;
#pragma unroll
                for (int i = 0; i < NE; ++i) z += h[i] * static_cast<double>(y[i]);
                z = wave_sum(z);
                mine = (lane == c) ? z : mine;
            }
            const double sign = ((code >> min(lane, 63)) & 1ull) ? -1.0 : 1.0;
            if (lane < len) acc += log_sigmoid(sign * mine);
            nodes += len;
            terms += 1;
        }
        acc = wave_sum(acc);
        if (lane == 0) {
            a.unit_ll[u] = acc;
            a.unit_nodes[u] = nodes;
            a.unit_terms[u] = terms;
        }
    }
}

// fixed-order sum of the work units' partials (terms: optional)
__global__ __launch_bounds__(1024) void k_sum_docs(const double *__restrict__ ll, const int64_t *__restrict__ nodes,
                                                   const int64_t *__restrict__ terms, int64_t n,
                                                   double *__restrict__ out_ll, int64_t *__restrict__ out_nodes,
                                                   int64_t *__restrict__ out_terms) {
    __shared__ double sl[1024];
    __shared__ int64_t sn[1024];
    __shared__ int64_t st_[1024];
    double a = 0.0;
    int64_t b = 0, t = 0;
    for (int64_t i = threadIdx.x; i < n; i += 1024) {
        a += ll[i];
        b += nodes[i];
        if (terms) t += terms[i];
    }
    sl[threadIdx.x] = a;
    sn[threadIdx.x] = b;
    st_[threadIdx.x] = t;
    __syncthreads();
    for (int st = 512; st > 0; st >>= 1) {
        if (threadIdx.x < st) {
            sl[threadIdx.x] += sl[threadIdx.x + st];
            sn[threadIdx.x] += sn[threadIdx.x + st];
            st_[threadIdx.x] += st_[threadIdx.x + st];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        *out_ll = sl[0];
        *out_nodes = sn[0];
        *out_terms = st_[0];
    }
}

using LLFn = void (*)(LLArgs);
// G window words per path walk: all of a window of half-width 5 for rows of up to 320 floats.
LLFn pick_ll(int dim) {
    const int ne = (dim + kWave - 1) / kWave;
    if (ne <= 1) return k_loglik<1, 10>;
    if (ne <= 2) return k_loglik<2, 10>;
    if (ne <= 4) return k_loglik<4, 10>;
    if (ne <= 5) return k_loglik<5, 8>;   // 159 VGPRs: 3 waves per SIMD (10 words: 171, 2 waves)
    if (ne <= 8) return k_loglik<8, 4>;
    return k_loglik<16, 2>;
}

LLFn pick_ll_cbow(int dim) {
    const int ne = (dim + kWave - 1) / kWave;
    if (ne <= 1) return k_loglik_cbow<1>;
    if (ne <= 2) return k_loglik_cbow<2>;
    if (ne <= 4) return k_loglik_cbow<4>;
    if (ne <= 5) return k_loglik_cbow<5>;
    if (ne <= 8) return k_loglik_cbow<8>;
    return k_loglik_cbow<16>;
}

}  // namespace

int64_t loglik_units(int64_t n_tokens, int32_t doc_len) {
    return std::max<int64_t>(1, ceil_div(n_tokens, doc_len)) * ll_segs_per_doc(doc_len);
}

size_t loglik_extra_bytes(int64_t n_units) {
    Carve c;
    c.take<double>(static_cast<size_t>(n_units));
    c.take<int64_t>(static_cast<size_t>(n_units));
    c.take<int64_t>(static_cast<size_t>(n_units));
    c.take<double>(1);
    c.take<int64_t>(2);
    return c.used();
}

int run_loglik(const w2v_model *m, const w2v_params *p, const SampleBufs &b, int64_t n_tokens, Carve &c,
               double *sum_ll_host, int64_t *n_pairs_host, int64_t *n_nodes_host, hipStream_t s) {
    const int64_t n_units = loglik_units(n_tokens, p->doc_len);
    LLArgs a{};
    a.syn0 = m->syn0;
    a.syn1 = m->syn1;
    a.dim = m->dim;
    a.stride = m->row_stride;
    a.codelen = m->codelen;
    a.code = m->code;
    a.point_off = m->point_off;
    a.points = m->points;
    a.kept_vid = b.kept_vid;
    a.kept_meta = b.kept_meta;
    a.doc_kept = b.doc_kept;
    a.segs_per_doc = ll_segs_per_doc(p->doc_len);
    a.n_units = n_tokens > 0 ? ceil_div(n_tokens, p->doc_len) * a.segs_per_doc : 0;
    a.doc_len = p->doc_len;
    a.unit_ll = c.take<double>(static_cast<size_t>(n_units));
    a.unit_nodes = c.take<int64_t>(static_cast<size_t>(n_units));
    a.unit_terms = c.take<int64_t>(static_cast<size_t>(n_units));
    double *out = c.take<double>(1);
    int64_t *out_nt = c.take<int64_t>(2);   // nodes, terms
    const bool cbow = p->arch == 1;
    if (a.n_units > 0) {
        // one unit per wavefront: the hardware hands out workgroups as others finish, which balances the
        // uneven units (a document's kept centres end in a partial unit, and units past them are empty)
        const unsigned grid = static_cast<unsigned>(std::min<int64_t>(ceil_div(a.n_units, 4), INT32_MAX));
        hipLaunchKernelGGL(cbow ? pick_ll_cbow(m->dim) : pick_ll(m->dim), dim3(grid), dim3(256), 0, s, a);
        W2V_LAUNCH_CHECK("k_loglik");
        k_sum_docs<<<1, 1024, 0, s>>>(a.unit_ll, a.unit_nodes, cbow ? a.unit_terms : nullptr, a.n_units, out,
                                      out_nt, out_nt + 1);
        W2V_LAUNCH_CHECK("k_sum_docs");
    }
    double hll = 0.0;
    int64_t nt[2] = {0, 0};
    int64_t tot[4] = {0, 0, 0, 0};
    if (a.n_units > 0) {
        W2V_HIP(hipMemcpyAsync(&hll, out, sizeof(hll), hipMemcpyDeviceToHost, s));
        W2V_HIP(hipMemcpyAsync(nt, out_nt, sizeof(nt), hipMemcpyDeviceToHost, s));
    }
    W2V_HIP(hipMemcpyAsync(tot, b.totals, sizeof(tot), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipStreamSynchronize(s));
    const int64_t nn = nt[0];
    *sum_ll_host = hll;
    *n_pairs_host = cbow ? nt[1] : tot[3];
    if (n_nodes_host) *n_nodes_host = nn;
    return W2V_OK;
}

}  // namespace w2v
