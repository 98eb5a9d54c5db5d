// Asynchronous HS training (Algorithm 1, Cached Skipgram HS), GPU form.
//
// Worker = one wavefront. Wavefronts claim whole documents from a queue and
// walk their kept centre words in order. Per centre v with window words
// w_1..w_P the path of v is walked once: each inner-node row is loaded once,
// updated by every window word in order (dot, sigmoid, gradient, two axpys)
// and its change written back once; the hidden-layer gradients of the window
// words stay in registers and are added to syn0 after the path. Swapping the
// window and node loops of Algorithm 1 this way is the same computation
// whenever a window holds no repeated word.
//
// Cache (§3.2): the cache owner is the workgroup. The rows of the top
// cache_k inner nodes (the k created last by the Huffman merge) sit in LDS as
// `val` (current) and `orig` (value at the last write-back); waves update
// `val` with LDS atomic adds of their change. Every flush_every centres of the
// workgroup, one wave writes val - orig back to HBM with an atomic add and
// re-bases both copies on the returned HBM value (the write-back plus the
// refill of Algorithm 1's flush, without stopping the other waves).
//
// Rows are spread over the 64 lanes element-strided: lane l holds elements
// l, l+64, l+128, ... so every row load is a run of coalesced 256-byte
// accesses and every dot product ends in one cross-lane reduction.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "w2v_internal.h"

namespace w2v {


namespace {

constexpr int kWavesPerBlock = 8;
constexpr int kBlock = kWavesPerBlock * kWave;

__device__ __forceinline__ float sigmoid_fast(float z) {
    return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

__device__ __forceinline__ void lds_add(float *p, float v) { atomicAdd(p, v); }

// One wave writes the cache's change back to HBM and re-bases val/orig on the result.
// flush_scale = 1 adds the change as in the paper; < 1 adds a fraction of it (the
// workgroups' local progress on the cached rows is then averaged rather than summed).
__device__ void flush_cache_wave(const TrainArgs &a, float *val, float *orig, int lane) {
    for (int s = 0; s < a.cache_k; ++s) {
        float *g = a.syn1 + static_cast<int64_t>(a.cache_first + s) * a.stride;
        float *vs = val + s * a.dim;
        float *os = orig + s * a.dim;
        for (int col = lane; col < a.dim; col += kWave) {
            const float c = vs[col];
            const float d = (c - os[col]) * a.flush_scale;
            if (d != 0.0f) {
                const float old = atomicAdd(g + col, d);
                const float nv = old + d;
                lds_add(vs + col, nv - c);
                os[col] = nv;
            }
        }
    }
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
__device__ __forceinline__ float dot_partial(const float (&x)[NE], const float (&y)[NE]) {
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < NE; ++i) s = fmaf(x[i], y[i], s);
    return s;
}

// ARCH 0: skip-gram; ARCH 1: CBOW. PMAX >= 2 * window.
template <int NE, int PMAX, int ARCH>
__global__ __launch_bounds__(kBlock) void k_train(TrainArgs a) {
    extern __shared__ float lds[];
    float *val = lds;
    float *orig = lds + a.cache_k * a.dim;
    __shared__ int s_centres;
    __shared__ int s_lock;
    const int lane = lane_id();
    if (threadIdx.x == 0) {
        s_centres = 0;
        s_lock = 0;
    }
    const int kd = a.cache_k * a.dim;
    for (int i = threadIdx.x; i < kd; i += blockDim.x) {
        const int s = i / a.dim, col = i - s * a.dim;
        const float v = a.syn1[static_cast<int64_t>(a.cache_first + s) * a.stride + col];
        val[i] = v;
        orig[i] = v;
    }
    __syncthreads();

    const int gw = blockIdx.x * kWavesPerBlock + static_cast<int>(threadIdx.x / kWave);
    uint64_t n_kept = 0, n_pairs = 0, n_nodes = 0;
    if (gw < a.workers) {
        while (true) {
            int doc = 0;
            if (lane == 0) doc = atomicAdd(a.queue, 1);
            doc = __builtin_amdgcn_readfirstlane(doc);
            if (doc >= a.n_docs) break;
            const int nk = a.doc_kept[doc];
            const int64_t base = static_cast<int64_t>(doc) * a.doc_len;
            const int32_t *kv = a.kept_vid + base;
            const uint32_t *km = a.kept_meta + base;
            for (int j = 0; j < nk; ++j) {
                const uint32_t meta = km[j];
                const int v = kv[j];
                const int eff = static_cast<int>(meta >> 16);
                const int lo = max(0, j - eff), hi = min(nk - 1, j + eff);
                const int P = hi - lo;   // window words, centre excluded
                ++n_kept;
                if (P > 0) {
                    const int64_t g = a.epoch_base + a.first_raw + base + static_cast<int64_t>(meta & 0xFFFFu);
                    const float alpha = a.alpha_tab[g / 10000 - a.blk0];
                    // window words: lane q holds the vocabulary index of the q-th one
                    int wv = 0;
                    if (lane < P) {
                        const int c = lo + lane + ((lo + lane >= j) ? 1 : 0);
                        wv = kv[c];
                    }
                    const int len = a.codelen[v];
                    const uint64_t code = a.code[v];
                    const int my_pt = (lane < len) ? a.points[a.point_off[v] + lane] : 0;

                    if constexpr (ARCH == 0) {
                        float x[PMAX][NE], e[PMAX][NE];
#pragma unroll
                        for (int p = 0; p < PMAX; ++p) {
                            if (p < P) {
                                const int w = __builtin_amdgcn_readlane(wv, p);
                                load_row<NE>(x[p], a.syn0 + static_cast<int64_t>(w) * a.stride, lane, a.dim);
                            }
#pragma unroll
                            for (int i = 0; i < NE; ++i) e[p][i] = 0.0f;
                        }
                        for (int jn = 0; jn < len; ++jn) {
                            const int n = __builtin_amdgcn_readlane(my_pt, jn);
                            const float t = static_cast<float>((code >> jn) & 1ull);
                            const bool cached = n >= a.cache_first;
                            float *lrow = val + (n - a.cache_first) * a.dim;
                            float *grow = a.syn1 + static_cast<int64_t>(n) * a.stride;
                            float y[NE], y0[NE];
                            if (cached) load_row<NE>(y, lrow, lane, a.dim);
                            else load_row<NE>(y, grow, lane, a.dim);
#pragma unroll
                            for (int i = 0; i < NE; ++i) y0[i] = y[i];
#pragma unroll
                            for (int p = 0; p < PMAX; ++p) {
                                if (p < P) {
                                    const float z = wave_sum(dot_partial<NE>(x[p], y));
                                    const float f = sigmoid_fast(z);
                                    const float gr = (1.0f - t - f) * alpha;
#pragma unroll
                                    for (int i = 0; i < NE; ++i) {
                                        e[p][i] = fmaf(gr, y[i], e[p][i]);
                                        y[i] = fmaf(gr, x[p][i], y[i]);
                                    }
                                }
                            }
#pragma unroll
                            for (int i = 0; i < NE; ++i) {
                                const int col = lane + i * kWave;
                                if (col < a.dim) {
                                    if (cached) lds_add(lrow + col, y[i] - y0[i]);
                                    else if (a.write_policy == 0) atomicAdd(grow + col, y[i] - y0[i]);
                                    else grow[col] = y[i];
                                }
                            }
                        }
#pragma unroll
                        for (int p = 0; p < PMAX; ++p) {
                            if (p < P) {
                                const int w = __builtin_amdgcn_readlane(wv, p);
                                float *xr = a.syn0 + static_cast<int64_t>(w) * a.stride;
#pragma unroll
                                for (int i = 0; i < NE; ++i) {
                                    const int col = lane + i * kWave;
                                    if (col < a.dim) atomicAdd(xr + col, e[p][i]);
                                }
                            }
                        }
                        n_nodes += static_cast<uint64_t>(P) * len;
                    } else {
                        // CBOW: h = mean of the window vectors; one path walk; e added to each window vector
                        float h[NE], e[NE];
#pragma unroll
                        for (int i = 0; i < NE; ++i) { h[i] = 0.0f; e[i] = 0.0f; }
                        for (int p = 0; p < P; ++p) {
                            const int w = __builtin_amdgcn_readlane(wv, p);
                            float xr[NE];
                            load_row<NE>(xr, a.syn0 + static_cast<int64_t>(w) * a.stride, lane, a.dim);
#pragma unroll
                            for (int i = 0; i < NE; ++i) h[i] += xr[i];
                        }
                        const float fP = static_cast<float>(P);
#pragma unroll
                        for (int i = 0; i < NE; ++i) h[i] = h[i] / fP;
                        for (int jn = 0; jn < len; ++jn) {
                            const int n = __builtin_amdgcn_readlane(my_pt, jn);
                            const float t = static_cast<float>((code >> jn) & 1ull);
                            const bool cached = n >= a.cache_first;
                            float *lrow = val + (n - a.cache_first) * a.dim;
                            float *grow = a.syn1 + static_cast<int64_t>(n) * a.stride;
                            float y[NE];
                            if (cached) load_row<NE>(y, lrow, lane, a.dim);
                            else load_row<NE>(y, grow, lane, a.dim);
                            const float z = wave_sum(dot_partial<NE>(h, y));
                            const float gr = (1.0f - t - sigmoid_fast(z)) * alpha;
#pragma unroll
                            for (int i = 0; i < NE; ++i) {
                                const int col = lane + i * kWave;
                                e[i] = fmaf(gr, y[i], e[i]);
                                const float d = gr * h[i];
                                if (col < a.dim) {
                                    if (cached) lds_add(lrow + col, d);
                                    else if (a.write_policy == 0) atomicAdd(grow + col, d);
                                    else grow[col] = y[i] + d;
                                }
                            }
                        }
                        for (int p = 0; p < P; ++p) {
                            const int w = __builtin_amdgcn_readlane(wv, p);
                            float *xr = a.syn0 + static_cast<int64_t>(w) * a.stride;
#pragma unroll
                            for (int i = 0; i < NE; ++i) {
                                const int col = lane + i * kWave;
                                if (col < a.dim) atomicAdd(xr + col, e[i]);
                            }
                        }
                        n_nodes += len;
                    }
                    n_pairs += P;
                }
                if (a.cache_k > 0) {
                    int go = 0;
                    if (lane == 0) {
                        const int c = atomicAdd(&s_centres, 1) + 1;
                        if (c % a.flush_every == 0) go = (atomicCAS(&s_lock, 0, 1) == 0) ? 1 : 0;
                    }
                    go = __builtin_amdgcn_readfirstlane(go);
                    if (go) {
                        flush_cache_wave(a, val, orig, lane);
                        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
                        if (lane == 0) atomicExch(&s_lock, 0);
                    }
                }
            }
        }
    }
    if (lane == 0 && n_kept) {
        atomicAdd(&a.stats[0], static_cast<unsigned long long>(n_kept));
        atomicAdd(&a.stats[1], static_cast<unsigned long long>(n_pairs));
        atomicAdd(&a.stats[2], static_cast<unsigned long long>(n_nodes));
    }
    __syncthreads();
    // final write-back of the cache
    for (int i = threadIdx.x; i < kd; i += blockDim.x) {
        const float d = (val[i] - orig[i]) * a.flush_scale;
        if (d != 0.0f) {
            const int s = i / a.dim, col = i - s * a.dim;
            atomicAdd(a.syn1 + static_cast<int64_t>(a.cache_first + s) * a.stride + col, d);
        }
    }
}

using TrainFn = void (*)(TrainArgs);

template <int NE, int ARCH>
TrainFn pick_pmax(int pmax) {
    if constexpr (ARCH == 1) {
        (void)pmax;
        return k_train<NE, 2, 1>;
    } else {
        if (pmax <= 4) return k_train<NE, 4, ARCH>;
        if (pmax <= 10) return k_train<NE, 10, ARCH>;
        return k_train<NE, 20, ARCH>;
    }
}

template <int ARCH>
TrainFn pick_ne(int dim, int pmax) {
    const int ne = (dim + kWave - 1) / kWave;
    if (ne <= 1) return pick_pmax<1, ARCH>(pmax);
    if (ne <= 2) return pick_pmax<2, ARCH>(pmax);
    if (ne <= 4) return pick_pmax<4, ARCH>(pmax);
    if (ne <= 5) return pick_pmax<5, ARCH>(pmax);
    if (ne <= 8) return pick_pmax<8, ARCH>(pmax);
    return pick_pmax<16, ARCH>(pmax);
}

__global__ void k_zero_train(int32_t *queue, unsigned long long *stats) {
    if (threadIdx.x == 0) *queue = 0;
    if (threadIdx.x < 3) stats[threadIdx.x] = 0;
}

__global__ void k_write_stats(const int64_t *totals, const unsigned long long *tstats, int64_t *out) {
    if (threadIdx.x == 0) {
        out[0] = totals[0];
        out[1] = totals[1];
        out[2] = static_cast<int64_t>(tstats[0]);
        out[3] = static_cast<int64_t>(tstats[1]);
        out[4] = static_cast<int64_t>(tstats[2]);
    }
}

}  // namespace

size_t train_lds_bytes(int32_t cache_k, int32_t dim) { return 2ull * cache_k * dim * sizeof(float); }

int launch_train_async(TrainArgs a, int arch, int window, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s,
                       int64_t *stats_out, const int64_t *totals) {
    const size_t lds = train_lds_bytes(a.cache_k, a.dim);
    TrainFn fn = arch == 0 ? pick_ne<0>(a.dim, 2 * window) : pick_ne<1>(a.dim, 2 * window);
    if (lds > 64 * 1024)
        W2V_HIP(hipFuncSetAttribute(reinterpret_cast<const void *>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                                    static_cast<int>(lds)));
    int grid;
    if (a.workers > 0) {
        grid = static_cast<int>(ceil_div(a.workers, kWavesPerBlock));
    } else {
        int per_cu = 0;
        W2V_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(fn), kBlock,
                                                             lds));
        grid = device_cu_count() * std::max(1, per_cu);
        a.workers = grid * kWavesPerBlock;
    }
    if (a.flush_scale <= 0.0f) a.flush_scale = 1.0f / static_cast<float>(grid);
    record_train_launch(grid, a.workers);
    k_zero_train<<<1, 64, 0, s>>>(a.queue, a.stats);
    W2V_LAUNCH_CHECK("k_zero_train");
    if (ev0) W2V_HIP(hipEventRecord(ev0, s));
    hipLaunchKernelGGL(fn, dim3(grid), dim3(kBlock), lds, s, a);
    W2V_LAUNCH_CHECK("k_train");
    if (ev1) W2V_HIP(hipEventRecord(ev1, s));
    if (stats_out) {
        k_write_stats<<<1, 64, 0, s>>>(totals, a.stats, stats_out);
        W2V_LAUNCH_CHECK("k_write_stats");
    }
    return W2V_OK;
}

}  // namespace w2v
