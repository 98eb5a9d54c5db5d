// Vocabulary: id histogram, (count desc, id asc) ordering, id -> index map, token remap.
//
// Counting follows "for each wordid v in text" (Algorithm 1) and the mintf
// setting of §4.1. The order is produced by a bitonic sort of (count, id)
// records in device memory; the sort is a one-off per corpus.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "w2v_internal.h"

namespace w2v {
namespace {

constexpr int kHotBins = 36864;   // ids below this are counted in LDS first (Zipf-ranked ids are hot); 144 KiB
constexpr int kCountThreads = 1024;   // one workgroup per CU (the bins take most of its LDS)

__global__ __launch_bounds__(kCountThreads) void k_count(const int32_t *__restrict__ tok, int64_t n,
                                                         int32_t id_space, unsigned long long *__restrict__ counts,
                                                         unsigned long long *__restrict__ bad) {
    __shared__ uint32_t hot[kHotBins];
    const int nhot = id_space < kHotBins ? id_space : kHotBins;
    for (int i = threadIdx.x; i < nhot; i += blockDim.x) hot[i] = 0;
    __syncthreads();
    uint32_t my_bad = 0;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x * 4;
    for (int64_t base = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * 4; base < n;
         base += stride) {
        int32_t t[4];
        if (base + 3 < n && ((reinterpret_cast<uintptr_t>(tok + base) & 15) == 0)) {
            const int4 q = *reinterpret_cast<const int4 *>(tok + base);
            t[0] = q.x; t[1] = q.y; t[2] = q.z; t[3] = q.w;
        } else {
#pragma unroll
            for (int k = 0; k < 4; ++k) t[k] = (base + k < n) ? tok[base + k] : -2;
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int32_t v = t[k];
            if (v == -2 && base + k >= n) continue;
            if (v < 0 || v >= id_space) {
                ++my_bad;
            } else if (v < nhot) {
                atomicAdd(&hot[v], 1u);
            } else {
                atomicAdd(&counts[v], 1ull);
            }
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nhot; i += blockDim.x)
        if (hot[i]) atomicAdd(&counts[i], static_cast<unsigned long long>(hot[i]));
    if (my_bad) atomicAdd(bad, static_cast<unsigned long long>(my_bad));
}

// Sort record: kept ids carry their count; dropped ids and padding sort last.
struct Rec {
    int64_t key;   // count (>= 0) if kept, -1 if dropped, -2 for padding
    int32_t id;
    int32_t pad;
};

// true if a must come before b: count descending, then id ascending
__device__ __forceinline__ bool before(const Rec &a, const Rec &b) {
    return a.key > b.key || (a.key == b.key && a.id < b.id);
}

__global__ void k_make_recs(const unsigned long long *__restrict__ counts, int32_t id_space, int64_t min_count,
                            Rec *__restrict__ r, int32_t n2) {
    const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n2) return;
    Rec x;
    if (i < id_space) {
        const int64_t c = static_cast<int64_t>(counts[i]);
        x.key = c >= min_count ? c : -1;
        x.id = i;
    } else {
        x.key = -2;
        x.id = i;
    }
    x.pad = 0;
    r[i] = x;
}

constexpr int kTile = 2048;            // records sorted in LDS by one block
constexpr int kTileThreads = kTile / 2;

__device__ __forceinline__ void cmpx(Rec *s, int i, int l, bool up) {
    Rec a = s[i], b = s[l];
    if (before(b, a) == up) {
        s[i] = b;
        s[l] = a;
    }
}

// Full bitonic sort of each kTile-record tile (direction alternates with the tile
// index so that pairs of tiles form a bitonic sequence for the global passes).
__global__ __launch_bounds__(kTileThreads) void k_sort_tile(Rec *__restrict__ r) {
    __shared__ Rec s[kTile];
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kTile;
    for (int i = threadIdx.x; i < kTile; i += blockDim.x) s[i] = r[base + i];
    __syncthreads();
    for (int k = 2; k <= kTile; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            const int t = threadIdx.x;
            const int i = (t / j) * 2 * j + (t % j);
            const int l = i + j;
            const int64_t gi = base + i;
            const bool up = ((gi & k) == 0);
            cmpx(s, i, l, up);
            __syncthreads();
        }
    }
    for (int i = threadIdx.x; i < kTile; i += blockDim.x) r[base + i] = s[i];
}

// One global compare-exchange pass (stage k, distance j >= kTile).
__global__ void k_sort_global(Rec *__restrict__ r, int32_t n2, int32_t k, int32_t j) {
    const int32_t t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n2 / 2) return;
    const int32_t i = (t / j) * 2 * j + (t % j);
    const int32_t l = i + j;
    const bool up = ((i & k) == 0);
    Rec a = r[i], b = r[l];
    if (before(b, a) == up) {
        r[i] = b;
        r[l] = a;
    }
}

// Remaining passes of stage k with distance < kTile, inside each tile.
__global__ __launch_bounds__(kTileThreads) void k_sort_tile_merge(Rec *__restrict__ r, int32_t k) {
    __shared__ Rec s[kTile];
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kTile;
    for (int i = threadIdx.x; i < kTile; i += blockDim.x) s[i] = r[base + i];
    __syncthreads();
    for (int j = kTile >> 1; j > 0; j >>= 1) {
        const int t = threadIdx.x;
        const int i = (t / j) * 2 * j + (t % j);
        const int l = i + j;
        const bool up = (((base + i) & k) == 0);
        cmpx(s, i, l, up);
        __syncthreads();
    }
    for (int i = threadIdx.x; i < kTile; i += blockDim.x) r[base + i] = s[i];
}

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

__global__ void k_finish_vocab(const Rec *__restrict__ r, int32_t id_space, int32_t *__restrict__ vocab_ids,
                               int64_t *__restrict__ vocab_counts, int32_t *__restrict__ id_to_vocab,
                               unsigned long long *__restrict__ nv, unsigned long long *__restrict__ tw) {
    const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= id_space) return;
    const Rec x = r[i];
    const bool kept = x.key >= 0;
    vocab_ids[i] = kept ? x.id : -1;
    vocab_counts[i] = kept ? x.key : 0;
    if (kept) id_to_vocab[x.id] = i;
    // block-level totals, then one atomic per block
    __shared__ unsigned long long s_n, s_w;
    if (threadIdx.x == 0) { s_n = 0; s_w = 0; }
    __syncthreads();
    if (kept) {
        atomicAdd(&s_n, 1ull);
        atomicAdd(&s_w, static_cast<unsigned long long>(x.key));
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        if (s_n) atomicAdd(nv, s_n);
        if (s_w) atomicAdd(tw, s_w);
    }
}

// Four tokens per thread and step (16-byte loads and stores where the stream is 16-byte aligned), so that
// each thread keeps four independent gathers from id_to_vocab in flight.
__global__ void k_remap(const int32_t *__restrict__ tok, int64_t n, const int32_t *__restrict__ id_to_vocab,
                        int32_t id_space, int32_t *__restrict__ out) {
    auto map = [&](int32_t v) { return (v >= 0 && v < id_space) ? id_to_vocab[v] : -1; };
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    const int64_t tid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    const bool aligned = ((reinterpret_cast<uintptr_t>(tok) | reinterpret_cast<uintptr_t>(out)) & 15) == 0;
    const int64_t nq = aligned ? n / 4 : 0;   // whole 16-byte groups
    for (int64_t q = tid; q < nq; q += stride) {
        const int4 t = reinterpret_cast<const int4 *>(tok)[q];
        reinterpret_cast<int4 *>(out)[q] = make_int4(map(t.x), map(t.y), map(t.z), map(t.w));
    }
    for (int64_t i = nq * 4 + tid; i < n; i += stride) out[i] = map(tok[i]);
}

__global__ void k_zero_u64(unsigned long long *p, int64_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

int32_t pow2_at_least(int32_t n) {
    int32_t p = kTile;
    while (p < n) p <<= 1;
    return p;
}

}  // namespace

size_t vocab_workspace_bytes(int32_t id_space) {
    Carve c;
    c.take<Rec>(pow2_at_least(id_space));
    c.take<unsigned long long>(4);
    return c.used();
}

int run_build_vocab(const int32_t *tokens, int64_t n_tokens, int32_t id_space, int64_t min_count,
                    int64_t *counts_by_id, int32_t *vocab_ids, int64_t *vocab_counts, int32_t *id_to_vocab,
                    int32_t *tokens_out, int32_t *V_host, int64_t *train_words_host, void *workspace,
                    hipStream_t s) {
    Carve c(workspace);
    const int32_t n2 = pow2_at_least(id_space);
    Rec *recs = c.take<Rec>(n2);
    unsigned long long *scal = c.take<unsigned long long>(4);   // bad, V, train_words
    unsigned long long *counts = reinterpret_cast<unsigned long long *>(counts_by_id);

    k_zero_u64<<<static_cast<unsigned>(ceil_div(id_space, 256)), 256, 0, s>>>(counts, id_space);
    k_zero_u64<<<1, 64, 0, s>>>(scal, 4);
    W2V_LAUNCH_CHECK("zero");
    if (n_tokens > 0) {
        const int cus = device_cu_count();
        const int64_t want = ceil_div(n_tokens, static_cast<int64_t>(kCountThreads) * 4 * 16);
        const unsigned grid = static_cast<unsigned>(std::max<int64_t>(1, std::min<int64_t>(want, 1LL * cus)));
        k_count<<<grid, kCountThreads, 0, s>>>(tokens, n_tokens, id_space, counts, scal + 0);
        W2V_LAUNCH_CHECK("k_count");
    }
    k_make_recs<<<static_cast<unsigned>(ceil_div(n2, 256)), 256, 0, s>>>(counts, id_space, min_count, recs, n2);
    k_sort_tile<<<static_cast<unsigned>(n2 / kTile), kTileThreads, 0, s>>>(recs);
    W2V_LAUNCH_CHECK("k_sort_tile");
    for (int32_t k = 2 * kTile; k <= n2; k <<= 1) {
        for (int32_t j = k >> 1; j >= kTile; j >>= 1)
            k_sort_global<<<static_cast<unsigned>(ceil_div(n2 / 2, 256)), 256, 0, s>>>(recs, n2, k, j);
        k_sort_tile_merge<<<static_cast<unsigned>(n2 / kTile), kTileThreads, 0, s>>>(recs, k);
    }
    W2V_LAUNCH_CHECK("sort");
    k_fill_i32<<<static_cast<unsigned>(ceil_div(id_space, 256)), 256, 0, s>>>(id_to_vocab, id_space, -1);
    k_finish_vocab<<<static_cast<unsigned>(ceil_div(id_space, 256)), 256, 0, s>>>(
        recs, id_space, vocab_ids, vocab_counts, id_to_vocab, scal + 1, scal + 2);
    W2V_LAUNCH_CHECK("k_finish_vocab");
    if (tokens_out && n_tokens > 0) {
        const unsigned grid = static_cast<unsigned>(std::min<int64_t>(ceil_div(n_tokens, 4 * 256), 8192));
        k_remap<<<grid, 256, 0, s>>>(tokens, n_tokens, id_to_vocab, id_space, tokens_out);
        W2V_LAUNCH_CHECK("k_remap");
    }
    unsigned long long h[3];
    W2V_HIP(hipMemcpyAsync(h, scal, sizeof(h), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipStreamSynchronize(s));
    *V_host = static_cast<int32_t>(h[1]);
    *train_words_host = static_cast<int64_t>(h[2]);
    if (h[0] != 0)
        return fail(W2V_E_RANGE, std::to_string(h[0]) + " token(s) outside [0, id_space)");
    return W2V_OK;
}

}  // namespace w2v
