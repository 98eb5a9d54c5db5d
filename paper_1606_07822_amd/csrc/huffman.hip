// Huffman tree of the vocabulary (§2: output layer of the hierarchical softmax).
//
// Construction rule: leaves in ascending count (vocabulary index V-1 first),
// inner nodes in creation order; each merge takes the smaller front twice, a
// leaf winning a count tie; the first child taken gets bit 0; merge a creates
// inner node a (root = V-2). The chain of merges is split into generations that
// are each computed in parallel (below). Parallel kernels then derive codes,
// offsets and points.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "w2v_internal.h"

namespace w2v {
namespace {

// Generations. Both queues are in ascending order, and the inner queue is first in,
// first out. Call the inner nodes that exist when a generation starts (indices
// ih .. a0-1) old. While an old node is still queued, the inner front is an old node,
// so every pick is the smaller of the leaf front and an old node: the picks are the
// stable merge S of the leaf queue with the old nodes (a leaf first on a tie), and
// merge a0+j takes S[2j] (bit 0) and S[2j+1] (bit 1). S ends with the last old node,
// after the leaves whose count is at most its count. If S has odd length, its last
// element (the last old node) opens one more merge whose second pick is the smaller of
// the leaf front and the first node of this generation (node a0), and the next
// generation starts. A Zipf vocabulary of 1M words takes 26 generations.
//
// One block computes a generation in chunks of kChunk elements of S: it copies the next
// kChunk leaves and old counts to LDS, and thread j finds how many leaves precede
// element 2j by a binary search on the merge path (the i with A[i-1] <= B[2j-i] and
// B[2j-i-1] < A[i], A the leaves, B the old nodes, a missing neighbour passing its
// test), then takes its two picks.
constexpr int kMergeThreads = 1024;
constexpr int kChunk = 2 * kMergeThreads;   // elements of S per chunk: one merge per thread

__global__ void k_check_descending(const int64_t *__restrict__ counts, int32_t V, int32_t *__restrict__ flags) {
    const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i + 1 < V && counts[i] < counts[i + 1]) atomicOr(&flags[2], 1);
}

// Leaves in ascending count: position p is vocabulary index V-1-p.
__device__ __forceinline__ int64_t leaf_val(const int64_t *__restrict__ counts, int32_t V, int32_t p) {
    return counts[V - 1 - p];
}

__global__ __launch_bounds__(kMergeThreads) void k_huff_merge(const int64_t *__restrict__ counts, int32_t V,
                                                              int32_t *__restrict__ parent, uint8_t *__restrict__ bit,
                                                              int64_t *__restrict__ icount, int32_t *__restrict__ flags) {
    __shared__ int64_t s_leaf[kChunk];    // A: leaf counts at queue positions pl+i0 ..
    __shared__ int64_t s_old[kChunk];     // B: old inner counts ih+j0 ..
    if (flags[2]) return;                 // counts not in descending order: no tree
    const int tid = threadIdx.x;
    // queue state, the same in every thread: leaf front pl, inner front ih, next merge a
    int32_t pl = 0, ih = 0, a = 0;
    // a step is a generation's start or a chunk; each chunk and each first merge performs at least one
    // merge, so a well-formed input takes at most 2(V-1) steps
    const int64_t max_steps = 2LL * V + 4;
    int64_t steps = 0;
    while (a < V - 1) {
        const int32_t a0 = a, T = a0 - ih;   // old nodes ih .. a0-1
        if (++steps > max_steps) break;
        if (T == 0) {   // no inner node yet (the first merge): two leaves
            if (tid == 0) {
                parent[V - 1 - pl] = a;
                bit[V - 1 - pl] = 0;
                parent[V - 2 - pl] = a;
                bit[V - 2 - pl] = 1;
                icount[a] = leaf_val(counts, V, pl) + leaf_val(counts, V, pl + 1);
            }
            pl += 2;
            a += 1;
            __threadfence_block();
            __syncthreads();
            continue;
        }
        const int64_t last = icount[a0 - 1];   // count of the last old node
        int32_t i0 = 0, j0 = 0;                // leaves and old nodes taken in this generation
        while (j0 < T) {
            if (++steps > max_steps) break;
            const int32_t lw = min(kChunk, V - pl - i0), iw = min(kChunk, T - j0);
            int32_t nle = 0;   // loaded leaves with count <= last
#pragma unroll
            for (int r = 0; r < kChunk / kMergeThreads; ++r) {
                const int32_t t = tid + r * kMergeThreads;
                int64_t x = 0;
                if (t < lw) {
                    x = leaf_val(counts, V, pl + i0 + t);
                    s_leaf[t] = x;
                }
                if (t < iw) s_old[t] = icount[ih + j0 + t];
                nle += __syncthreads_count(t < lw && x <= last);
            }
            // elements of S in this chunk: all kChunk, or up to the last old node when it is loaded (the
            // leaves at most its count come before it; if every loaded leaf does, S reaches past the chunk)
            const int32_t out = iw == T - j0 ? min(kChunk, iw + nle) : kChunk;
            const int32_t M = out >> 1;
            bool leaf0 = false, leaf1 = false;
            if (tid < M) {
                const int32_t k = 2 * tid;
                int32_t lo = max(0, k - iw), hi = min(k, lw);
                while (lo < hi) {
                    const int32_t mid = (lo + hi) >> 1;
                    if (s_leaf[mid] <= s_old[k - mid - 1]) lo = mid + 1;
                    else hi = mid;
                }
                int32_t i = lo;
                leaf0 = i < lw && (k - i >= iw || s_leaf[min(i, kChunk - 1)] <= s_old[min(k - i, kChunk - 1)]);
                const int64_t v0 = leaf0 ? s_leaf[i] : s_old[k - i];
                const int32_t c0 = leaf0 ? V - 1 - (pl + i0 + i) : V + ih + j0 + (k - i);
                i += leaf0;
                leaf1 = i < lw &&
                        (k + 1 - i >= iw || s_leaf[min(i, kChunk - 1)] <= s_old[min(k + 1 - i, kChunk - 1)]);
                const int64_t v1 = leaf1 ? s_leaf[i] : s_old[k + 1 - i];
                const int32_t c1 = leaf1 ? V - 1 - (pl + i0 + i) : V + ih + j0 + (k + 1 - i);
                parent[c0] = a + tid;
                bit[c0] = 0;
                parent[c1] = a + tid;
                bit[c1] = 1;
                icount[a + tid] = v0 + v1;
            }
            __threadfence_block();
            const int32_t taken = __syncthreads_count(leaf0) + __syncthreads_count(leaf1);
            a += M;
            i0 += taken;
            j0 += 2 * M - taken;
            if (out & 1) {
                __syncthreads();   // node a0's count, written by another thread
                // S ended on the last old node (ih+j0, count `last`) as the first pick of a merge; the second
                // is the leaf front or the first node of this generation, a leaf winning a tie. Thread 0
                // decides, and the barrier's count hands the decision to every thread.
                const int32_t nl = V - pl - i0;
                const bool fresh = a > a0;
                int64_t lf = 0, fn = 0;
                bool leaf_t0 = false;
                if (tid == 0) {
                    lf = nl > 0 ? leaf_val(counts, V, pl + i0) : 0;
                    fn = fresh ? icount[a0] : 0;
                    leaf_t0 = nl > 0 && (!fresh || lf <= fn);
                }
                const bool take_leaf = __syncthreads_count(leaf_t0) != 0;
                if (tid == 0) {
                    parent[V + ih + j0] = a;
                    bit[V + ih + j0] = 0;
                    const int32_t c1 = take_leaf ? V - 1 - (pl + i0) : V + a0;
                    parent[c1] = a;
                    bit[c1] = 1;
                    icount[a] = last + (take_leaf ? lf : fn);
                }
                j0 += 1;
                if (take_leaf) ++i0;
                else ++ih;   // node a0 leaves the queue; the generation ends here (j0 == T)
                ++a;
                __threadfence_block();
                __syncthreads();
            }
        }
        pl += i0;
        ih += j0;
    }
    if (a < V - 1 && tid == 0) atomicOr(&flags[2], 1);   // step cap reached: malformed counts
}

// codelen / code per leaf; maxlen and error flag (code longer than 64).
__global__ void k_huff_codes(const int32_t *__restrict__ parent, const uint8_t *__restrict__ bit, int32_t V,
                             uint8_t *__restrict__ codelen, uint64_t *__restrict__ code, int32_t *__restrict__ flags) {
    const int32_t v = blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= V) return;
    const int32_t root = V + V - 2;
    int32_t node = v, depth = 0;
    uint64_t rev = 0;
    while (node != root) {
        const int32_t up = parent[node];
        if (depth >= 64 || up < 0 || up > V - 2) {
            atomicOr(&flags[1], 1);
            codelen[v] = 0;
            code[v] = 0;
            return;
        }
        rev |= static_cast<uint64_t>(bit[node]) << depth;
        ++depth;
        node = V + up;
    }
    codelen[v] = static_cast<uint8_t>(depth);
    code[v] = depth ? (__brevll(rev) >> (64 - depth)) : 0;
    atomicMax(&flags[0], depth);
}

// Exclusive prefix sum of codelen into point_off[0..V] in three passes: the sum of each tile of
// kScanTile code lengths, one block scanning the tile sums, and each tile's own scan plus its offset.
// (At V = 1M this takes well under 0.1 ms; the one-workgroup block_exclusive_scan that the smaller
// per-document scans use would take about 0.8 ms here.)
constexpr int kScanTile = 1024;

// inclusive block scan of one value per thread (kScanTile threads); returns the inclusive prefix, *sum the total
__device__ __forceinline__ int64_t block_incl_scan(int64_t x, int64_t *wsum, int64_t *sum) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    int64_t inc = x;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int64_t y = __shfl_up(inc, d, 64);
        if (lane >= d) inc += y;
    }
    if (lane == 63) wsum[wid] = inc;
    __syncthreads();
    int64_t before = 0, total = 0;
    for (int w = 0; w < kScanTile / 64; ++w) {
        before += w < wid ? wsum[w] : 0;
        total += wsum[w];
    }
    *sum = total;
    __syncthreads();   // wsum is reused by the next call
    return before + inc;
}

__global__ __launch_bounds__(kScanTile) void k_scan_tiles(const uint8_t *__restrict__ codelen, int32_t V,
                                                          int64_t *__restrict__ tile_sum) {
    __shared__ int64_t wsum[kScanTile / 64];
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kScanTile + threadIdx.x;
    int64_t total;
    block_incl_scan(i < V ? codelen[i] : 0, wsum, &total);
    if (threadIdx.x == 0) tile_sum[blockIdx.x] = total;
}

// tile_sum -> exclusive tile offsets in place; *total = sum of all code lengths
__global__ __launch_bounds__(kScanTile) void k_scan_tile_sums(int64_t *__restrict__ tile_sum, int32_t n_tiles,
                                                              int64_t *__restrict__ total) {
    __shared__ int64_t wsum[kScanTile / 64];
    int64_t carry = 0;
    for (int32_t base = 0; base < n_tiles; base += kScanTile) {
        const int32_t i = base + threadIdx.x;
        const int64_t x = i < n_tiles ? tile_sum[i] : 0;
        int64_t chunk;
        const int64_t inc = block_incl_scan(x, wsum, &chunk);
        if (i < n_tiles) tile_sum[i] = carry + inc - x;
        carry += chunk;
    }
    if (threadIdx.x == 0) *total = carry;
}

__global__ __launch_bounds__(kScanTile) void k_scan_apply(const uint8_t *__restrict__ codelen, int32_t V,
                                                          const int64_t *__restrict__ tile_off,
                                                          const int64_t *__restrict__ total,
                                                          int32_t *__restrict__ point_off) {
    __shared__ int64_t wsum[kScanTile / 64];
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kScanTile + threadIdx.x;
    const int64_t x = i < V ? codelen[i] : 0;
    int64_t chunk;
    const int64_t inc = block_incl_scan(x, wsum, &chunk);
    if (i < V) point_off[i] = static_cast<int32_t>(tile_off[blockIdx.x] + inc - x);
    if (i == V) point_off[V] = static_cast<int32_t>(*total);
}

__global__ void k_huff_points(const int32_t *__restrict__ parent, int32_t V, const uint8_t *__restrict__ codelen,
                              const int32_t *__restrict__ point_off, int32_t *__restrict__ points) {
    const int32_t v = blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= V) return;
    const int32_t len = codelen[v];
    int32_t *out = points + point_off[v];
    int32_t node = v;
    for (int32_t s = 0; s < len; ++s) {
        const int32_t p = parent[node];
        out[len - 1 - s] = p;
        node = V + p;
    }
}

__global__ void k_fill_parent(int32_t *p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = -1;
}

__global__ void k_zero_i32(int32_t *p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

}  // namespace

size_t huffman_workspace_bytes(int32_t V) {
    Carve c;
    c.take<int32_t>(2 * static_cast<size_t>(V));   // parent
    c.take<uint8_t>(2 * static_cast<size_t>(V));   // bit
    c.take<int64_t>(static_cast<size_t>(V));       // icount
    c.take<int32_t>(4);                            // flags
    c.take<int64_t>(2);                            // total
    c.take<int64_t>(static_cast<size_t>(ceil_div(V, kScanTile)));   // tile sums of the code-length scan
    return c.used();
}

int run_build_huffman(const int64_t *vocab_counts, int32_t V, uint8_t *codelen, uint64_t *code, int32_t *point_off,
                      int32_t *points, int64_t points_cap, int64_t *points_len_host, int32_t *max_len_host,
                      void *workspace, hipStream_t s) {
    Carve c(workspace);
    int32_t *parent = c.take<int32_t>(2 * static_cast<size_t>(V));
    uint8_t *bit = c.take<uint8_t>(2 * static_cast<size_t>(V));
    int64_t *icount = c.take<int64_t>(static_cast<size_t>(V));
    int32_t *flags = c.take<int32_t>(4);
    int64_t *total = c.take<int64_t>(2);
    const int32_t n_tiles = static_cast<int32_t>(ceil_div(V, kScanTile));
    int64_t *tile_sum = c.take<int64_t>(static_cast<size_t>(n_tiles));
    const unsigned gv = static_cast<unsigned>(ceil_div(V, 256));
    k_zero_i32<<<1, 64, 0, s>>>(flags, 4);
    k_fill_parent<<<static_cast<unsigned>(ceil_div(2LL * V, 256)), 256, 0, s>>>(parent, 2 * V);
    k_check_descending<<<gv, 256, 0, s>>>(vocab_counts, V, flags);
    W2V_LAUNCH_CHECK("k_check_descending");
    k_huff_merge<<<1, kMergeThreads, 0, s>>>(vocab_counts, V, parent, bit, icount, flags);
    W2V_LAUNCH_CHECK("k_huff_merge");
    k_huff_codes<<<gv, 256, 0, s>>>(parent, bit, V, codelen, code, flags);
    W2V_LAUNCH_CHECK("k_huff_codes");
    k_scan_tiles<<<static_cast<unsigned>(n_tiles), kScanTile, 0, s>>>(codelen, V, tile_sum);
    k_scan_tile_sums<<<1, kScanTile, 0, s>>>(tile_sum, n_tiles, total);
    // one more thread than V writes point_off[V]
    k_scan_apply<<<static_cast<unsigned>(ceil_div(static_cast<int64_t>(V) + 1, kScanTile)), kScanTile, 0, s>>>(
        codelen, V, tile_sum, total, point_off);
    W2V_LAUNCH_CHECK("k_scan_codelen");
    int32_t hflags[3];
    int64_t htotal = 0;
    W2V_HIP(hipMemcpyAsync(hflags, flags, sizeof(hflags), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipMemcpyAsync(&htotal, total, sizeof(htotal), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipStreamSynchronize(s));
    if (hflags[2]) return fail(W2V_E_ARG, "vocab_counts must be in descending order");
    if (hflags[1]) return fail(W2V_E_RANGE, "a Huffman code is longer than 64 bits");
    *points_len_host = htotal;
    *max_len_host = hflags[0];
    if (points) {
        if (points_cap < htotal)
            return fail(W2V_E_ARG, "points_cap " + std::to_string(points_cap) + " < points length " +
                                       std::to_string(htotal));
        k_huff_points<<<gv, 256, 0, s>>>(parent, V, codelen, point_off, points);
        W2V_LAUNCH_CHECK("k_huff_points");
        W2V_HIP(hipStreamSynchronize(s));
    }
    return W2V_OK;
}

}  // namespace w2v
