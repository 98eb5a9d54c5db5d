// Huffman tree of the vocabulary (§2: output layer of the hierarchical softmax).
//
// Construction rule: leaves in ascending count (vocabulary index V-1 first),
// inner nodes in creation order; each merge takes the smaller front twice, a
// leaf winning a count tie; the first child taken gets bit 0; merge a creates
// inner node a (root = V-2). The merge is a sequential chain except where it
// runs through many equal-kind merges in a row (the tail of a skewed
// vocabulary); those runs are written by the whole block, the rest by one lane.
// Parallel kernels then derive codes, offsets and points.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "w2v_internal.h"

namespace w2v {
namespace {

constexpr int kMergeThreads = 256;
constexpr int kRunMin = 32;   // runs of at least this many merges are written by the whole block
constexpr int kBurst = 8;     // single merges between two checks for a run (2 kBurst < 2 kRunMin)

// Leaves in ascending count: position p is vocabulary index V-1-p.
__device__ __forceinline__ int64_t leaf_val(const int64_t *__restrict__ counts, int32_t V, int32_t p) {
    return counts[V - 1 - p];
}

// Two-queue merge, written in phases. While the next merges alternate between the
// queues, lane 0 performs them one by one. When the next >= kRunMin merges all take
// two leaves (every leaf up to the 2m-th is <= the inner front, which those merges
// leave in place) or all take two inner nodes (every one of the next 2m inner nodes
// is < the leaf front), the block writes the whole run at once: merge a+i takes
// elements 2i (bit 0) and 2i+1 (bit 1) of that queue. New inner nodes join the back
// of their queue and never take part in the run that creates them.
//
// Lane 0 reads both queues from LDS: each phase starts with the block copying the next
// kWin leaves and the next kWin inner counts (those created before the phase) into LDS,
// and the counts lane 0 creates go to a third LDS window as well as to memory. A phase
// whose merges would reach past a window ends early and the next one refills them.
constexpr int kWin = 1024;

__global__ __launch_bounds__(kMergeThreads) void k_huff_merge(const int64_t *__restrict__ counts, int32_t V,
                                                              int32_t *__restrict__ parent, uint8_t *__restrict__ bit,
                                                              int64_t *__restrict__ icount, int32_t *__restrict__ flags) {
    __shared__ int32_t s_pl, s_ih, s_a, s_mode;
    __shared__ int64_t s_front;
    __shared__ int64_t s_leaf[kWin];    // leaf values at queue positions [lb, lb + kWin)
    __shared__ int64_t s_inner[kWin];   // inner counts [ib, ib + kWin), those below a0
    __shared__ int64_t s_new[kWin];     // inner counts created in this phase: a0, a0 + 1, ...
    const int tid = threadIdx.x;
    if (tid == 0) {
        s_pl = 0;
        s_ih = 0;
        s_a = 0;
    }
    __syncthreads();
    const int64_t max_phases = 4LL * V + 16;   // every phase merges at least once
    for (int64_t phase = 0; phase < max_phases; ++phase) {
        const int32_t lb = s_pl, ib = s_ih, a0 = s_a;
        for (int i = tid; i < kWin; i += kMergeThreads) {
            s_leaf[i] = lb + i < V ? leaf_val(counts, V, lb + i) : 0;
            s_inner[i] = ib + i < a0 ? icount[ib + i] : 0;
        }
        __syncthreads();
        if (tid == 0) {
            int32_t pl = lb, ih = ib, a = a0;
            int mode = 0;   // 0 done, 1 leaf run, 2 inner run, 3 refill the windows
            int64_t front = 0;
            // queue values by position / index. The positions a merge uses lie inside the windows (checked
            // below); the reads are clamped to the windows so that all of a merge's reads can be issued
            // before any branch on their values (a clamped value is never used).
            auto leafv = [&](int32_t q) { return s_leaf[min(max(q - lb, 0), kWin - 1)]; };
            auto innerv = [&](int32_t q) {
                return q < a0 ? s_inner[min(max(q - ib, 0), kWin - 1)] : s_new[min(q - a0, kWin - 1)];
            };
            while (a < V - 1) {
                // checks for the next burst of up to kBurst merges: they read leaves pl .. pl+2kBurst-1 and inner
                // nodes ih .. ih+2kBurst-1 (both within the probes' reach, pl+2kRunMin-1 and
                // min(ih+2kRunMin, a)-1, or created in this phase) and write counts a .. a+kBurst-1
                const int32_t hi = min(ih + 2 * kRunMin, a);
                const bool leaf_ok = lb + kWin >= V || pl + 2 * kRunMin <= lb + kWin;
                const bool inner_ok =
                    min(hi, a0) - ib <= kWin && (hi <= a0 || hi - a0 <= kWin) && a + kBurst - a0 <= kWin;
                if (!leaf_ok || !inner_ok) {
                    mode = 3;
                    break;
                }
                {
                    const int32_t nl = V - pl, ni = a - ih;
                    const int64_t FI = ni > 0 ? innerv(ih) : 0;
                    const int64_t FL = nl > 0 ? leafv(pl) : 0;
                    const int64_t probe_l = leafv(pl + 2 * kRunMin - 1), probe_i = innerv(ih + 2 * kRunMin - 1);
                    if (ni > 0 && nl >= 2 * kRunMin && probe_l <= FI) {
                        mode = 1;
                        front = FI;
                        break;
                    }
                    if (ni >= 2 * kRunMin && (nl == 0 || probe_i < FL)) {
                        mode = 2;
                        front = nl > 0 ? FL : INT64_MAX;
                        break;
                    }
                }
                for (int u = 0; u < kBurst && a < V - 1; ++u) {
                    const int32_t nl = V - pl, ni = a - ih;
                    // both fronts and the elements behind them, read together (one LDS round trip per merge)
                    const int64_t fi = innerv(ih), fl = leafv(pl), i1 = innerv(ih + 1), l1 = leafv(pl + 1);
                    const int64_t FI = ni > 0 ? fi : 0;
                    const int64_t FL = nl > 0 ? fl : 0;
                    const int64_t I1 = ni > 1 ? i1 : 0;
                    const int64_t L1 = nl > 1 ? l1 : 0;
                    // one merge: a leaf wins a tie; the second pick compares the fronts left by the first
                    const bool leaf0 = nl > 0 && (ni == 0 || FL <= FI);
                    const int32_t nl1 = leaf0 ? nl - 1 : nl, ni1 = leaf0 ? ni : ni - 1;
                    const int64_t fl1 = leaf0 ? L1 : FL, fi1 = leaf0 ? FI : I1;
                    const bool leaf1 = nl1 > 0 && (ni1 == 0 || fl1 <= fi1);
                    const int32_t child0 = leaf0 ? V - 1 - pl : V + ih;
                    if (leaf0) ++pl;
                    else ++ih;
                    const int32_t child1 = leaf1 ? V - 1 - pl : V + ih;
                    if (leaf1) ++pl;
                    else ++ih;
                    const int64_t sum = (leaf0 ? FL : FI) + (leaf1 ? fl1 : fi1);
                    parent[child0] = a;
                    bit[child0] = 0;
                    parent[child1] = a;
                    bit[child1] = 1;
                    icount[a] = sum;
                    s_new[a - a0] = sum;
                    ++a;
                }
            }
            s_pl = pl;
            s_ih = ih;
            s_a = a;
            s_mode = mode;
            s_front = front;
            __threadfence_block();
        }
        __syncthreads();
        const int mode = s_mode;
        if (mode == 0) return;
        if (mode == 3) continue;   // windows refilled at the top of the next phase
        const int32_t pl = s_pl, ih = s_ih, a = s_a;
        const int64_t front = s_front;
        // length of the run: the queue's elements below the other front form a prefix (both queues are in
        // ascending order). The block narrows [lo, hi] around its end: each round probes the first element
        // of kMergeThreads equal blocks of the interval, so a run of any length takes a few rounds.
        const int32_t avail = mode == 1 ? V - pl : a - ih;
        int32_t lo = 0, hi = avail;   // the prefix covers [0, lo) and ends before hi
        while (lo < hi) {
            const int32_t step = (hi - lo + kMergeThreads - 1) / kMergeThreads;
            const int32_t q = lo + tid * step;
            const bool ok =
                q < hi && (mode == 1 ? leaf_val(counts, V, pl + q) <= front : icount[ih + q] < front);
            const int c = __syncthreads_count(ok);   // the probes of blocks 0 .. c-1 lie in the prefix
            const int32_t nlo = c > 0 ? lo + (c - 1) * step + 1 : lo;
            hi = min(hi, lo + c * step);
            lo = nlo;
        }
        const int32_t n = lo;
        const int32_t m = n / 2;
        if (m == 0) {   // impossible for descending counts (the probe saw a run of kRunMin)
            if (tid == 0) atomicOr(&flags[2], 1);
            return;
        }
        for (int32_t i = tid; i < m; i += kMergeThreads) {
            int32_t c0, c1;
            int64_t v0, v1;
            if (mode == 1) {
                c0 = V - 1 - (pl + 2 * i);
                c1 = c0 - 1;
                v0 = leaf_val(counts, V, pl + 2 * i);
                v1 = leaf_val(counts, V, pl + 2 * i + 1);
            } else {
                c0 = V + ih + 2 * i;
                c1 = c0 + 1;
                v0 = icount[ih + 2 * i];
                v1 = icount[ih + 2 * i + 1];
            }
            parent[c0] = a + i;
            bit[c0] = 0;
            parent[c1] = a + i;
            bit[c1] = 1;
            icount[a + i] = v0 + v1;
        }
        __threadfence_block();
        __syncthreads();
        if (tid == 0) {
            if (mode == 1) s_pl = pl + 2 * m;
            else s_ih = ih + 2 * m;
            s_a = a + m;
        }
        __syncthreads();
    }
    if (tid == 0) atomicOr(&flags[2], 1);   // phase cap reached: malformed counts
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

// Exclusive prefix sum of codelen into point_off[0..V], one block walking the array.
constexpr int kScanThreads = 1024;
__global__ __launch_bounds__(kScanThreads) void k_scan_codelen(const uint8_t *__restrict__ codelen, int32_t V,
                                                               int32_t *__restrict__ point_off,
                                                               int64_t *__restrict__ total) {
    __shared__ int64_t wsum[kScanThreads / 64];
    __shared__ int64_t carry;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    for (int32_t base = 0; base < V; base += kScanThreads) {
        const int32_t i = base + threadIdx.x;
        const int64_t x = i < V ? codelen[i] : 0;
        // inclusive wave scan
        int64_t inc = x;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int64_t y = __shfl_up(inc, d, 64);
            if (lane >= d) inc += y;
        }
        if (lane == 63) wsum[wid] = inc;
        __syncthreads();
        int64_t before = carry;
        for (int w = 0; w < wid; ++w) before += wsum[w];
        if (i < V) point_off[i] = static_cast<int32_t>(before + inc - x);
        __syncthreads();
        if (threadIdx.x == kScanThreads - 1) carry = before + inc;
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        point_off[V] = static_cast<int32_t>(carry);
        *total = carry;
    }
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
    const unsigned gv = static_cast<unsigned>(ceil_div(V, 256));
    k_zero_i32<<<1, 64, 0, s>>>(flags, 4);
    k_fill_parent<<<static_cast<unsigned>(ceil_div(2LL * V, 256)), 256, 0, s>>>(parent, 2 * V);
    k_huff_merge<<<1, kMergeThreads, 0, s>>>(vocab_counts, V, parent, bit, icount, flags);
    W2V_LAUNCH_CHECK("k_huff_merge");
    k_huff_codes<<<gv, 256, 0, s>>>(parent, bit, V, codelen, code, flags);
    W2V_LAUNCH_CHECK("k_huff_codes");
    k_scan_codelen<<<1, kScanThreads, 0, s>>>(codelen, V, point_off, total);
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
