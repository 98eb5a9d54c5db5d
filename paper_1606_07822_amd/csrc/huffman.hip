// Huffman tree of the vocabulary (§2: output layer of the hierarchical softmax).
//
// Construction rule: leaves in ascending count (vocabulary index V-1 first),
// inner nodes in creation order; each merge takes the smaller front twice, a
// leaf winning a count tie; the first child taken gets bit 0; merge a creates
// inner node a (root = V-2). The merge is an inherently sequential chain; one
// lane runs it out of LDS (leaf counts and old inner counts are staged in
// chunks by the whole wave, recent inner counts sit in a ring), then parallel
// kernels derive codes, offsets and points.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "w2v_internal.h"

namespace w2v {
namespace {

constexpr int kChunk = 1024;   // leaf / inner counts staged per refill
constexpr int kRing = 4096;    // most recent inner counts

__global__ __launch_bounds__(64) void k_huff_merge(const int64_t *__restrict__ leaf_count, int32_t V,
                                                   int32_t *__restrict__ parent, uint8_t *__restrict__ bit,
                                                   int64_t *__restrict__ icount) {
    __shared__ int64_t lstage[kChunk];   // lstage[i] = count of leaf (l_hi - i)
    __shared__ int64_t istage[kChunk];   // istage[i] = icount[i_lo + i], i < i_n
    __shared__ int64_t ring[kRing];      // ring[a % kRing] = icount[a] for the last kRing merges
    __shared__ int32_t st[6];            // lf, ih, a, l_hi, i_lo, i_n
    __shared__ int32_t need;             // 1 = leaves, 2 = inner counts
    const int lane = threadIdx.x;
    if (lane == 0) {
        st[0] = V - 1; st[1] = 0; st[2] = 0; st[3] = -1; st[4] = 0; st[5] = 0;
        need = 1;
    }
    __syncthreads();
    while (true) {
        const int32_t nd = need;
        if (nd == 1) {
            const int32_t hi = st[0];
            for (int i = lane; i < kChunk; i += 64) lstage[i] = (hi - i >= 0) ? leaf_count[hi - i] : 0;
            __syncthreads();
            if (lane == 0) st[3] = hi;
        } else if (nd == 2) {
            const int32_t lo = st[1], a = st[2];
            const int32_t n = min(kChunk, a - lo);
            for (int i = lane; i < n; i += 64) istage[i] = icount[lo + i];
            __syncthreads();
            if (lane == 0) { st[4] = lo; st[5] = n; }
        }
        __syncthreads();
        if (lane == 0) {
            int32_t lf = st[0], ih = st[1], a = st[2];
            const int32_t l_hi = st[3], i_lo = st[4], i_n = st[5];
            int32_t want = 0;
            // leaf idx is readable iff staged; inner idx (< a) iff in the ring or the stage
            auto leaf_ok = [&](int32_t idx) { return idx < 0 || (idx <= l_hi && idx > l_hi - kChunk); };
            auto inner_ok = [&](int32_t idx, int32_t aa) {
                return idx >= aa || aa - idx <= kRing || (idx >= i_lo && idx < i_lo + i_n);
            };
            auto leaf_at = [&](int32_t idx) { return lstage[l_hi - idx]; };
            auto inner_at = [&](int32_t idx, int32_t aa) {
                return (aa - idx <= kRing) ? ring[idx % kRing] : istage[idx - i_lo];
            };
            while (a < V - 1) {
                if (!leaf_ok(lf) || !leaf_ok(lf - 1)) { want = 1; break; }
                if (!inner_ok(ih, a) || !inner_ok(ih + 1, a)) { want = 2; break; }
                // the two fronts of each queue, read together
                const int64_t L0 = lf >= 0 ? leaf_at(lf) : 0;
                const int64_t L1 = lf >= 1 ? leaf_at(lf - 1) : 0;
                const int64_t I0 = ih < a ? inner_at(ih, a) : 0;
                const int64_t I1 = ih + 1 < a ? inner_at(ih + 1, a) : 0;
                // first child (bit 0): a leaf wins a tie
                const bool t1 = lf >= 0 && (ih >= a || L0 <= I0);
                const int32_t c1 = t1 ? lf : V + ih;
                const int64_t v1 = t1 ? L0 : I0;
                const int32_t lf2 = t1 ? lf - 1 : lf, ih2 = t1 ? ih : ih + 1;
                const int64_t lv = t1 ? L1 : L0, iv = t1 ? I0 : I1;
                // second child (bit 1)
                const bool t2 = lf2 >= 0 && (ih2 >= a || lv <= iv);
                const int32_t c2 = t2 ? lf2 : V + ih2;
                const int64_t v2 = t2 ? lv : iv;
                lf = t2 ? lf2 - 1 : lf2;
                ih = t2 ? ih2 : ih2 + 1;
                parent[c1] = a;
                bit[c1] = 0;
                parent[c2] = a;
                bit[c2] = 1;
                const int64_t sum = v1 + v2;
                icount[a] = sum;
                ring[a % kRing] = sum;
                ++a;
            }
            st[0] = lf; st[1] = ih; st[2] = a;
            need = want;
            // make this lane's global icount stores visible to the wave before a stage refill
            __threadfence_block();
        }
        __syncthreads();
        if (need == 0) break;
    }
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
    k_huff_merge<<<1, 64, 0, s>>>(vocab_counts, V, parent, bit, icount);
    W2V_LAUNCH_CHECK("k_huff_merge");
    k_huff_codes<<<gv, 256, 0, s>>>(parent, bit, V, codelen, code, flags);
    W2V_LAUNCH_CHECK("k_huff_codes");
    k_scan_codelen<<<1, kScanThreads, 0, s>>>(codelen, V, point_off, total);
    W2V_LAUNCH_CHECK("k_scan_codelen");
    int32_t hflags[2];
    int64_t htotal = 0;
    W2V_HIP(hipMemcpyAsync(hflags, flags, sizeof(hflags), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipMemcpyAsync(&htotal, total, sizeof(htotal), hipMemcpyDeviceToHost, s));
    W2V_HIP(hipStreamSynchronize(s));
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
