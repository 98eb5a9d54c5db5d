// One-workgroup exclusive prefix sum shared by the per-document and noise-weight scans.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "w2v_internal.h"

namespace w2v {

// Exclusive prefix sum by one workgroup of kScanThreads threads: out[i] = in[0] + ... + in[i-1] (i < n),
// summed in int64; returns the sum of all n values (in every thread). Each thread adds kScanPer consecutive
// values per step, so a step covers kScanThreads * kScanPer values with two workgroup barriers.
constexpr int kScanThreads = 1024;
constexpr int kScanPer = 16;
template <typename In, typename Out>
__device__ int64_t block_exclusive_scan(const In *__restrict__ in, int64_t n, Out *__restrict__ out) {
    __shared__ int64_t wsum[kScanThreads / kWave];
    const int lane = lane_id(), wid = static_cast<int>(threadIdx.x / kWave);
    int64_t carry = 0;
    for (int64_t base = 0; base < n; base += static_cast<int64_t>(kScanThreads) * kScanPer) {
        const int64_t i0 = base + static_cast<int64_t>(threadIdx.x) * kScanPer;
        int64_t v[kScanPer];
        int64_t mine = 0;
#pragma unroll
        for (int k = 0; k < kScanPer; ++k) {
            v[k] = i0 + k < n ? static_cast<int64_t>(in[i0 + k]) : 0;
            mine += v[k];
        }
        int64_t inc = mine;   // inclusive scan of the threads' sums within the wavefront
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) {
            const int64_t y = __shfl_up(inc, d, kWave);
            if (lane >= d) inc += y;
        }
        if (lane == kWave - 1) wsum[wid] = inc;
        __syncthreads();
        int64_t before = carry, step = 0;
        for (int w = 0; w < kScanThreads / kWave; ++w) {
            before += w < wid ? wsum[w] : 0;
            step += wsum[w];
        }
        __syncthreads();   // wsum is rewritten by the next step
        int64_t run = before + inc - mine;
#pragma unroll
        for (int k = 0; k < kScanPer; ++k) {
            if (i0 + k < n) out[i0 + k] = static_cast<Out>(run);
            run += v[k];
        }
        carry += step;
    }
    return carry;
}

}  // namespace w2v
