// Memory-system probe for the roofline of the training kernel: rows of a
// row-major float matrix chosen by a hash, read (mode 0) or read, changed and
// written back (mode 1) by many wavefronts with four rows in flight each. The
// training kernel's HBM traffic is exactly this pattern (scattered inner-node
// and word rows), so the probe's rate is its practical memory ceiling. Modes 2
// and 3 read, or write, every row exactly once with the same per-lane dword
// accesses: dispatches of known size for scaling the HBM byte counters.
#include <hip/hip_runtime.h>

#include "w2v_internal.h"

// Receives the sum of a read probe in a case that never happens; visible
// outside this file, so that the reads it depends on are kept.
__device__ float w2v_probe_sink;

namespace w2v {
namespace {

constexpr int kProbeRows = 4;   // rows in flight per wavefront

__device__ __forceinline__ uint32_t mix32(uint32_t x) {
    x ^= x >> 16;
    x *= 0x7feb352dU;
    x ^= x >> 15;
    x *= 0x846ca68bU;
    x ^= x >> 16;
    return x;
}

// NB = 64-column blocks per row (cols <= 64 NB); no block is wholly masked off, so every
// memory instruction moves data, as in the training kernel.
template <int MODE, int NB>
__global__ __launch_bounds__(768) void k_probe(float *m, int64_t rows, int cols, int stride, int iters) {
    const int lane = static_cast<int>(threadIdx.x) & (kWave - 1);
    const uint32_t w = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    float acc = 0.0f;
    for (int it = 0; it < iters; ++it) {
        float *p[kProbeRows];
        bool live[kProbeRows];
#pragma unroll
        for (int r = 0; r < kProbeRows; ++r) {
            int64_t row;
            if (MODE <= 1) {
                row = mix32(w * 0x9E3779B1u + static_cast<uint32_t>(it * kProbeRows + r)) % static_cast<uint64_t>(rows);
            } else {
                row = (static_cast<int64_t>(w) * iters + it) * kProbeRows + r;   // each row once
            }
            live[r] = row < rows;
            p[r] = m + (live[r] ? row : 0) * stride;
        }
        // all of a round's loads are issued before its stores: a load waited for after a store
        // also waits for that store, which would serialise the blocks
        float v[kProbeRows][NB];
        if (MODE != 3) {
#pragma unroll
            for (int r = 0; r < kProbeRows; ++r)
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    const int col = b * kWave + lane;
                    v[r][b] = (live[r] && col < cols) ? p[r][col] : 0.0f;
                }
        }
#pragma unroll
        for (int r = 0; r < kProbeRows; ++r)
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const int col = b * kWave + lane;
                if (MODE == 0 || MODE == 2) acc += v[r][b];
                else if (MODE == 1 && live[r] && col < cols) p[r][col] = v[r][b] + 1.0f;
                else if (MODE == 3 && live[r] && col < cols) p[r][col] = static_cast<float>(it);
            }
    }
    if (acc == -1.0f) w2v_probe_sink = acc;
}

}  // namespace

template <int NB>
void launch_nb(int mode, int wg, hipStream_t s, float *m, int64_t rows, int cols, int stride, int iters) {
    switch (mode) {
        case 0: k_probe<0, NB><<<wg, 768, 0, s>>>(m, rows, cols, stride, iters); break;
        case 1: k_probe<1, NB><<<wg, 768, 0, s>>>(m, rows, cols, stride, iters); break;
        case 2: k_probe<2, NB><<<wg, 768, 0, s>>>(m, rows, cols, stride, iters); break;
        default: k_probe<3, NB><<<wg, 768, 0, s>>>(m, rows, cols, stride, iters); break;
    }
}

void launch_probe(int mode, int nb, int wg, hipStream_t s, float *m, int64_t rows, int cols, int stride, int iters) {
    switch (nb) {
        case 1: launch_nb<1>(mode, wg, s, m, rows, cols, stride, iters); break;
        case 2: launch_nb<2>(mode, wg, s, m, rows, cols, stride, iters); break;
        case 4: launch_nb<4>(mode, wg, s, m, rows, cols, stride, iters); break;
        case 5: launch_nb<5>(mode, wg, s, m, rows, cols, stride, iters); break;
        case 8: launch_nb<8>(mode, wg, s, m, rows, cols, stride, iters); break;
        default: launch_nb<16>(mode, wg, s, m, rows, cols, stride, iters); break;
    }
}

int run_probe_rows(float *matrix, int64_t rows, int32_t cols, int32_t row_stride, int32_t mode, int32_t workgroups,
                   int32_t iters, float *ms_host, hipStream_t s) {
    hipEvent_t e0 = nullptr, e1 = nullptr;
    W2V_HIP(hipEventCreate(&e0));
    W2V_HIP(hipEventCreate(&e1));
    W2V_HIP(hipEventRecord(e0, s));
    const int nb = (cols + kWave - 1) / kWave;
    const int pick = nb <= 1 ? 1 : nb <= 2 ? 2 : nb <= 4 ? 4 : nb <= 5 ? 5 : nb <= 8 ? 8 : 16;
    launch_probe(mode, pick, workgroups, s, matrix, rows, cols, row_stride, iters);
    W2V_LAUNCH_CHECK("k_probe");
    W2V_HIP(hipEventRecord(e1, s));
    W2V_HIP(hipEventSynchronize(e1));
    W2V_HIP(hipEventElapsedTime(ms_host, e0, e1));
    W2V_HIP(hipEventDestroy(e0));
    W2V_HIP(hipEventDestroy(e1));
    return W2V_OK;
}

}  // namespace w2v
