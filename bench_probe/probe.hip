// Memory-system probe for the benchmark's roofline (not part of the method or
// of libw2v's interface): rows of a row-major float matrix chosen by a hash,
// read (mode 0) or read, changed and written back (mode 1) by many wavefronts
// with four rows in flight each. The training kernel's HBM traffic is this
// pattern (scattered inner-node and word rows), so the probe's rate is its
// practical memory ceiling. Modes 2 and 3 read, or write, every row exactly
// once with the same per-lane dword accesses: dispatches of known size for
// scaling the HBM byte counters. Built into its own library, libw2v_probe.so.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

// Receives the sum of a read probe in a case that never happens; visible
// outside this file, so that the reads it depends on are kept.
__device__ float w2v_probe_sink;

namespace w2v_probe {

constexpr int kWave = 64;
thread_local std::string g_err;

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

int probe_fail(const std::string &m) {
    g_err = m;
    return -1;
}
int hip_check(hipError_t e, const char *what) {
    if (e == hipSuccess) return 0;
    g_err = std::string(what) + ": " + hipGetErrorString(e);
    return -4;
}
#define PROBE_HIP(call)                                        \
    do {                                                       \
        if (int _rc = hip_check((call), #call)) return _rc;    \
    } while (0)

int run_probe_rows(float *matrix, int64_t rows, int32_t cols, int32_t row_stride, int32_t mode, int32_t workgroups,
                   int32_t iters, float *ms_host, hipStream_t s) {
    hipEvent_t e0 = nullptr, e1 = nullptr;
    PROBE_HIP(hipEventCreate(&e0));
    PROBE_HIP(hipEventCreate(&e1));
    PROBE_HIP(hipEventRecord(e0, s));
    const int nb = (cols + kWave - 1) / kWave;
    const int pick = nb <= 1 ? 1 : nb <= 2 ? 2 : nb <= 4 ? 4 : nb <= 5 ? 5 : nb <= 8 ? 8 : 16;
    launch_probe(mode, pick, workgroups, s, matrix, rows, cols, row_stride, iters);
    PROBE_HIP(hipGetLastError());
    PROBE_HIP(hipEventRecord(e1, s));
    PROBE_HIP(hipEventSynchronize(e1));
    PROBE_HIP(hipEventElapsedTime(ms_host, e0, e1));
    PROBE_HIP(hipEventDestroy(e0));
    PROBE_HIP(hipEventDestroy(e1));
    return 0;
}

}  // namespace w2v_probe

extern "C" {

/* Kernel milliseconds of one probe dispatch over matrix (float[rows][row_stride], device memory,
   16-byte aligned): wavefronts (12 per workgroup, four rows in flight each) visit rows picked by a
   32-bit hash, iters times four rows each, and read the first cols floats (mode 0) or read them,
   add 1 and write them back (mode 1; the matrix is modified). Modes 2 and 3 visit rows 0, 1, 2, ...
   instead, each at most once (wavefront w, round i: rows 4 (w iters + i) .. +3), reading (2) or
   writing (3, the matrix is modified) the first cols floats. Synchronises the stream. Returns 0;
   -1 for NULL pointers, rows < 1, cols < 1 or > min(row_stride, 1024), mode not in 0..3,
   workgroups or iters < 1 (nothing launched); -4 for a HIP failure. */
int w2v_probe_rows(float *matrix, int64_t rows, int32_t cols, int32_t row_stride, int32_t mode, int32_t workgroups,
                   int32_t iters, float *ms_host, void *hip_stream) {
    using namespace w2v_probe;
    g_err.clear();
    if (!matrix || !ms_host) return probe_fail("matrix/ms_host is NULL");
    if (rows < 1 || cols < 1 || row_stride < cols || cols > 1024)
        return probe_fail("need rows >= 1 and 1 <= cols <= min(row_stride, 1024)");
    if (mode < 0 || mode > 3) return probe_fail("mode must be in 0..3");
    if (workgroups < 1 || iters < 1) return probe_fail("workgroups and iters must be >= 1");
    return run_probe_rows(matrix, rows, cols, row_stride, mode, workgroups, iters, ms_host,
                          static_cast<hipStream_t>(hip_stream));
}

/* Message of the calling thread's last failed w2v_probe_rows call ("" after a success). */
const char *w2v_probe_last_error(void) { return w2v_probe::g_err.c_str(); }

}  // extern "C"
