// Internal declarations shared by the library's translation units (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "../../include/w2v.h"

namespace w2v {

constexpr int kWave = 64;

// ---------------------------------------------------------------- errors
void set_error(const std::string &msg);
int fail(int code, const std::string &msg);
int hip_fail(hipError_t e, const char *what);

#define W2V_HIP(call)                                            \
    do {                                                         \
        hipError_t _e = (call);                                  \
        if (_e != hipSuccess) return ::w2v::hip_fail(_e, #call); \
    } while (0)

#define W2V_LAUNCH_CHECK(what)                                            \
    do {                                                                  \
        hipError_t _e = hipGetLastError();                                \
        if (_e != hipSuccess) return ::w2v::hip_fail(_e, "launch " what); \
    } while (0)

// Bump allocator over the caller's workspace (256-byte aligned carving).
struct Carve {
    char *base;
    size_t cap, off;
    explicit Carve(void *p = nullptr, size_t c = 0) : base(static_cast<char *>(p)), cap(c), off(0) {}
    template <class T>
    T *take(size_t n) {
        off = (off + 255) & ~size_t(255);
        T *r = base ? reinterpret_cast<T *>(base + off) : nullptr;
        off += n * sizeof(T);
        return r;
    }
    size_t used() const { return (off + 255) & ~size_t(255); }
};

int device_cu_count();
size_t device_max_lds();
// Launch shape and resources of a training kernel launch, for w2v_last_train_launch / _resources.
void record_train_launch(int groups, int waves, const void *fn, int block, size_t dyn_lds);

// ----------------------------------------------------------- device helpers
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): counter (c0..c3), key (k0, k1).
struct U4 {
    uint32_t x, y, z, w;
};

__device__ __forceinline__ U4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                            uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint32_t lo0 = 0xD2511F53u * c0, hi0 = __umulhi(0xD2511F53u, c0);
        const uint32_t lo1 = 0xCD9E8D57u * c2, hi1 = __umulhi(0xCD9E8D57u, c2);
        const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return U4{c0, c1, c2, c3};
}

// The two words a raw token draws: .x decides the keep, .y the window.
__device__ __forceinline__ U4 token_draw(uint64_t seed, int64_t raw, int32_t epoch) {
    return philox4x32_10(static_cast<uint32_t>(raw), static_cast<uint32_t>(static_cast<uint64_t>(raw) >> 32),
                         static_cast<uint32_t>(epoch), 0u, static_cast<uint32_t>(seed),
                         static_cast<uint32_t>(seed >> 32));
}

__device__ __forceinline__ uint64_t fmix64(uint64_t k) {
    k ^= k >> 33;
    k *= 0xFF51AFD7ED558CCDull;
    k ^= k >> 33;
    k *= 0xC4CEB9FE1A85EC53ull;
    k ^= k >> 33;
    return k;
}

__device__ __forceinline__ int lane_id() { return static_cast<int>(threadIdx.x & (kWave - 1)); }

// Buffer-resource row access: a row is a raw buffer of dim floats at base + row * stride; columns
// past dim read as zeros and are not written, and an empty range (num_records 0) turns the row's
// loads into zeros and its stores into no-ops, so a loop can issue the same memory instructions
// every iteration without a branch.
constexpr int kRawBufferWord3 = 0x00020000;   // gfx9 raw buffer: no swizzle, 32-bit data

__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(float *base, int64_t row, int stride, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(base + row * stride, 0, bytes, kRawBufferWord3);
}

// The lane's byte offset is passed through an empty asm statement where it is used, so that the
// element steps (i * 256 bytes) stay constants of each access and become its immediate offset
// (range-checked like the lane offset) instead of one loop-invariant register per element.
__device__ __forceinline__ int lane_bytes(int lane) {
    int b = lane * 4;
    asm volatile("" : "+v"(b));
    return b;
}

template <int NE>
__device__ __forceinline__ void buf_load_row(float (&r)[NE], __amdgpu_buffer_rsrc_t rs, int lane) {
    const int b = lane_bytes(lane);
#pragma unroll
    for (int i = 0; i < NE; ++i)
        r[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, b + i * kWave * 4, 0, 0));
}

template <int NE>
__device__ __forceinline__ void buf_store_row(const float (&r)[NE], __amdgpu_buffer_rsrc_t rs, int lane) {
    const int b = lane_bytes(lane);
#pragma unroll
    for (int i = 0; i < NE; ++i)
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, r[i]), rs, b + i * kWave * 4, 0, 0);
}

// ------------------------------------------------------------------ cross-lane sums
// A row is 16 lanes; DPP moves stay within a row, permlane16/32 swaps move between rows.
template <int CTRL>
__device__ __forceinline__ float dpp_row(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}

// Sum over the 16 lanes of each row, result in every lane of the row.
__device__ __forceinline__ float row_sum(float v) {
    v += dpp_row<0xB1>(v);    // quad_perm [1,0,3,2]
    v += dpp_row<0x4E>(v);    // quad_perm [2,3,0,1]
    v += dpp_row<0x141>(v);   // row_half_mirror
    v += dpp_row<0x140>(v);   // row_mirror
    return v;
}

// Swap the upper 32 lanes of a with the lower 32 lanes of b (permlane32), or the
// odd rows of a with the even rows of b (permlane16).
__device__ __forceinline__ void swap32(float &a, float &b) {
    const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, a), __builtin_bit_cast(unsigned, b),
                                                    false, false);
    a = __builtin_bit_cast(float, static_cast<unsigned>(r[0]));
    b = __builtin_bit_cast(float, static_cast<unsigned>(r[1]));
}
__device__ __forceinline__ void swap16(float &a, float &b) {
    const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(unsigned, a), __builtin_bit_cast(unsigned, b),
                                                    false, false);
    a = __builtin_bit_cast(float, static_cast<unsigned>(r[0]));
    b = __builtin_bit_cast(float, static_cast<unsigned>(r[1]));
}

// Four per-lane partial sums -> one register whose row j (lanes 16j..16j+15)
// holds the full 64-lane sum of a_j: two permlane32 swaps, one permlane16 swap, four DPP adds.
__device__ __forceinline__ float reduce4(float a0, float a1, float a2, float a3) {
    swap32(a0, a2);
    float r = a0 + a2;   // lanes 0-31: a0, lanes 32-63: a2 (each summed over lane pairs l, l+32)
    swap32(a1, a3);
    float q = a1 + a3;   // lanes 0-31: a1, lanes 32-63: a3
    swap16(r, q);
    return row_sum(r + q);   // rows: a0 a1 a2 a3
}

// The lane's share of a dot product of two rows held element-strided (element i at column lane + 64 i).
template <int NE>
__device__ __forceinline__ float dot_partial(const float (&x)[NE], const float (&y)[NE]) {
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < NE; ++i) s = fmaf(x[i], y[i], s);
    return s;
}

// Full-wave sum, result in every lane.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
    return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
    return v;
}
__device__ __forceinline__ int64_t wave_sum(int64_t v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
    return v;
}

// ---------------------------------------------------------- sampling layout
// Per document d, slots [d*doc_len, d*doc_len + n_kept[d]) of:
//   kept_vid  int32   vocabulary index of the kept token
//   kept_meta uint32  raw offset in the document (bits 0..15) | effective half-width (bits 16..23)
struct SampleBufs {
    int32_t *kept_vid;
    uint32_t *kept_meta;
    int32_t *doc_kept;     // [n_docs]
    int64_t *doc_pairs;    // [n_docs]
    uint64_t *thr;         // [V]
    int64_t *totals;       // [4]: raw, in-vocab, kept, pairs
};

size_t sample_bufs_bytes(int32_t V, int64_t n_tokens, int32_t doc_len);
SampleBufs sample_bufs_carve(Carve &c, int32_t V, int64_t n_tokens, int32_t doc_len);

// Launches: thresholds, zero totals, per-document subsampling + window draws.
int launch_sampling(const int32_t *tokens, int64_t n_tokens, int32_t V, const int64_t *vocab_counts,
                    int64_t train_words, const w2v_params *p, const SampleBufs &b, uint8_t *keep_mask,
                    hipStream_t s);
int launch_thresholds(const int64_t *vocab_counts, int32_t V, double sample, int64_t train_words, uint64_t *thr,
                      hipStream_t s);

// Learning-rate table: alpha of 10,000-token blocks [blk0, blk0 + nblk).
int launch_alpha_table(const w2v_params *p, int64_t blk0, int64_t nblk, float *tab, hipStream_t s);

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Every inner-node row of the walk is written back by a store: uncached rows to HBM (write_policy bit 0)
// and cached rows into the workgroup's LDS copy (bit 2, or no cache), with no hot rows taking atomic adds.
// Dims above 512 columns keep the general walk.
inline bool train_stores_only(int32_t write_policy, int32_t cache_k, int32_t hot_k, int32_t dim) {
    return (write_policy & 1) && (cache_k == 0 || (write_policy & 4)) && hot_k == 0 && dim <= 512;
}

// Work units of the training kernels: a document's kept centres in segments of kSegLen, so that a
// small corpus still spreads over the whole GPU (windows still read the whole document).
constexpr int kSegLen = 128;
inline int32_t segs_per_doc(int32_t doc_len) { return static_cast<int32_t>(ceil_div(doc_len, kSegLen)); }

// Arguments of the asynchronous training kernel.
struct TrainArgs {
    float *syn0;
    float *syn1;
    int32_t V, dim, stride;
    const uint8_t *codelen;
    const uint64_t *code;
    const int32_t *point_off;
    const int32_t *points;
    const int32_t *kept_vid;
    const uint32_t *kept_meta;
    const int32_t *doc_kept;
    int64_t n_docs;
    int32_t doc_len;
    int32_t seg_len;         // work unit: up to seg_len consecutive kept centres of one document
    int32_t segs_per_doc;    // ceil(doc_len / seg_len); unit u = (document u / segs_per_doc, segment u % segs_per_doc)
    int64_t n_units;         // n_docs * segs_per_doc
    int64_t first_raw;
    int64_t epoch_base;      // epoch * corpus_tokens
    const float *alpha_tab;
    int64_t blk0;
    int32_t cache_k, cache_first, flush_every;
    int32_t atomic_first;    // uncached rows from here up take atomic adds even under the store policy
    int32_t workers;
    int32_t write_policy;
    int32_t full_rows;       // row_stride covers the variant's NE*64 columns: whole-row writes
    int32_t stores_only;     // train_stores_only(): every inner-node row is written back by a store
    float flush_scale;       // fraction of the cached rows' change written back (1 = all of it)
    int32_t cache_delta;     // delta-only cache: LDS holds the workgroup's change of each cached row only
    int32_t span_refresh;    // word-row span: words below this index are written back and re-read every centre
    int32_t span_stash;      // word-row span: the re-entering centre row may wait in a per-wave LDS row
    int32_t stash_from;      // word-row span: the stash takes words of vocabulary index >= stash_from only
    int32_t stash_off;       // word-row span: floats into the dynamic LDS of the per-wave stash row (-1: none)
    int32_t *queue;
    unsigned long long *stats;   // [3]: kept, pairs, node updates
    float *egrad;            // per wavefront egrad_slots rows of row_stride floats (parked gradients), or null
    int32_t egrad_slots;
};

// The log-likelihood call's argument checks and body (workspace of w2v_hs_loglik_workspace_bytes bytes),
// shared by w2v_hs_loglik and its variant on the library's static scratch.
int check_loglik_args(const w2v_model *m, const int32_t *tokens, int64_t n_tokens, const w2v_params *p,
                      const double *sum_ll_host, const int64_t *n_pairs_host);
int loglik_run(const w2v_model *m, const int32_t *tokens, int64_t n_tokens, const w2v_params *p, double *sum_ll_host,
               int64_t *n_pairs_host, int64_t *n_nodes_host, void *workspace, hipStream_t s);

}  // namespace w2v
