// Asynchronous HS training (Algorithm 1, Cached Skipgram HS), GPU form.
//
// Worker = one wavefront. Wavefronts claim work units from a queue -- segments
// of up to 128 consecutive kept centres of one document -- and walk their
// centre words in order (windows still read the whole document). Per centre v with window words
// w_1..w_P the path of v is walked once, four inner nodes at a time: the
// four rows are loaded together (the next four are prefetched), every window
// word in order updates all four (dot, sigmoid, gradient, two axpys), and the
// change of each row is written back once. The hidden-layer gradients of the
// window words stay in registers and are added to syn0 after the path.
// Swapping the window and node loops of Algorithm 1 this way is the same
// computation whenever a window holds no repeated word; the four nodes of a
// chunk never interact (a path visits distinct nodes).
//
// Cross-lane work of one window word and a chunk: the four dot products are
// reduced together (two permlane32 swaps, one permlane16 swap, four DPP adds),
// leaving node j's value in the 16 lanes of row j; the sigmoid and gradient
// are then evaluated for the four nodes at once.
//
// Cache (§3.2): the cache owner is the workgroup. The rows of the top
// cache_k inner nodes (the k created last by the Huffman merge) sit in LDS as
// `val` (current) and `orig` (value at the last write-back); waves update
// `val` with LDS atomic adds of their change, or (write_policy bit 2) store
// their new row into it, lock-free like the HBM rows. Every flush_every centres of the
// workgroup, one wave writes flush_scale * (val - orig) back to HBM with an
// atomic add and re-bases both copies on the returned HBM value (write-back
// plus refill, without stopping the other waves).
//
// Rows are spread over the 64 lanes element-strided: lane l holds elements
// l, l+64, l+128, ... so every row access is a run of coalesced 256-byte
// accesses.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "w2v_internal.h"

namespace w2v {
namespace {

constexpr int kChunk = 4;            // inner nodes per step (one per 16-lane row)
constexpr int kMinUnitsPerWave = 8;  // automatic launch size: work units (document segments) per wavefront, at least

__device__ __forceinline__ float sigmoid_fast(float z) { return __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }

__device__ __forceinline__ void lds_add(float *p, float v) { atomicAdd(p, v); }

// One wave writes the cache's change back to HBM and re-bases val/orig on the
// result. LDS rows are ls floats apart (ls >= dim, padding kept at zero). The
// cache_k * dim elements go B per lane at a time: their atomic adds are
// all issued before the first returned value is used, so a flush costs a few
// round trips to memory rather than one per row and column. (B = 16; a kernel
// that keeps word rows in registers across centres uses fewer, as those rows
// stay live through the flush.)
constexpr int kFlushBatch = 16;

template <int B>
__device__ void flush_cache_wave(const TrainArgs &a, bool delta, float *val, float *orig, int ls, int lane) {
    const int n = a.cache_k * a.dim;
    if (delta) {
        // delta-only cache: add the scaled change to HBM and take the whole of it out of LDS (changes
        // that other waves add meanwhile stay); the next reads see the HBM row with the written share
        for (int i = lane; i < n; i += kWave) {
            const int s = i / a.dim, col = i - s * a.dim;
            const float d = val[s * ls + col];
            if (d != 0.0f) {
                atomicAdd(a.syn1 + static_cast<int64_t>(a.cache_first + s) * a.stride + col, d * a.flush_scale);
                lds_add(val + s * ls + col, -d);
            }
        }
        return;
    }
    for (int i0 = 0; i0 < n; i0 += B * kWave) {
        float c[B], d[B], old[B];
        int li[B];
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int i = i0 + b * kWave + lane;
            const int s = i / a.dim, col = i - s * a.dim;
            li[b] = s * ls + col;
            c[b] = 0.0f;
            d[b] = 0.0f;
            old[b] = 0.0f;
            if (i < n) {
                c[b] = val[li[b]];
                d[b] = (c[b] - orig[li[b]]) * a.flush_scale;
                if (d[b] != 0.0f) old[b] = atomicAdd(a.syn1 + static_cast<int64_t>(a.cache_first + s) * a.stride + col, d[b]);
            }
        }
#pragma unroll
        for (int b = 0; b < B; ++b) {
            if (d[b] != 0.0f) {
                const float nv = old[b] + d[b];
                lds_add(val + li[b], nv - c[b]);
                orig[li[b]] = nv;
            }
        }
    }
}

// Global row -> registers; columns past dim read as zero.
template <int NE>
__device__ __forceinline__ void load_row(float (&r)[NE], const float *__restrict__ p, int lane, int dim) {
#pragma unroll
    for (int i = 0; i < NE; ++i) {
        const int col = lane + i * kWave;
        r[i] = (col < dim) ? p[col] : 0.0f;
    }
}

// Cached rows in LDS. Up to 8 elements per lane they are padded with zeros to
// NE*64 columns, so that whole rows are read and added without lane masks; the
// widest variant keeps them dim floats apart to fit 2 cache_k rows in LDS.
template <int NE>
constexpr bool pad_lds() { return NE <= 8; }

template <int NE>
__host__ __device__ __forceinline__ int lds_stride(int dim) { return pad_lds<NE>() ? NE * kWave : dim; }

// Centre records of a segment in LDS (16 bytes per centre and wave), except for the widest rows.
template <int NE>
constexpr bool rec_slots() { return NE <= 8; }

template <int NE>
__device__ __forceinline__ void load_row_lds(float (&r)[NE], const float *p, int lane, int dim) {
    if constexpr (pad_lds<NE>()) {
#pragma unroll
        for (int i = 0; i < NE; ++i) r[i] = p[lane + i * kWave];
    } else {
        load_row<NE>(r, p, lane, dim);
    }
}

template <int NE>
__device__ __forceinline__ void store_row_lds(float *p, const float (&r)[NE], int lane, int dim) {
#pragma unroll
    for (int i = 0; i < NE; ++i)
        if (pad_lds<NE>() || lane + i * kWave < dim) p[lane + i * kWave] = r[i];
}

// Row writes. With full rows (row_stride >= NE*64) all NE*64 columns are written
// (the padding columns receive zeros / zero changes) and no lane is masked.
template <int NE>
__device__ __forceinline__ void store_row(float *p, const float (&r)[NE], int lane, int dim, bool full) {
    if (full) {
#pragma unroll
        for (int i = 0; i < NE; ++i) p[lane + i * kWave] = r[i];
    } else {
#pragma unroll
        for (int i = 0; i < NE; ++i)
            if (lane + i * kWave < dim) p[lane + i * kWave] = r[i];
    }
}

template <int NE>
__device__ __forceinline__ void atomic_add_row(float *p, const float (&r)[NE], int lane, int dim, bool full) {
    if (full) {
#pragma unroll
        for (int i = 0; i < NE; ++i) atomicAdd(p + lane + i * kWave, r[i]);
    } else {
#pragma unroll
        for (int i = 0; i < NE; ++i)
            if (lane + i * kWave < dim) atomicAdd(p + lane + i * kWave, r[i]);
    }
}

template <int NE>
__device__ __forceinline__ void zero_row(float (&r)[NE]) {
#pragma unroll
    for (int i = 0; i < NE; ++i) r[i] = 0.0f;
}

// Rows of nodes c0 .. c0+3 of the path (zeros past its end), from LDS when cached.
template <int NE>
__device__ __forceinline__ void load_chunk(float (&y)[kChunk][NE], const TrainArgs &a, const float *val, int my_pt,
                                           int c0, int len, int lane) {
#pragma unroll
    for (int j = 0; j < kChunk; ++j) {
        if (c0 + j < len) {
            const int n = __builtin_amdgcn_readlane(my_pt, c0 + j);
            if (n >= a.cache_first && !a.cache_delta) {
                load_row_lds<NE>(y[j], val + (n - a.cache_first) * lds_stride<NE>(a.dim), lane, a.dim);
            } else {
                load_row<NE>(y[j], a.syn1 + static_cast<int64_t>(n) * a.stride, lane, a.dim);
                if (n >= a.cache_first) {   // delta-only cache: the HBM row plus the workgroup's change
                    float d[NE];
                    load_row_lds<NE>(d, val + (n - a.cache_first) * lds_stride<NE>(a.dim), lane, a.dim);
#pragma unroll
                    for (int i = 0; i < NE; ++i) y[j][i] += d[i];
                }
            }
        } else {
            zero_row<NE>(y[j]);
        }
    }
}

// HBM rows of path nodes c0 .. c0+3; cached rows and rows past the path's end read as zeros.
template <int NE>
__device__ __forceinline__ void load_chunk_buf(float (&y)[kChunk][NE], const TrainArgs &a, int my_pt, int c0,
                                               int len, int lane) {
#pragma unroll
    for (int j = 0; j < kChunk; ++j) {
        const int n = __builtin_amdgcn_readlane(my_pt, min(c0 + j, kWave - 1));
        const bool hbm = c0 + j < len && n < a.cache_first;
        buf_load_row<NE>(y[j], row_rsrc(a.syn1, hbm ? n : 0, a.stride, hbm ? a.dim * 4 : 0), lane);
    }
}

// The window words and the path of centre q of the segment (record r, kept position j0 + q): lane l of wv receives the vocabulary index of the l-th window word, lane l of pt the
// l-th node of the path (PATH false: none). Lanes past the window or the path read zero through
// the buffers' range checks, so the loads issue without a branch and stay in flight while the
// centre before is trained.
// Record of centre q of the segment starting at kept position j0: vocabulary index, meta, path
// offset, path length. REC: from the wave's LDS slots; else from the kept and tree arrays (the
// widest rows leave no LDS for the slots).
template <bool REC>
__device__ __forceinline__ int4 centre_record(const TrainArgs &a, const int4 *rec, const int32_t *kv,
                                              const uint32_t *km, int j0, int q) {
    if constexpr (REC) {
        return rec[q];
    } else {
        const int v = kv[j0 + q];
        return make_int4(v, static_cast<int>(km[j0 + q]), a.point_off[v], static_cast<int>(a.codelen[v]));
    }
}

template <bool PATH, bool WV = true>
__device__ __forceinline__ void fetch_centre(const TrainArgs &a, int4 r, const int32_t *kv, int nk, int j0, int q,
                                             int lane, int &wv, int &pt) {
    const int j = j0 + q;
    const int eff = static_cast<int>(static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(r.y)) >> 16);
    const int lo = max(0, j - eff), hi = min(nk - 1, j + eff);
    const int c = lo + lane + ((lo + lane >= j) ? 1 : 0);
    const auto kr = __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t *>(kv), 0, nk * 4, kRawBufferWord3);
    if constexpr (WV) wv = static_cast<int>(__builtin_amdgcn_raw_buffer_load_b32(kr, lane < hi - lo ? c * 4 : nk * 4, 0, 0));
    if constexpr (PATH) {
        const int po = __builtin_amdgcn_readfirstlane(r.z), len = __builtin_amdgcn_readfirstlane(r.w);
        const auto pr = __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t *>(a.points) + po, 0, len * 4,
                                                          kRawBufferWord3);
        pt = static_cast<int>(__builtin_amdgcn_raw_buffer_load_b32(pr, lane_bytes(lane), 0, 0));
    }
}

// Every input x[p0..p1), in order, updates the nc live rows of the chunk held in
// yc (dot, sigmoid, gradient, then e += g y and y += g x for each row).
template <int NE, int PG>
__device__ __forceinline__ void chunk_update(float (&yc)[kChunk][NE], const float (&x)[PG][NE], float (&e)[PG][NE],
                                             int p0, int p1, int nc, int c0, uint64_t code, float alpha,
                                             int lane) {
    // row j's code bit t (lane >> 4 = j; bits past the path only reach rows that are not live), folded
    // into the gradient g = alpha (1 - t) - alpha sigmoid(z)
    const uint32_t bits = static_cast<uint32_t>(code >> min(c0, 63));
    const float a1t = ((bits >> (lane >> 4)) & 1u) ? 0.0f : alpha;
    const float nalpha = -alpha;
#pragma unroll
    for (int p = 0; p < PG; ++p) {
        if (p >= p0 && p < p1) {
            const float z = reduce4(dot_partial<NE>(x[p], yc[0]), dot_partial<NE>(x[p], yc[1]),
                                    dot_partial<NE>(x[p], yc[2]), dot_partial<NE>(x[p], yc[3]));
            const float gr = fmaf(sigmoid_fast(z), nalpha, a1t);
#pragma unroll
            for (int j = 0; j < kChunk; ++j) {
                if (j < nc) {
                    const float gj =
                        __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gr), 16 * j));
#pragma unroll
                    for (int i = 0; i < NE; ++i) {
                        e[p][i] = fmaf(gj, yc[j][i], e[p][i]);
                        yc[j][i] = fmaf(gj, x[p][i], yc[j][i]);
                    }
                }
            }
        }
    }
}

// Write-back of a chunk from its change yc - y0: LDS atomic add for cached rows,
// HBM store of the new row (write_policy bit 0) or atomic add of the change.
template <int NE>
__device__ __forceinline__ void chunk_write_delta(const TrainArgs &a, float *val, const float (&yc)[kChunk][NE],
                                                  const float (&y0)[kChunk][NE], int my_pt, int c0, int nc, int lane) {
#pragma unroll
    for (int j = 0; j < kChunk; ++j) {
        if (j < nc) {
            const int n = __builtin_amdgcn_readlane(my_pt, c0 + j);
            float d[NE];
#pragma unroll
            for (int i = 0; i < NE; ++i) d[i] = yc[j][i] - y0[j][i];
            if (n >= a.cache_first) {
                float *lrow = val + (n - a.cache_first) * lds_stride<NE>(a.dim);
                if (a.write_policy & 4) {
                    store_row_lds<NE>(lrow, yc[j], lane, a.dim);
                } else {
#pragma unroll
                    for (int i = 0; i < NE; ++i)
                        if (pad_lds<NE>() || lane + i * kWave < a.dim) lds_add(lrow + lane + i * kWave, d[i]);
                }
            } else {
                float *grow = a.syn1 + static_cast<int64_t>(n) * a.stride;
                if ((a.write_policy & 1) && n < a.atomic_first) store_row<NE>(grow, yc[j], lane, a.dim, a.full_rows);
                else atomic_add_row<NE>(grow, d, lane, a.dim, a.full_rows);
            }
        }
    }
}

// Prefetch modes of the path walk.
//   kPfNone   : each chunk is loaded after the previous one is written back.
//   kPfAll    : the next chunk is loaded while the current one is updated.
//   kPfSuffix : the path's cached and hot nodes form a prefix (an inner node is
//               created after its children, so indices fall from the root down
//               and the top indices sit at the top of every path). Chunks that
//               hold a row written back as a change (atomic add) keep their
//               loaded values (y0); the chunks after them, whose rows are
//               stored, need no copy, and those registers hold the prefetched
//               next chunk instead. With every row stored the whole path is
//               prefetched.
//   kPfBuf    : every row is written back by a store; buffer loads and stores with
//               empty ranges keep each chunk's memory instructions the same, so
//               the next chunk's loads stay in flight through the compute.
[[maybe_unused]] constexpr int kPfNone = 0;
constexpr int kPfAll = 1, kPfSuffix = 2, kPfBuf = 3;

// One chunk of the pipelined walk: issue the loads of the next chunk (c0 + 4 ..) into nxt, fill the
// cached rows of this chunk from LDS, update it, and store it (LDS copy or HBM).
template <int NE, int PG>
__device__ __forceinline__ void walk_chunk_buf(const TrainArgs &a, float *val, float (&cur)[kChunk][NE],
                                               float (&nxt)[kChunk][NE], const float (&x)[PG][NE],
                                               float (&e)[PG][NE], int p0, int p1, int my_pt, int c0, int len,
                                               uint64_t code, float alpha, int lane) {
    load_chunk_buf<NE>(nxt, a, my_pt, c0 + kChunk, len, lane);
    int node[kChunk];   // read once, used by the LDS fill and the write-back
#pragma unroll
    for (int j = 0; j < kChunk; ++j) {
        node[j] = __builtin_amdgcn_readlane(my_pt, min(c0 + j, kWave - 1));
        if (c0 + j < len && node[j] >= a.cache_first)
            load_row_lds<NE>(cur[j], val + (node[j] - a.cache_first) * lds_stride<NE>(a.dim), lane, a.dim);
    }
    const int nc = min(kChunk, len - c0);
    chunk_update<NE, PG>(cur, x, e, p0, p1, nc, c0, code, alpha, lane);
#pragma unroll
    for (int j = 0; j < kChunk; ++j) {
        const int n = node[j];
        const bool live = j < nc;
        if (live && n >= a.cache_first)
            store_row_lds<NE>(val + (n - a.cache_first) * lds_stride<NE>(a.dim), cur[j], lane, a.dim);
        const bool hbm = live && n < a.cache_first;
        buf_store_row<NE>(cur[j], row_rsrc(a.syn1, hbm ? n : 0, a.stride, hbm ? a.dim * 4 : 0), lane);
    }
}

// Walk the path of the centre with the inputs x[p0..p1) (in order), accumulating
// the hidden-layer gradients into e[p0..p1). PG = size of the input arrays.
template <int NE, int PG, int PF>
__device__ __forceinline__ void walk_path(const TrainArgs &a, float *val, const float (&x)[PG][NE],
                                          float (&e)[PG][NE], int p0, int p1, int my_pt, int len, uint64_t code, float alpha,
                                          int lane) {
    float yc[kChunk][NE], y0[kChunk][NE];
    if constexpr (PF == kPfBuf) {
        // Every row is written back by a store (HBM rows to HBM, cached rows into the LDS copy):
        // the pipelined walk. Each chunk issues the same memory instructions -- buffer loads of the
        // next chunk and buffer stores of this one, with empty ranges where a row is cached or past
        // the path's end -- so the wait before a chunk's first use counts only the memory operations
        // issued after its loads, and the next chunk's loads stay in flight during the compute.
        if constexpr (NE == 5) {
            // the two register sets take turns (the loop body walks two chunks), so no chunk is copied
            // (measured faster at five elements per lane, slower at two and four, where the doubled
            // loop body costs more than the copies)
            load_chunk_buf<NE>(yc, a, my_pt, 0, len, lane);
            for (int c0 = 0; c0 < len; c0 += 2 * kChunk) {
                walk_chunk_buf<NE, PG>(a, val, yc, y0, x, e, p0, p1, my_pt, c0, len, code, alpha, lane);
                if (c0 + kChunk >= len) break;
                walk_chunk_buf<NE, PG>(a, val, y0, yc, x, e, p0, p1, my_pt, c0 + kChunk, len, code, alpha, lane);
            }
        } else {
            // the prefetched rows are copied at the end of the loop body, behind this chunk's stores, so
            // that their wait is counted within one iteration
            load_chunk_buf<NE>(y0, a, my_pt, 0, len, lane);
#pragma unroll
            for (int j = 0; j < kChunk; ++j)
#pragma unroll
                for (int i = 0; i < NE; ++i) yc[j][i] = y0[j][i];
            for (int c0 = 0; c0 < len; c0 += kChunk) {
                walk_chunk_buf<NE, PG>(a, val, yc, y0, x, e, p0, p1, my_pt, c0, len, code, alpha, lane);
#pragma unroll
                for (int j = 0; j < kChunk; ++j)
#pragma unroll
                    for (int i = 0; i < NE; ++i) yc[j][i] = y0[j][i];
            }
        }
        return;
    }
    if constexpr (PF == kPfAll) {
        float yn[kChunk][NE];
        load_chunk<NE>(yc, a, val, my_pt, 0, len, lane);
        for (int c0 = 0; c0 < len; c0 += kChunk) {
            if (c0 + kChunk < len) load_chunk<NE>(yn, a, val, my_pt, c0 + kChunk, len, lane);
#pragma unroll
            for (int j = 0; j < kChunk; ++j)
#pragma unroll
                for (int i = 0; i < NE; ++i) y0[j][i] = yc[j][i];
            const int nc = min(kChunk, len - c0);
            chunk_update<NE, PG>(yc, x, e, p0, p1, nc, c0, code, alpha, lane);
            chunk_write_delta<NE>(a, val, yc, y0, my_pt, c0, nc, lane);
            if (c0 + kChunk < len) {
#pragma unroll
                for (int j = 0; j < kChunk; ++j)
#pragma unroll
                    for (int i = 0; i < NE; ++i) yc[j][i] = yn[j][i];
            }
        }
        return;
    }
    int end_delta = len;   // chunks starting below this keep y0
    if constexpr (PF == kPfSuffix) {
        if (a.write_policy & 1) {
            // changes are needed for hot rows (atomic adds) and for cached rows unless those are stored
            const bool adds = !(a.write_policy & 4) || a.atomic_first < a.cache_first;
            const uint64_t kept = __ballot(adds && lane < len && my_pt >= a.atomic_first);
            end_delta = __popcll(kept);
        }
    }
    int c0 = 0;
    for (; c0 < end_delta; c0 += kChunk) {
        load_chunk<NE>(yc, a, val, my_pt, c0, len, lane);
#pragma unroll
        for (int j = 0; j < kChunk; ++j)
#pragma unroll
            for (int i = 0; i < NE; ++i) y0[j][i] = yc[j][i];
        const int nc = min(kChunk, len - c0);
        chunk_update<NE, PG>(yc, x, e, p0, p1, nc, c0, code, alpha, lane);
        chunk_write_delta<NE>(a, val, yc, y0, my_pt, c0, nc, lane);
    }
    if constexpr (PF == kPfSuffix) {
        // rows written back by stores (LDS for cached rows); y0's registers carry the next chunk
        if (c0 < len) load_chunk<NE>(yc, a, val, my_pt, c0, len, lane);
        for (; c0 < len; c0 += kChunk) {
            if (c0 + kChunk < len) load_chunk<NE>(y0, a, val, my_pt, c0 + kChunk, len, lane);
            const int nc = min(kChunk, len - c0);
            chunk_update<NE, PG>(yc, x, e, p0, p1, nc, c0, code, alpha, lane);
#pragma unroll
            for (int j = 0; j < kChunk; ++j) {
                if (j < nc) {
                    const int n = __builtin_amdgcn_readlane(my_pt, c0 + j);
                    if (n >= a.cache_first)
                        store_row_lds<NE>(val + (n - a.cache_first) * lds_stride<NE>(a.dim), yc[j], lane, a.dim);
                    else
                        store_row<NE>(a.syn1 + static_cast<int64_t>(n) * a.stride, yc[j], lane, a.dim, a.full_rows);
                }
            }
            if (c0 + kChunk < len) {
#pragma unroll
                for (int j = 0; j < kChunk; ++j)
#pragma unroll
                    for (int i = 0; i < NE; ++i) yc[j][i] = y0[j][i];
            }
        }
    }
}

// Word rows kept across centres (write_policy bit 3, skip-gram): while a wavefront walks the
// centres of a segment in order, the rows of the words at kept positions j-H .. j-1 and
// j+1 .. j+H of the current centre j (H = PG/2) stay in registers. Slot q < H holds position
// j-H+q, slot q >= H position j+1+q-H, so a centre's window words are the contiguous slots
// H-(j-lo) .. H+(hi-j)-1, in window order. A row is loaded when its position comes within H of
// the centre and stored when it leaves the span or becomes the centre, so each word row is read
// and written about twice per centre instead of once per pair. Slots holding the same word are
// kept equal (up to the order in which they add each other's changes): a change made to one is added to
// the others, and a word entering the span is copied
// from a slot that holds it rather than read from memory.
template <int PG>
__device__ __forceinline__ int span_pairs(int sid, int lane) {
    int n = 0;
#pragma unroll
    for (int q = 0; q < PG - 1; ++q) {
        const int w = __builtin_amdgcn_readlane(sid, q);
        n += __popcll(__ballot(w >= 0 && lane > q && lane < PG && sid == w));
    }
    return n;
}

// Row of slot q from memory (zeros when the slot lies outside the document).
template <int NE, int PG>
__device__ __forceinline__ void span_load(float (&xw)[PG][NE], int q, const TrainArgs &a, int sid, int lane) {
    const int w = __builtin_amdgcn_readlane(sid, q);
    buf_load_row<NE>(xw[q], row_rsrc(a.syn0, w >= 0 ? w : 0, a.stride, w >= 0 ? a.dim * 4 : 0), lane);
}

template <int NE, int PG>
__device__ __forceinline__ void span_store(const float (&xw)[PG][NE], int q, const TrainArgs &a, int sid, int lane) {
    const int w = __builtin_amdgcn_readlane(sid, q);
    store_row<NE>(a.syn0 + static_cast<int64_t>(w) * a.stride, xw[q], lane, a.dim, a.full_rows);
}

// Slot DST takes a new word w (sid already updated): a copy of a slot below PG - 1 other than DST
// that holds w, else the row from memory. Returns the slot's dirty bit.
// pre: when pre_ok, the row of w as this wavefront last held it, which memory also holds in a one-wavefront
// run (the stashed row of the centre word, re-entering the span as slot H-1).
template <int NE, int PG, int DST>
__device__ __forceinline__ uint32_t span_enter(float (&xw)[PG][NE], const TrainArgs &a, int sid, uint32_t dirty,
                                               int &pairs, int lane, const float (&pre)[NE], bool pre_ok) {
    const int w = __builtin_amdgcn_readlane(sid, DST);
    const uint64_t m = w >= 0 ? __ballot(lane < PG - 1 && lane != DST && sid == w) : 0ull;
    pairs += __popcll(m);
    if (m == 0ull) {
        if (pre_ok) {
#pragma unroll
            for (int i = 0; i < NE; ++i) xw[DST][i] = pre[i];
        } else {
            span_load<NE, PG>(xw, DST, a, sid, lane);
        }
        return 0u;
    }
    // the copy goes through an empty asm statement per slot, which keeps the slots' branches apart (merged,
    // they would become an indexed read of xw and move the whole array to scratch memory)
    const uint64_t first = m & (~m + 1ull);
#pragma unroll
    for (int q = 0; q < PG - 1; ++q) {
        if (first == (1ull << q)) {
#pragma unroll
            for (int i = 0; i < NE; ++i) {
                float t = xw[q][i];
                asm volatile("" : "+v"(t));
                xw[DST][i] = t;
            }
        }
    }
    return (dirty >> __builtin_ctzll(m)) & 1u;
}

// After a centre: the active slots take their changes, which also go to every other slot of the same word.
template <int NE, int PG>
__device__ __forceinline__ void span_apply(float (&xw)[PG][NE], const float (&e)[PG][NE], int p0, int p1, int sid,
                                           bool dup, uint32_t &dirty, int lane) {
#pragma unroll
    for (int q = 0; q < PG; ++q)
        if (q >= p0 && q < p1)
#pragma unroll
            for (int i = 0; i < NE; ++i) xw[q][i] += e[q][i];
    dirty |= ((1u << p1) - 1u) & ~((1u << p0) - 1u);
    if (!dup) return;
#pragma unroll
    for (int q = 0; q < PG; ++q) {
        if (q >= p0 && q < p1) {
            const int w = __builtin_amdgcn_readlane(sid, q);
            const uint64_t m = __ballot(lane < PG && lane != q && sid == w);
#pragma unroll
            for (int r = 0; r < PG; ++r) {
                if ((m >> r) & 1ull) {
#pragma unroll
                    for (int i = 0; i < NE; ++i) xw[r][i] += e[q][i];
                    dirty |= 1u << r;
                }
            }
        }
    }
}

// The same after a CBOW centre, where every active slot takes the one gradient e.
template <int NE, int PG>
__device__ __forceinline__ void span_apply_same(float (&xw)[PG][NE], const float (&e)[NE], int p0, int p1, int sid,
                                                bool dup, uint32_t &dirty, int lane) {
    // a slot's total: e once per active slot holding its word (itself included when active)
    uint32_t mult[PG];
#pragma unroll
    for (int r = 0; r < PG; ++r) mult[r] = (r >= p0 && r < p1) ? 1u : 0u;
    if (dup) {
#pragma unroll
        for (int q = 0; q < PG; ++q) {
            if (q >= p0 && q < p1) {
                const int w = __builtin_amdgcn_readlane(sid, q);
                const uint64_t m = __ballot(lane < PG && lane != q && sid == w);
#pragma unroll
                for (int r = 0; r < PG; ++r) mult[r] += static_cast<uint32_t>((m >> r) & 1ull);
            }
        }
    }
#pragma unroll
    for (int r = 0; r < PG; ++r) {
        for (uint32_t c = 0; c < mult[r]; ++c)
#pragma unroll
            for (int i = 0; i < NE; ++i) xw[r][i] += e[i];
        if (mult[r]) dirty |= 1u << r;
    }
}

// Move the span from centre j to centre j+1: slot 0 (position j-H) and slot H (position j+1, the
// next centre) leave, stored if changed; the rest shift down one slot; slot H-1 takes the old centre
// word v and slot PG-1 the word at position j+1+H (w_edge, -1 past the document's end).
// stash (LDS, one row per wavefront, or null): slot H's row is the next centre's word, which leaves the span
// now and comes back as slot H-1 at the next shift; its row is kept in the stash meanwhile (stash_w: the
// word stashed, -1 for none) and taken from there instead of memory, unless another slot holds the word,
// a slot leaving at that shift wrote it back, or the word is a frequent one (index below stash_from or
// span_refresh), whose row other wavefronts are likely to have changed meanwhile.
template <int NE, int PG>
__device__ __forceinline__ void span_shift(float (&xw)[PG][NE], const TrainArgs &a, int &sid, uint32_t &dirty,
                                           int &pairs, int v, int w_edge, int lane, float *stash, int &stash_w) {
    constexpr int H = PG / 2;
    constexpr uint32_t low = (1u << (H - 1)) - 1u;
    float back[NE];            // the current centre's row, stashed at the previous shift
    bool back_ok = false;
    if (stash) {
        const int w0 = __builtin_amdgcn_readlane(sid, 0), wh = __builtin_amdgcn_readlane(sid, H);
        back_ok = stash_w >= 0 && stash_w == v && !((dirty & 1u) && w0 == v) && !(((dirty >> H) & 1u) && wh == v) &&
                  !(v < a.span_refresh) && v >= a.stash_from;
        if (back_ok) {
#pragma unroll
            for (int i = 0; i < NE; ++i) back[i] = stash[lane + i * kWave];
        }
#pragma unroll
        for (int i = 0; i < NE; ++i) stash[lane + i * kWave] = xw[H][i];
        stash_w = wh;
    }
    // frequent words (index below span_refresh) that stay in the span are written back here and read
    // again after the shift, which bounds how long other wavefronts' updates to them can be overwritten
    const bool refresh = a.span_refresh > 0;
    if (refresh) {
#pragma unroll
        for (int q = 1; q < PG; ++q) {
            if (q == H) continue;
            const int w = __builtin_amdgcn_readlane(sid, q);
            if (w >= 0 && w < a.span_refresh && ((dirty >> q) & 1u)) {
                span_store<NE, PG>(xw, q, a, sid, lane);
                dirty &= ~(1u << q);
            }
        }
    }
    if (dirty & 1u) span_store<NE, PG>(xw, 0, a, sid, lane);
    if ((dirty >> H) & 1u) span_store<NE, PG>(xw, H, a, sid, lane);
    if (pairs > 0) {   // equal pairs that slots 0 and H leave behind
        const int w0 = __builtin_amdgcn_readlane(sid, 0), wh = __builtin_amdgcn_readlane(sid, H);
        pairs -= w0 >= 0 ? __popcll(__ballot(lane > 0 && lane < PG && sid == w0)) : 0;
        pairs -= wh >= 0 ? __popcll(__ballot(lane != 0 && lane != H && lane < PG && sid == wh)) : 0;
    }
#pragma unroll
    for (int q = 0; q + 1 < H; ++q)
#pragma unroll
        for (int i = 0; i < NE; ++i) xw[q][i] = xw[q + 1][i];
#pragma unroll
    for (int q = H; q + 1 < PG; ++q)
#pragma unroll
        for (int i = 0; i < NE; ++i) xw[q][i] = xw[q + 1][i];
    dirty = ((dirty >> 1) & low) | (((dirty >> (H + 1)) & low) << H);
    const int src = (lane < H - 1 || (lane >= H && lane < PG - 1)) ? lane + 1 : lane;
    sid = __shfl(sid, src, kWave);
    sid = lane == H - 1 ? v : (lane == PG - 1 ? w_edge : sid);
    if (refresh) {
#pragma unroll
        for (int q = 0; q < PG - 1; ++q) {
            if (q == H - 1) continue;
            const int w = __builtin_amdgcn_readlane(sid, q);
            if (w >= 0 && w < a.span_refresh) span_load<NE, PG>(xw, q, a, sid, lane);
        }
    }
    dirty |= span_enter<NE, PG, H - 1>(xw, a, sid, dirty, pairs, lane, back, back_ok) << (H - 1);
    dirty |= span_enter<NE, PG, PG - 1>(xw, a, sid, dirty, pairs, lane, back, false) << (PG - 1);
}


// ARCH 0: skip-gram, window words in groups of PG; ARCH 1: CBOW (one input, the mean); ARCH 2: skip-gram
// with the reversed orientation (the window word's path, the centre's vector as input).
// SLIDE (skip-gram, windows of at most PG/2 each side): word rows kept across centres.
template <int NE, int PG, int ARCH, int WPB, int PF, bool SLIDE = false>
__global__ __launch_bounds__(WPB *kWave) void k_train(TrainArgs a) {
    static_assert(!SLIDE || (ARCH == 0 && PF == kPfBuf && PG % 2 == 0) || (ARCH == 1 && PG % 2 == 0),
                  "word rows kept across centres: skip-gram on the store-only walk, or CBOW");
    const int LS = lds_stride<NE>(a.dim);
    extern __shared__ float lds[];
    float *val = lds;
    float *orig = lds + a.cache_k * LS;
    __shared__ unsigned s_centres;   // centres of the workgroup since its last write-back, modulo flush_every
    __shared__ int s_lock;
    constexpr bool kRec = rec_slots<NE>();
    __shared__ int4 s_rec[kRec ? WPB : 1][kRec ? kSegLen : 1];   // per wave: its current segment's centre records
    const int lane = lane_id();
    const int wib = static_cast<int>(threadIdx.x / kWave);
    // the store-only walk never runs with the delta-only cache (its cached rows take LDS adds)
    const bool delta = PF != kPfBuf && a.cache_delta != 0;
    if (threadIdx.x == 0) {
        s_centres = 0;
        s_lock = 0;
    }
    const int kd = a.cache_k * LS;
    for (int i = threadIdx.x; i < kd; i += blockDim.x) {
        if (delta) {   // delta-only cache: no change yet (and no copy of the original)
            val[i] = 0.0f;
            continue;
        }
        const int s = i / LS, col = i - s * LS;
        const float v = col < a.dim ? a.syn1[static_cast<int64_t>(a.cache_first + s) * a.stride + col] : 0.0f;
        val[i] = v;
        orig[i] = v;
    }
    __syncthreads();

    const int gw = blockIdx.x * WPB + wib;
    uint64_t n_kept = 0, n_pairs = 0, n_nodes = 0;
    if (gw < a.workers) {
        while (true) {
            int unit = 0;
            if (lane == 0) unit = atomicAdd(a.queue, 1);
            unit = __builtin_amdgcn_readfirstlane(unit);
            if (unit >= a.n_units) break;
            const int doc = unit / a.segs_per_doc;
            const int nk = a.doc_kept[doc];
            const int j0 = (unit - doc * a.segs_per_doc) * a.seg_len;
            if (j0 >= nk) continue;
            const int j1 = min(nk, j0 + a.seg_len);
            const int64_t base = static_cast<int64_t>(doc) * a.doc_len;
            const int32_t *kv = a.kept_vid + base;
            const uint32_t *km = a.kept_meta + base;
            // stage the segment's centre records in the wave's LDS slots: one round of gathers per
            // segment instead of a chain of dependent loads per centre
            int4 *rec = s_rec[kRec ? wib : 0];
            if constexpr (kRec) {
                for (int q = lane; q < j1 - j0; q += kWave) {
                    const int v = kv[j0 + q];
                    rec[q] = make_int4(v, static_cast<int>(km[j0 + q]), a.point_off[v], static_cast<int>(a.codelen[v]));
                }
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            }
            int wv_next = 0, pt_next = 0;
            fetch_centre<ARCH != 2, !SLIDE>(a, centre_record<kRec>(a, rec, kv, km, j0, 0), kv, nk, j0, 0, lane, wv_next,
                                    pt_next);
            constexpr int H = PG / 2;
            float xw[SLIDE ? PG : 1][NE];
            int sid = -1;
            uint32_t dirty = 0;
            int pairs = 0;   // slot pairs holding the same word
            float *stash = (SLIDE && a.stash_off >= 0) ? lds + a.stash_off + wib * NE * kWave : nullptr;
            int stash_w = -1;
            if constexpr (SLIDE) {
                const int pos = lane < H ? j0 - H + lane : j0 + 1 + lane - H;
                sid = (lane < PG && pos >= 0 && pos < nk) ? kv[pos] : -1;
#pragma unroll
                for (int q = 0; q < PG; ++q) span_load<NE, PG>(xw, q, a, sid, lane);
                pairs = span_pairs<PG>(sid, lane);
            }
            for (int j = j0; j < j1; ++j) {
                const int4 r = centre_record<kRec>(a, rec, kv, km, j0, j - j0);
                const int v = __builtin_amdgcn_readfirstlane(r.x);
                const uint32_t meta = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(r.y));
                // window words (lane q: the q-th one) and path nodes of this centre, fetched during the
                // centre before; the next centre's are issued now
                int wv = wv_next, my_pt = pt_next;
                asm volatile("" : "+v"(wv), "+v"(my_pt));   // one wait for the fetched values here, none at their uses
                const int qn = min(j + 1, j1 - 1) - j0;
                fetch_centre<ARCH != 2, !SLIDE>(a, centre_record<kRec>(a, rec, kv, km, j0, qn), kv, nk, j0, qn, lane, wv_next,
                                        pt_next);
                const int eff = static_cast<int>(meta >> 16);
                const int lo = max(0, j - eff), hi = min(nk - 1, j + eff);
                const int P = hi - lo;   // window words, centre excluded
                [[maybe_unused]] const int w_edge = (SLIDE && j + 1 + H < nk) ? kv[j + 1 + H] : -1;
                ++n_kept;
                if (P > 0) {
                    const int64_t g = a.epoch_base + a.first_raw + base + static_cast<int64_t>(meta & 0xFFFFu);
                    const float alpha = a.alpha_tab[g / 10000 - a.blk0];
                    const int len = ARCH == 2 ? 0 : __builtin_amdgcn_readfirstlane(r.w);
                    const uint64_t code = ARCH == 2 ? 0 : a.code[v];

                    if constexpr (SLIDE && ARCH == 1) {
                        // CBOW: h = mean of the active slots' rows (window order); one path walk; every
                        // active slot takes the hidden-layer gradient
                        const int p0 = H - (j - lo), p1 = H + (hi - j);
                        float h[1][NE], e[1][NE];
                        zero_row<NE>(h[0]);
                        zero_row<NE>(e[0]);
#pragma unroll
                        for (int q = 0; q < PG; ++q)
                            if (q >= p0 && q < p1)
#pragma unroll
                                for (int i = 0; i < NE; ++i) h[0][i] += xw[q][i];
                        const float fP = static_cast<float>(P);
#pragma unroll
                        for (int i = 0; i < NE; ++i) h[0][i] = h[0][i] / fP;
                        walk_path<NE, 1, PF>(a, val, h, e, 0, 1, my_pt, len, code, alpha, lane);
                        span_apply_same<NE, PG>(xw, e[0], p0, p1, sid, pairs > 0, dirty, lane);
                        n_nodes += len;
                    } else if constexpr (SLIDE) {
                        const int p0 = H - (j - lo), p1 = H + (hi - j);
                        // only the active slots' gradients are accumulated, read and applied
                        float e[PG][NE];
#pragma unroll
                        for (int q = 0; q < PG; ++q)
                            if (q >= p0 && q < p1) zero_row<NE>(e[q]);
                        walk_path<NE, PG, PF>(a, val, xw, e, p0, p1, my_pt, len, code, alpha, lane);
                        span_apply<NE, PG>(xw, e, p0, p1, sid, pairs > 0, dirty, lane);
                        n_nodes += static_cast<uint64_t>(P) * len;
                    } else if constexpr (ARCH == 0) {
                        // groups of PG window words walk the path in turn (one group when P <= PG). With
                        // several groups the hidden-layer gradients are parked in the wavefront's egrad
                        // rows and added to syn0 after the last group, so that every group reads the
                        // window vectors as they were before this centre (as a single walk does).
                        const bool defer = P > PG;
                        float *eg = a.egrad + static_cast<int64_t>(gw) * a.egrad_slots * a.stride;
                        for (int g0 = 0; g0 < P; g0 += PG) {
                            const int nx = min(PG, P - g0);
                            float x[PG][NE], e[PG][NE];
#pragma unroll
                            for (int p = 0; p < PG; ++p) {
                                if (p < nx) {
                                    const int w = __builtin_amdgcn_readlane(wv, g0 + p);
                                    if constexpr (PF == kPfBuf)
                                        buf_load_row<NE>(x[p], row_rsrc(a.syn0, w, a.stride, a.dim * 4), lane);
                                    else
                                        load_row<NE>(x[p], a.syn0 + static_cast<int64_t>(w) * a.stride, lane, a.dim);
                                } else {
                                    zero_row<NE>(x[p]);
                                }
                                zero_row<NE>(e[p]);
                            }
                            walk_path<NE, PG, PF>(a, val, x, e, 0, nx, my_pt, len, code, alpha, lane);
                            if (defer) {
#pragma unroll
                                for (int p = 0; p < PG; ++p)
                                    if (p < nx) store_row<NE>(eg + static_cast<int64_t>(g0 + p) * a.stride, e[p],
                                                              lane, a.dim, a.full_rows);
                                continue;
                            }
#pragma unroll
                            for (int p = 0; p < PG; ++p) {
                                if (p < nx) {
                                    const int w = __builtin_amdgcn_readlane(wv, g0 + p);
                                    float *xr = a.syn0 + static_cast<int64_t>(w) * a.stride;
                                    // a word repeated in the window: its first position stores the row
                                    // read before the centre plus its change, later ones add theirs
                                    const bool rep = (a.write_policy & 2) && __ballot(lane < g0 + p && wv == w) != 0ull;
                                    if ((a.write_policy & 2) && !rep) {
                                        float nx_[NE];
#pragma unroll
                                        for (int i = 0; i < NE; ++i) nx_[i] = x[p][i] + e[p][i];
                                        store_row<NE>(xr, nx_, lane, a.dim, a.full_rows);
                                    } else {
                                        atomic_add_row<NE>(xr, e[p], lane, a.dim, a.full_rows);
                                    }
                                }
                            }
                        }
                        if (defer) {
                            for (int q = 0; q < P; ++q) {
                                const int w = __builtin_amdgcn_readlane(wv, q);
                                float *xr = a.syn0 + static_cast<int64_t>(w) * a.stride;
                                float eq[NE];
                                load_row<NE>(eq, eg + static_cast<int64_t>(q) * a.stride, lane, a.dim);
                                if (a.write_policy & 2) {
                                    float cur[NE];
                                    load_row<NE>(cur, xr, lane, a.dim);
#pragma unroll
                                    for (int i = 0; i < NE; ++i) cur[i] += eq[i];
                                    store_row<NE>(xr, cur, lane, a.dim, a.full_rows);
                                } else {
                                    atomic_add_row<NE>(xr, eq, lane, a.dim, a.full_rows);
                                }
                            }
                        }
                        n_nodes += static_cast<uint64_t>(P) * len;
                    } else if constexpr (ARCH == 2) {
                        // reversed orientation: for each window word w in order, the path of w is walked with
                        // the centre's vector as input, which then gains that pair's hidden-layer gradient
                        // before the next pair (pair-major, as Algorithm 1 with the roles of v and w swapped)
                        float x[1][NE], e[1][NE], x0[NE];
                        float *xr = a.syn0 + static_cast<int64_t>(v) * a.stride;
                        load_row<NE>(x[0], xr, lane, a.dim);
#pragma unroll
                        for (int i = 0; i < NE; ++i) x0[i] = x[0][i];
                        int nodes = 0;
                        for (int q = 0; q < P; ++q) {
                            const int w = __builtin_amdgcn_readlane(wv, q);
                            const int lw = a.codelen[w];
                            const uint64_t cw = a.code[w];
                            const int pw = (lane < lw) ? a.points[a.point_off[w] + lane] : 0;
                            zero_row<NE>(e[0]);
                            walk_path<NE, 1, PF>(a, val, x, e, 0, 1, pw, lw, cw, alpha, lane);
#pragma unroll
                            for (int i = 0; i < NE; ++i) x[0][i] += e[0][i];
                            nodes += lw;
                        }
                        if (a.write_policy & 2) {
                            store_row<NE>(xr, x[0], lane, a.dim, a.full_rows);
                        } else {
#pragma unroll
                            for (int i = 0; i < NE; ++i) x0[i] = x[0][i] - x0[i];
                            atomic_add_row<NE>(xr, x0, lane, a.dim, a.full_rows);
                        }
                        n_nodes += nodes;
                    } else {
                        // CBOW: h = mean of the window vectors; one path walk; e added to each window vector
                        float h[1][NE], e[1][NE];
                        zero_row<NE>(h[0]);
                        zero_row<NE>(e[0]);
                        for (int p = 0; p < P; ++p) {
                            const int w = __builtin_amdgcn_readlane(wv, p);
                            float xr[NE];
                            load_row<NE>(xr, a.syn0 + static_cast<int64_t>(w) * a.stride, lane, a.dim);
#pragma unroll
                            for (int i = 0; i < NE; ++i) h[0][i] += xr[i];
                        }
                        const float fP = static_cast<float>(P);
#pragma unroll
                        for (int i = 0; i < NE; ++i) h[0][i] = h[0][i] / fP;
                        walk_path<NE, 1, PF>(a, val, h, e, 0, 1, my_pt, len, code, alpha, lane);
                        for (int p = 0; p < P; ++p) {
                            const int w = __builtin_amdgcn_readlane(wv, p);
                            float *xr = a.syn0 + static_cast<int64_t>(w) * a.stride;
                            if (a.write_policy & 2) {
                                float cur[NE];
                                load_row<NE>(cur, xr, lane, a.dim);
#pragma unroll
                                for (int i = 0; i < NE; ++i) cur[i] += e[0][i];
                                store_row<NE>(xr, cur, lane, a.dim, a.full_rows);
                            } else {
                                atomic_add_row<NE>(xr, e[0], lane, a.dim, a.full_rows);
                            }
                        }
                        n_nodes += len;
                    }
                    n_pairs += P;
                }
                if (a.cache_k > 0) {
                    // the counter wraps at flush_every (ds_inc), so the increment that completes a multiple
                    // of flush_every centres returns flush_every - 1
                    int go = 0;
                    if (lane == 0) {
                        const unsigned c = atomicInc(&s_centres, static_cast<unsigned>(a.flush_every - 1));
                        if (c == static_cast<unsigned>(a.flush_every - 1)) go = (atomicCAS(&s_lock, 0, 1) == 0) ? 1 : 0;
                    }
                    go = __builtin_amdgcn_readfirstlane(go);
                    if (go) {
                        flush_cache_wave<SLIDE ? 2 : kFlushBatch>(a, delta, val, orig, LS, lane);
                        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
                        if (lane == 0) atomicExch(&s_lock, 0);
                    }
                }
                if constexpr (SLIDE) {
                    if (j + 1 < j1) span_shift<NE, PG>(xw, a, sid, dirty, pairs, v, w_edge, lane, stash, stash_w);
                }
            }
            if constexpr (SLIDE) {
#pragma unroll
                for (int q = 0; q < PG; ++q)
                    if ((dirty >> q) & 1u) span_store<NE, PG>(xw, q, a, sid, lane);
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
        const float d = (delta ? val[i] : val[i] - orig[i]) * a.flush_scale;
        const int s = i / LS, col = i - s * LS;
        if (d != 0.0f && col < a.dim) atomicAdd(a.syn1 + static_cast<int64_t>(a.cache_first + s) * a.stride + col, d);
    }
}

struct Variant {
    void (*fn)(TrainArgs);
    int waves_per_block;
    int ne;   // elements per lane
    int pg;   // window words per path walk (skip-gram)
    int (*ls)(int);
    int rec_bytes;   // static LDS of the centre records
};

template <int NE, int PG, int WPB, int PF>
Variant variant(int arch, bool slide) {
    constexpr int rb = rec_slots<NE>() ? WPB * kSegLen * static_cast<int>(sizeof(int4)) : 0;
    if constexpr (PF == kPfBuf && NE >= 4 && PG % 2 == 0)
        if (arch == 0 && slide) return Variant{k_train<NE, PG, 0, WPB, PF, true>, WPB, NE, PG, lds_stride<NE>, rb};
    if constexpr (NE >= 4 && NE <= 8)   // CBOW keeps ten word slots (its walk has a single input row)
        if (arch == 1 && slide) return Variant{k_train<NE, 10, 1, WPB, PF, true>, WPB, NE, 10, lds_stride<NE>, rb};
    if (arch == 0) return Variant{k_train<NE, PG, 0, WPB, PF>, WPB, NE, PG, lds_stride<NE>, rb};
    if (arch == 2) return Variant{k_train<NE, 1, 2, WPB, PF>, WPB, NE, 1, lds_stride<NE>, rb};
    return Variant{k_train<NE, 1, 1, WPB, PF>, WPB, NE, 1, lds_stride<NE>, rb};
}

// Register budget per lane: x and e take 2*PG*NE, the chunk rows 2 (3 with the
// prefetch) * 4 * NE. Occupancy beats prefetch: at dim 300, 3 waves per SIMD
// without the prefetch ran 21 % faster than 2 with it.
// buf: every row is written back by a store (train_stores_only), the pipelined walk.
// slide: skip-gram word rows kept across centres (the pipelined walk only; the caller checks the window).
Variant pick_variant(int arch, int dim, bool buf, bool slide = false) {
    const int ne = (dim + kWave - 1) / kWave;
    if (ne <= 1) return buf ? variant<1, 20, 16, kPfBuf>(arch, false) : variant<1, 20, 16, kPfAll>(arch, false);
    if (ne <= 2) return buf ? variant<2, 20, 12, kPfBuf>(arch, false) : variant<2, 20, 12, kPfAll>(arch, false);
    if (ne <= 4) return buf ? variant<4, 10, 12, kPfBuf>(arch, slide) : variant<4, 10, 12, kPfAll>(arch, slide);
    if (ne <= 5) return buf ? variant<5, 10, 12, kPfBuf>(arch, slide) : variant<5, 10, 12, kPfSuffix>(arch, slide);
    if (ne <= 8) return buf ? variant<8, 4, 8, kPfBuf>(arch, slide) : variant<8, 4, 8, kPfSuffix>(arch, slide);
    return variant<16, 2, 8, kPfSuffix>(arch, false);
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

size_t train_lds_bytes(int32_t cache_k, int32_t dim, bool delta) {
    const Variant v = pick_variant(0, dim, false);   // the LDS layout is the same for every path
    return (delta ? 1ull : 2ull) * cache_k * v.ls(dim) * sizeof(float) + static_cast<size_t>(v.rec_bytes);
}

// Dynamic LDS of the word-row span's stash (one row per wavefront) when it is asked for (span_stash) and
// fits beside the cache and the centre records; 0 otherwise (the span then reads the re-entering centre
// word from memory).
size_t span_stash_bytes(const Variant &v, size_t cache_lds, bool slide) {
    if (!slide) return 0;
    const size_t b = static_cast<size_t>(v.waves_per_block) * v.ne * kWave * sizeof(float);
    return cache_lds + b + static_cast<size_t>(v.rec_bytes) + 1024 <= device_max_lds() ? b : 0;
}

int train_launch_shape(int arch, int dim, int cache_k, bool delta, bool buf, int workers, int64_t n_units, int *grid,
                       int *waves, bool slide, bool stash) {
    const Variant v = pick_variant(arch, dim, buf, slide);
    if (workers > 0) {
        *grid = static_cast<int>(ceil_div(workers, v.waves_per_block));
        *waves = workers;
        return W2V_OK;
    }
    const size_t cache_lds = (delta ? 1ull : 2ull) * cache_k * v.ls(dim) * sizeof(float);
    const size_t lds = cache_lds + span_stash_bytes(v, cache_lds, slide && stash);
    int per_cu = 0;
    W2V_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(v.fn),
                                                         v.waves_per_block * kWave, lds));
    int64_t g = static_cast<int64_t>(device_cu_count()) * std::max(1, per_cu);
    // every wavefront gets at least kMinUnitsPerWave work units, so that every workgroup
    // (cache owner) contributes to the averaged write-back of the cached rows
    const int64_t by_units = ceil_div(n_units, static_cast<int64_t>(v.waves_per_block) * kMinUnitsPerWave);
    g = std::max<int64_t>(1, std::min<int64_t>(g, by_units));
    *grid = static_cast<int>(g);
    *waves = *grid * v.waves_per_block;
    return W2V_OK;
}

int64_t train_egrad_floats(int arch, int dim, bool buf, int stride, int window, int waves) {
    const Variant v = pick_variant(arch, dim, buf);
    if (arch != 0 || 2 * window <= v.pg) return 0;
    return static_cast<int64_t>(waves) * 2 * window * stride;
}

// Word rows kept across centres (write_policy bit 3 with bit 1): skip-gram on the pipelined walk or CBOW,
// rows of 129 to 512 floats (the narrower variants measured no faster with it), and a window whose both
// sides fit the variant's register slots.
bool train_slide(int arch, int dim, bool buf, int write_policy, int window) {
    if ((arch == 0 && !buf) || arch == 2 || (write_policy & 10) != 10 || dim <= 2 * kWave || dim > 8 * kWave)
        return false;
    return 2 * window <= pick_variant(arch, dim, buf, true).pg;
}

int train_word_span(int arch, int dim, bool buf, int write_policy, int window) {
    return train_slide(arch, dim, buf, write_policy, window) ? pick_variant(arch, dim, buf, true).pg / 2 : 0;
}

int launch_train_async(TrainArgs a, int arch, int window, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s,
                       int64_t *stats_out, const int64_t *totals) {
    const bool slide = train_slide(arch, a.dim, a.stores_only != 0, a.write_policy, window);
    const Variant v = pick_variant(arch, a.dim, a.stores_only != 0, slide);
    const size_t cache_lds = (a.cache_delta ? 1ull : 2ull) * a.cache_k * v.ls(a.dim) * sizeof(float);
    const size_t stash = span_stash_bytes(v, cache_lds, slide && a.span_stash != 0);
    a.stash_off = stash ? static_cast<int32_t>(cache_lds / sizeof(float)) : -1;
    const size_t lds = cache_lds + stash;
    const int block = v.waves_per_block * kWave;
    a.full_rows = a.stride >= v.ne * kWave ? 1 : 0;
    if (lds + v.rec_bytes > 64 * 1024)   // static (records) plus dynamic (cache) LDS above the default limit
        W2V_HIP(hipFuncSetAttribute(reinterpret_cast<const void *>(v.fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                                    static_cast<int>(lds)));
    int grid = 0, waves = 0;
    if (int rc = train_launch_shape(arch, a.dim, a.cache_k, a.cache_delta != 0, a.stores_only != 0, a.workers,
                                    a.n_units, &grid, &waves, slide, a.span_stash != 0))
        return rc;
    a.workers = waves;
    if (train_egrad_floats(arch, a.dim, a.stores_only != 0, a.stride, window, waves) > 0) {
        if (!a.egrad) return fail(W2V_E_ARG, "internal: egrad rows missing");
        a.egrad_slots = 2 * window;
    }
    if (a.flush_scale <= 0.0f) a.flush_scale = 1.0f / static_cast<float>(grid);
    record_train_launch(grid, a.workers, reinterpret_cast<const void *>(v.fn), block, lds);
    k_zero_train<<<1, 64, 0, s>>>(a.queue, a.stats);
    W2V_LAUNCH_CHECK("k_zero_train");
    if (ev0) W2V_HIP(hipEventRecord(ev0, s));
    hipLaunchKernelGGL(v.fn, dim3(grid), dim3(block), lds, s, a);
    W2V_LAUNCH_CHECK("k_train");
    if (ev1) W2V_HIP(hipEventRecord(ev1, s));
    if (stats_out) {
        k_write_stats<<<1, 64, 0, s>>>(totals, a.stats, stats_out);
        W2V_LAUNCH_CHECK("k_write_stats");
    }
    return W2V_OK;
}

}  // namespace w2v
