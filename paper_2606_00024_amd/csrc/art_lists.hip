// Traversal lists for the decode call (Sec. 3.4): the importance-first list
// of a policy that scores KV blocks, and the sink-preserving recency-first
// list of a policy that keeps sink tokens plus a recent window.
//
// Two launches:
//   1. block scores (importance lists only), one wavefront per KV block of a
//      (sequence, KV head) group, written as doubles:
//        key norm:    max over the block's tokens of sum_d k_d^2
//        query bound: max over the group's query heads of
//                     sum_d max(q_d * min_j k_jd, q_d * max_j k_jd)
//      Every sum runs over d = 0, 1, ..., 127 in order in fp64, on exact
//      products of bf16 values, so the scores do not depend on how the work
//      is split: equal inputs give equal bits on any implementation that
//      keeps that order.
//   2. selection, one workgroup per group: a bitonic sort of (score, id)
//      pairs in LDS, descending score and ascending id; the forced blocks
//      (the first sink_blocks, and the last when asked) and the best others
//      up to the budget are kept in sorted order.  Streaming lists need no
//      scores: sinks in increasing order, then the most recent blocks.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>

#include "art.h"
#include "art_internal.h"

namespace art {
namespace {

constexpr int kListThreads = 1024;   // selection workgroup
constexpr int kMaxListBlocks = 8192; // blocks per sequence the selection sorts in LDS

struct ListParams {
    int32_t batch, num_q_heads, num_kv_heads, block_size, page_shift, num_pages;
    int32_t max_pages, max_blocks, max_list, sort_n;
    int64_t ks_page, ks_head, ks_tok;
    int32_t policy, score_kind, budget, sink_blocks, keep_last;
    const uint16_t* q;
    const uint16_t* k;
    const int32_t* page_table;
    const int32_t* seq_lens;
    int32_t* list;
    int32_t* list_len;
    double* scores;   // [groups][max_blocks]
};

typedef unsigned int u32x4_l __attribute__((ext_vector_type(4)));

__device__ __forceinline__ double bf16_lo(uint32_t w) { return (double)__uint_as_float(w << 16); }
__device__ __forceinline__ double bf16_hi(uint32_t w) { return (double)__uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ int seq_len_of(const ListParams& P, int b) {
    const int64_t cap = (int64_t)P.max_pages << P.page_shift;
    const int L = P.seq_lens[b];
    return L < 0 ? 0 : (int)(L > cap ? cap : L);
}


// wave-wide max of a double (exact)
__device__ __forceinline__ double wave_max(double x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x = fmax(x, __shfl_xor(x, o));
    return x;
}

// A wavefront reads 64 tokens (one 16 KiB tile) of a block with coalesced
// 16-byte loads: load i of lane l holds bytes 16*(l & 15) .. +15 of token
// 4i + (l >> 4), which lies in 16-token piece i / 4 of the tile (a piece
// never straddles a page: pages hold at least 16 tokens).
constexpr int kTileLoads = 16;
constexpr int kRowPitch = 272;   // bytes per token row in the LDS tile (256 + 16 of padding)

// The score kernels are persistent: wavefront w walks the blocks w, w + W,
// ... of the flattened (group, block) range (W = wavefronts in the grid),
// skipping blocks past their sequence's end, one 64-token tile at a time.
// The loads of the next tile are issued before the current tile is
// processed, and the page ids two tiles ahead before that, so that every
// wavefront keeps one tile of keys in flight while it computes.  Two things
// keep that overlap intact: every load is issued by every lane on every
// path (addresses are clamped instead of branched around, so the compiler
// can count the loads still in flight instead of waiting for all of them),
// and the two tile buffers swap roles in an unrolled pair of steps instead
// of being copied (a copy would wait for the next tile's loads).  The
// sequence lengths of the first kListLenCache sequences are read from LDS.
constexpr int kListLenCache = 256;

struct TilePos {
    int64_t item;   // flattened group * max_blocks + block; >= n_items when done
    int gidx, b, kvh, blk, t0, j1;
};

__device__ __forceinline__ int cached_len(const ListParams& P, const int* s_len, int b) {
    return b < kListLenCache ? s_len[b] : seq_len_of(P, b);
}

// The first tile of the first block at or after `item` that holds tokens.
__device__ __forceinline__ TilePos first_tile(const ListParams& P, const int* s_len, int64_t item,
                                              int64_t stride, int64_t n_items) {
    TilePos t;
    t.gidx = t.b = t.kvh = t.blk = t.t0 = 0;
    t.j1 = 1;
    for (; item < n_items; item += stride) {
        const int gidx = (int)(item / P.max_blocks), blk = (int)(item % P.max_blocks);
        const int b = gidx / P.num_kv_heads;
        const int L = cached_len(P, s_len, b);
        const int j0 = blk * P.block_size;
        if (j0 < L) {
            t.gidx = gidx; t.b = b; t.kvh = gidx % P.num_kv_heads; t.blk = blk;
            t.t0 = j0; t.j1 = min(j0 + P.block_size, L);
            break;
        }
    }
    t.item = item;
    return t;
}

__device__ __forceinline__ TilePos next_tile(const ListParams& P, const int* s_len, TilePos t,
                                             int64_t stride, int64_t n_items) {
    if (t.item >= n_items) return t;
    if (t.t0 + 64 < t.j1) {
        t.t0 += 64;
        return t;
    }
    return first_tile(P, s_len, t.item + stride, stride, n_items);
}

// Page of 16-token piece (lane & 3) of the tile, in lane n (n < 4).  Every
// lane reads a valid entry; a tile past the end reads the first one.
__device__ __forceinline__ int tile_pages(const ListParams& P, const TilePos& t, int64_t n_items,
                                          int lane) {
    const bool live = t.item < n_items;
    const int tok = live ? min(t.t0 + 16 * (lane & 3), t.j1 - 1) : 0;
    const int64_t at = live ? (int64_t)t.b * P.max_pages + (tok >> P.page_shift) : 0;
    int pg = P.page_table[at];
    return pg < 0 ? 0 : (pg >= P.num_pages ? P.num_pages - 1 : pg);
}

// Rows past the tile's end read the tile's first row again, and every row
// of a tile past the end of the work reads the pool's first row: the
// callers ignore them, and they add no memory traffic beyond a line or two.
__device__ __forceinline__ void load_tile(const ListParams& P, const TilePos& t, int pages, int64_t n_items,
                                          int lane, u32x4_l (&v)[kTileLoads]) {
    const int pmask = (1 << P.page_shift) - 1;
    const bool live = t.item < n_items;
#pragma unroll
    for (int i = 0; i < kTileLoads; ++i) {
        int tok = t.t0 + 4 * i + (lane >> 4);
        int pg = __builtin_amdgcn_readlane(pages, i >> 2);
        if (tok >= t.j1) {
            tok = t.t0;
            pg = __builtin_amdgcn_readlane(pages, 0);
        }
        const uint16_t* row = live ? P.k + pg * P.ks_page + t.kvh * P.ks_head + (int64_t)(tok & pmask) * P.ks_tok
                                   : P.k;
        v[i] = reinterpret_cast<const u32x4_l*>(row)[lane & 15];
    }
}

__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's LDS accesses are done
    __builtin_amdgcn_wave_barrier();
}

// Loads the lengths of the first kListLenCache sequences into LDS (every
// thread of the workgroup takes part; a barrier follows).
__device__ __forceinline__ void cache_lens(const ListParams& P, int* s_len) {
    for (int i = threadIdx.x; i < min(P.batch, kListLenCache); i += blockDim.x) s_len[i] = seq_len_of(P, i);
    __syncthreads();
}

// Walks this wavefront's tiles with the loads one tile ahead; `pre_fn(t)`
// issues the loads that the current tile's `block_fn` will need (before the
// next tile's keys, so that waiting for them does not wait for the keys),
// `tile_fn(t, v)` consumes a tile, `block_fn(t)` ends a block (after its
// last tile).
template <class PreFn, class TileFn, class BlockFn>
__device__ __forceinline__ void stream_tiles(const ListParams& P, const int* s_len, PreFn pre_fn,
                                             TileFn tile_fn, BlockFn block_fn) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int64_t stride = (int64_t)gridDim.x * 4;
    const int64_t n_items = (int64_t)P.batch * P.num_kv_heads * P.max_blocks;
    TilePos cur = first_tile(P, s_len, (int64_t)blockIdx.x * 4 + wave, stride, n_items);
    if (cur.item >= n_items) return;
    TilePos nxt = next_tile(P, s_len, cur, stride, n_items);
    const int pg_cur = tile_pages(P, cur, n_items, lane);
    int pg_nxt = tile_pages(P, nxt, n_items, lane);
    u32x4_l a[kTileLoads], b[kTileLoads];
    load_tile(P, cur, pg_cur, n_items, lane, a);
    // One step: the page ids two tiles ahead, the keys of the next tile into
    // `nb`, then the current tile (in `cb`).  False once the work is done.
    auto step = [&](u32x4_l (&cb)[kTileLoads], u32x4_l (&nb)[kTileLoads]) -> bool {
        const TilePos nn = next_tile(P, s_len, nxt, stride, n_items);
        const int pg_nn = tile_pages(P, nn, n_items, lane);
        pre_fn(cur);
        load_tile(P, nxt, pg_nxt, n_items, lane, nb);
        tile_fn(cur, cb);
        if (nxt.item != cur.item) block_fn(cur);
        if (nxt.item >= n_items) return false;
        cur = nxt;
        nxt = nn;
        pg_nxt = pg_nn;
        return true;
    };
    while (step(a, b) && step(b, a)) {
    }
}

// Lane j sums the 128 squares of token j in dimension order: the tile goes
// through LDS (64 rows per wavefront).  Each square of a bf16 value is exact
// in fp64, so the fused multiply-add rounds once per term, as the separate
// product and sum would.  Rows past the block's end hold its first row
// again (load_tile), which leaves the maximum unchanged.
constexpr int kKeyNormLds = 4 * 64 * kRowPitch;   // bytes per workgroup

__global__ void __launch_bounds__(256) score_key_norm_kernel(const ListParams P) {
    extern __shared__ __align__(16) unsigned char tiles[];
    __shared__ __align__(16) int s_len[kListLenCache];
    cache_lens(P, s_len);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    unsigned char* tile = tiles + w * 64 * kRowPitch;
    double best = -1.0;   // below any sum of squares
    stream_tiles(P, s_len, [](const TilePos&) {},
        [&](const TilePos&, const u32x4_l (&v)[kTileLoads]) {
#pragma unroll
            for (int i = 0; i < kTileLoads; ++i)
                *reinterpret_cast<u32x4_l*>(tile + (4 * i + (lane >> 4)) * kRowPitch + 16 * (lane & 15)) = v[i];
            wave_lds_fence();
            const unsigned char* row = tile + lane * kRowPitch;
            double s = 0.0;
#pragma unroll
            for (int c = 0; c < 16; ++c) {
                const u32x4_l x = *reinterpret_cast<const u32x4_l*>(row + 16 * c);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const double x0 = bf16_lo(x[e]), x1 = bf16_hi(x[e]);
                    s = __builtin_fma(x0, x0, s);   // dimension 8c + 2e
                    s = __builtin_fma(x1, x1, s);   // dimension 8c + 2e + 1
                }
            }
            best = fmax(best, s);
            wave_lds_fence();   // the rows are read before they are written again
        },
        [&](const TilePos& t) {
            // every lane stores the same value (no branch around the store)
            P.scores[(int64_t)t.gidx * P.max_blocks + t.blk] = wave_max(best);
            best = -1.0;
        });
}

// Lane l keeps the extremes of dimensions 8*(l & 15) .. +7 over the tokens
// its loads cover; at the end of a block the four lane rows are combined,
// the per-dimension terms of every query head go to LDS, and lane h sums
// head h's 128 terms in order.
//
// The extremes are taken on the raw bf16 words, two dimensions per
// instruction, with no conversion: a bf16 is sign and magnitude, so over a
// set of values the largest is the largest as a signed 16-bit integer when
// that one is non-negative and otherwise (all negative) the smallest as a
// signed integer; the smallest is the largest as an unsigned integer when
// any sign bit is set and otherwise the smallest as an unsigned integer.
// Four packed extremes per word (signed and unsigned, largest and
// smallest) give both.  This holds for every value but NaN (keys hold
// none) and treats -0 as the smallest negative, which changes no term:
// q * (+-0) is a zero either way and adding a zero of either sign to the
// running sum, which starts at +0, gives the same bits.  Rows past the
// block's end hold its first row again (load_tile), which changes no
// extreme.
typedef short s16x2_l __attribute__((ext_vector_type(2)));
typedef unsigned short u16x2_l __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pk_smax(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(s16x2_l, a),
                                                                  __builtin_bit_cast(s16x2_l, b)));
}
__device__ __forceinline__ uint32_t pk_smin(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_min(__builtin_bit_cast(s16x2_l, a),
                                                                  __builtin_bit_cast(s16x2_l, b)));
}
__device__ __forceinline__ uint32_t pk_umax(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(u16x2_l, a),
                                                                  __builtin_bit_cast(u16x2_l, b)));
}
__device__ __forceinline__ uint32_t pk_umin(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_min(__builtin_bit_cast(u16x2_l, a),
                                                                  __builtin_bit_cast(u16x2_l, b)));
}

// The value (as a float) of the largest and the smallest bf16 of one half
// (shift 0: low, 16: high) of the four packed extremes.
__device__ __forceinline__ void half_extremes(uint32_t smax, uint32_t smin, uint32_t umax, uint32_t umin,
                                              int shift, float& lo, float& hi) {
    const uint32_t sx = (smax >> shift) & 0xffffu, sn = (smin >> shift) & 0xffffu;
    const uint32_t ux = (umax >> shift) & 0xffffu, un = (umin >> shift) & 0xffffu;
    hi = __uint_as_float((sx < 0x8000u ? sx : sn) << 16);
    lo = __uint_as_float((ux >= 0x8000u ? ux : un) << 16);
}

template <int G>
__global__ void __launch_bounds__(256) score_query_bound_kernel(const ListParams P) {
    __shared__ double terms[4][G][128];
    __shared__ __align__(16) int s_len[kListLenCache];
    cache_lens(P, s_len);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    // word e of the lane's 16 bytes: dimensions 8c + 2e (low half), 8c + 2e + 1
    uint32_t smax[4], smin[4], umax[4], umin[4];
    auto reset = [&]() {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            smax[e] = 0x80008000u; smin[e] = 0x7fff7fffu; umax[e] = 0u; umin[e] = 0xffffffffu;
        }
    };
    reset();
    // lane row r holds dimensions 8*(lane & 15) .. +7 of query heads r, r + 4, ...
    constexpr int QR = (G + 3) / 4;
    u32x4_l qw[QR];
    const int c = lane & 15, r = lane >> 4;
    stream_tiles(P, s_len,
        [&](const TilePos& t) {
#pragma unroll
            for (int h0 = 0, u = 0; h0 < G; h0 += 4, ++u) {
                const int h = min(h0 + r, G - 1);
                qw[u] = reinterpret_cast<const u32x4_l*>(
                    P.q + ((int64_t)t.b * P.num_q_heads + t.kvh * G + h) * kHeadDim)[c];
            }
        },
        [&](const TilePos&, const u32x4_l (&v)[kTileLoads]) {
#pragma unroll
            for (int i = 0; i < kTileLoads; ++i) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    smax[e] = pk_smax(smax[e], v[i][e]); smin[e] = pk_smin(smin[e], v[i][e]);
                    umax[e] = pk_umax(umax[e], v[i][e]); umin[e] = pk_umin(umin[e], v[i][e]);
                }
            }
        },
        [&](const TilePos& t) {
            // lanes l, l ^ 16, l ^ 32, l ^ 48 hold the same dimensions
#pragma unroll
            for (int e = 0; e < 4; ++e) {
#pragma unroll
                for (int o = 16; o <= 32; o <<= 1) {
                    smax[e] = pk_smax(smax[e], (uint32_t)__shfl_xor((int)smax[e], o));
                    smin[e] = pk_smin(smin[e], (uint32_t)__shfl_xor((int)smin[e], o));
                    umax[e] = pk_umax(umax[e], (uint32_t)__shfl_xor((int)umax[e], o));
                    umin[e] = pk_umin(umin[e], (uint32_t)__shfl_xor((int)umin[e], o));
                }
            }
            float lo[8], hi[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                half_extremes(smax[e], smin[e], umax[e], umin[e], 0, lo[2 * e], hi[2 * e]);
                half_extremes(smax[e], smin[e], umax[e], umin[e], 16, lo[2 * e + 1], hi[2 * e + 1]);
            }
            // lane row r writes the terms of heads r, r + 4, ...
#pragma unroll
            for (int h0 = 0, u = 0; h0 < G; h0 += 4, ++u) {
                const int h = h0 + r;
                if (h < G) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const double q0 = bf16_lo(qw[u][e]), q1 = bf16_hi(qw[u][e]);
                        terms[w][h][8 * c + 2 * e] = fmax(q0 * (double)lo[2 * e], q0 * (double)hi[2 * e]);
                        terms[w][h][8 * c + 2 * e + 1] = fmax(q1 * (double)lo[2 * e + 1], q1 * (double)hi[2 * e + 1]);
                    }
                }
            }
            wave_lds_fence();
            double s = -INFINITY;
            if (lane < G) {
                s = 0.0;
                for (int d = 0; d < 128; ++d) s = s + terms[w][lane][d];
            }
            P.scores[(int64_t)t.gidx * P.max_blocks + t.blk] = wave_max(s);
            wave_lds_fence();   // the terms are read before the next block writes them
            reset();
        });
}

// A persistent launch of 256-thread workgroups: as many as are resident at
// once (never more than one wavefront per work item), so that no workgroup
// waits for another to finish before it starts its share.
template <class Kernel>
hipError_t launch_persistent(Kernel kernel, int64_t items, size_t lds, hipStream_t stream, const ListParams& P) {
    int dev = 0, cus = 0, per_cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, 256, lds);
    if (e != hipSuccess) return e;
    if (per_cu < 1) per_cu = 1;
    const int64_t grid = std::min<int64_t>((items + 3) / 4, (int64_t)cus * per_cu);
    hipLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(256), lds, stream, P);
    return hipGetLastError();
}

// The value that lane (lane ^ S) holds, S one of 1, 2, 4, 8, 16, 32, by
// the cross-lane moves of the vector ALU instead of a round trip through
// the LDS unit: quad permutes for 1 and 2, rotations within a row of 16
// lanes for 4 and 8 (row_ror:n hands lane i the value of lane i - n of
// its row), and the swaps of 16- and 32-lane halves for 16 and 32.
template <int S>
__device__ __forceinline__ int xor_lane(int x) {
    const int lane = threadIdx.x & 63;
    if constexpr (S == 1) {
        return __builtin_amdgcn_mov_dpp(x, 0xB1, 0xf, 0xf, false);   // quad_perm [1,0,3,2]
    } else if constexpr (S == 2) {
        return __builtin_amdgcn_mov_dpp(x, 0x4E, 0xf, 0xf, false);   // quad_perm [2,3,0,1]
    } else if constexpr (S == 4) {
        const int from_above = __builtin_amdgcn_mov_dpp(x, 0x12C, 0xf, 0xf, false);   // row_ror:12
        const int from_below = __builtin_amdgcn_mov_dpp(x, 0x124, 0xf, 0xf, false);   // row_ror:4
        return (lane & 4) ? from_below : from_above;
    } else if constexpr (S == 8) {
        return __builtin_amdgcn_mov_dpp(x, 0x128, 0xf, 0xf, false);  // row_ror:8
    } else if constexpr (S == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
        return (lane & 16) ? r[0] : r[1];
    } else {
        static_assert(S == 32, "a power of two up to 32");
        const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
        return (lane & 32) ? r[0] : r[1];
    }
}

template <int S>
__device__ __forceinline__ double xor_lane(double x) {
    const long long w = __double_as_longlong(x);
    const int lo = xor_lane<S>((int)(w & 0xffffffffll)), hi = xor_lane<S>((int)(w >> 32));
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// a before b: larger score, then smaller id
__device__ __forceinline__ bool before(double sa, int ia, double sb, int ib) {
    return sa > sb || (sa == sb && ia < ib);
}

// exclusive prefix sum of one int per thread over the workgroup
__device__ int block_exclusive_scan(int v, int* scratch, int& total) {
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    int incl = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
    }
    if (lane == 63) scratch[w] = incl;
    __syncthreads();
    if (w == 0) {
        const int nw = kListThreads / 64;
        int x = lane < nw ? scratch[lane] : 0;
        int xi = x;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(xi, o);
            if (lane >= o) xi += y;
        }
        if (lane < nw) scratch[lane] = xi - x;   // exclusive offset of wave `lane`
        if (lane == nw - 1) scratch[nw] = xi;    // total
    }
    __syncthreads();
    const int r = scratch[w] + incl - v;
    total = scratch[kListThreads / 64];
    __syncthreads();
    return r;
}

// One lane's element (k, i) at position pos through the bitonic stages
// with strides S, S/2, ..., 1 of a run of `size` positions: the lower
// position of each pair keeps whichever element comes first in a run that
// puts "before" first (up), the upper one the other; the other runs the
// other way round.
template <int S>
__device__ __forceinline__ void register_stages(double& k, int& i, bool up, int lane) {
    const double pk = xor_lane<S>(k);
    const int pi = xor_lane<S>(i);
    const bool lower = (lane & S) == 0;
    if ((lower == up) != before(k, i, pk, pi)) {
        k = pk;
        i = pi;
    }
    if constexpr (S > 1) register_stages<S / 2>(k, i, up, lane);
}

__global__ void __launch_bounds__(kListThreads) select_kernel(const ListParams P) {
    extern __shared__ __align__(16) unsigned char lds[];
    const int gidx = blockIdx.x, tid = threadIdx.x;
    const int b = gidx / P.num_kv_heads;
    const int L = seq_len_of(P, b);
    const int n = L > 0 ? (L + P.block_size - 1) / P.block_size : 0;
    int32_t* out = P.list + (int64_t)gidx * P.max_list;
    if (P.policy == ART_LIST_STREAMING) {
        const int ns = min(P.sink_blocks, n);
        const int nr = min(P.budget, n - ns);
        for (int i = tid; i < ns + nr; i += kListThreads) out[i] = i < ns ? i : n - 1 - (i - ns);
        if (tid == 0) P.list_len[gidx] = ns + nr;
        return;
    }
    // importance: sort (score, id) pairs of blocks 0..n-1, padded to sort_n
    const int N = P.sort_n;
    double* key = reinterpret_cast<double*>(lds);
    int* id = reinterpret_cast<int*>(lds + (size_t)N * sizeof(double));
    int* scratch = id + N;
    const double* sc = P.scores + (int64_t)gidx * P.max_blocks;
    for (int i = tid; i < N; i += kListThreads) {
        key[i] = i < n ? sc[i] : -INFINITY;
        id[i] = i < n ? i : 0x7fffffff;
    }
    __syncthreads();
    // Bitonic sort of positions 0..N-1 (N a power of two) into descending
    // score, ties by ascending id.  Stages with a stride of 64 or more go
    // through LDS, one pair per thread and a workgroup barrier each.  Stages
    // below a stride of 64 never leave a 64-position segment: they run in
    // registers, each wavefront taking whole segments (lane l holds position
    // 64 s + l) and exchanging with lane l ^ stride (xor_lane), so that a
    // segment is read and written once per run of such stages.  Sizes up to
    // 64 have no other stages and run in a single pass.
    const int wave = tid >> 6, lane = tid & 63;
    auto segment_pass = [&](int size_from, int size_to) {
        for (int seg = wave; seg * 64 < N; seg += kListThreads / 64) {
            const int pos = seg * 64 + lane;
            double k = pos < N ? key[pos] : -INFINITY;
            int i = pos < N ? id[pos] : 0x7fffffff;
            for (int size = size_from; size <= size_to; size <<= 1) {
                const bool up = (pos & size) == 0;   // this run sorts "before" first
                switch (min(size >> 1, 32)) {
                    case 32: register_stages<32>(k, i, up, lane); break;
                    case 16: register_stages<16>(k, i, up, lane); break;
                    case 8: register_stages<8>(k, i, up, lane); break;
                    case 4: register_stages<4>(k, i, up, lane); break;
                    case 2: register_stages<2>(k, i, up, lane); break;
                    default: register_stages<1>(k, i, up, lane); break;
                }
            }
            if (pos < N) {
                key[pos] = k;
                id[pos] = i;
            }
        }
    };
    segment_pass(2, min(N, 64));
    __syncthreads();
    for (int size = 128; size <= N; size <<= 1) {
        for (int stride = size >> 1; stride >= 64; stride >>= 1) {
            for (int p = tid; p < N / 2; p += kListThreads) {
                const int i = (p / stride) * 2 * stride + (p % stride), j = i + stride;
                const bool up = (i & size) == 0;
                const double ki = key[i], kj = key[j];
                const int ii = id[i], ij = id[j];
                const bool swap = up ? before(kj, ij, ki, ii) : before(ki, ii, kj, ij);
                if (swap) {
                    key[i] = kj; key[j] = ki;
                    id[i] = ij; id[j] = ii;
                }
            }
            __syncthreads();
        }
        segment_pass(size, size);
        __syncthreads();
    }
    // forced blocks and the budget for the others
    const int ns = min(P.sink_blocks, n);
    const int nf = ns + ((P.keep_last && n > 0 && n - 1 >= ns) ? 1 : 0);
    const int others = max(0, P.budget - nf);
    // each thread takes a run of consecutive sorted positions
    const int per = (N + kListThreads - 1) / kListThreads;
    const int p0 = tid * per;
    int cnt_other = 0;
    for (int p = p0; p < min(p0 + per, n); ++p) {
        const int i = id[p];
        const bool forced = i < ns || (P.keep_last && i == n - 1);
        cnt_other += forced ? 0 : 1;
    }
    int tot;
    int rank_other = block_exclusive_scan(cnt_other, scratch, tot);
    int cnt_sel = 0;
    {
        int r = rank_other;
        for (int p = p0; p < min(p0 + per, n); ++p) {
            const int i = id[p];
            const bool forced = i < ns || (P.keep_last && i == n - 1);
            if (forced) ++cnt_sel;
            else { if (r < others) ++cnt_sel; ++r; }
        }
    }
    int total_sel;
    int pos = block_exclusive_scan(cnt_sel, scratch, total_sel);
    {
        int r = rank_other;
        for (int p = p0; p < min(p0 + per, n); ++p) {
            const int i = id[p];
            const bool forced = i < ns || (P.keep_last && i == n - 1);
            bool take = forced;
            if (!forced) { take = r < others; ++r; }
            if (take) out[pos++] = i;
        }
    }
    if (tid == 0) P.list_len[gidx] = total_sel;
}

int ilog2_exact(int v) {
    int s = 0;
    while ((1 << s) < v) ++s;
    return (1 << s) == v ? s : -1;
}

art_status check_list(const art_decode_shape* s, const art_list_opts* o, int& max_blocks, int& sort_n) {
    if (!s || !o) return ART_ERR_INVALID_ARG;
    if (s->batch < 0 || s->num_kv_heads <= 0 || s->num_q_heads <= 0 ||
        s->num_q_heads % s->num_kv_heads != 0 || s->block_size <= 0 || s->page_size <= 0 ||
        s->num_pages <= 0 || s->max_pages_per_seq <= 0 || s->max_blocks_per_list <= 0 ||
        s->list_per_head != 1 || s->k_stride_page < 0 || s->k_stride_head < 0 || s->k_stride_token < 0)
        return ART_ERR_INVALID_ARG;
    if ((o->policy != ART_LIST_IMPORTANCE && o->policy != ART_LIST_STREAMING) || o->budget < 0 ||
        o->sink_blocks < 0 || (o->keep_last != 0 && o->keep_last != 1) ||
        (o->policy == ART_LIST_IMPORTANCE && o->score_kind != ART_SCORE_KEY_NORM &&
         o->score_kind != ART_SCORE_QUERY_BOUND))
        return ART_ERR_INVALID_ARG;
    const int g = s->num_q_heads / s->num_kv_heads;
    if (s->head_dim != kHeadDim || ilog2_exact(s->page_size) < 0) return ART_ERR_UNSUPPORTED;
    if (o->policy == ART_LIST_IMPORTANCE && o->score_kind == ART_SCORE_QUERY_BOUND &&
        g != 1 && g != 2 && g != 4 && g != 8 && g != 16)
        return ART_ERR_UNSUPPORTED;
    const int64_t mb = ((int64_t)s->max_pages_per_seq * s->page_size + s->block_size - 1) / s->block_size;
    if (mb > kMaxListBlocks) return ART_ERR_UNSUPPORTED;
    max_blocks = (int)mb;
    sort_n = 1;
    while (sort_n < max_blocks) sort_n <<= 1;
    // the longest list this call can write must fit a row
    int64_t longest;
    if (o->policy == ART_LIST_STREAMING) {
        longest = std::min<int64_t>(mb, (int64_t)o->sink_blocks + o->budget);
    } else {
        const int64_t forced = std::min<int64_t>(mb, o->sink_blocks) + (o->keep_last ? 1 : 0);
        longest = std::min<int64_t>(mb, std::max<int64_t>(o->budget, forced));
    }
    if (longest > s->max_blocks_per_list) return ART_ERR_INVALID_ARG;
    return ART_OK;
}

}  // namespace
}  // namespace art

extern "C" {

size_t art_block_list_workspace_bytes(const art_decode_shape* shape, const art_list_opts* opts,
                                      int32_t* status) {
    int mb = 0, sn = 0;
    const art_status st = art::check_list(shape, opts, mb, sn);
    if (status) *status = st;
    if (st != ART_OK) return 0;
    return (size_t)shape->batch * shape->num_kv_heads * mb * sizeof(double);
}

art_status art_build_block_list(const art_decode_shape* shape, const art_list_opts* opts,
                                const void* q, const void* k_cache, const int32_t* page_table,
                                const int32_t* seq_lens, int32_t* block_list,
                                int32_t* block_list_len, double* block_scores, void* workspace,
                                size_t workspace_bytes, hipStream_t stream) {
    using namespace art;
    int mb = 0, sn = 0;
    art_status st = check_list(shape, opts, mb, sn);
    if (st != ART_OK) return st;
    if (shape->batch == 0) return ART_OK;
    const bool importance = opts->policy == ART_LIST_IMPORTANCE;
    if (!seq_lens || !block_list || !block_list_len) return ART_ERR_INVALID_ARG;
    if (importance && (!k_cache || !page_table)) return ART_ERR_INVALID_ARG;
    if (importance && opts->score_kind == ART_SCORE_QUERY_BOUND && !q) return ART_ERR_INVALID_ARG;
    if (importance && (((uintptr_t)k_cache | (uintptr_t)(q ? q : k_cache)) % 16 ||
                       shape->k_stride_token % 8 || shape->k_stride_head % 8 || shape->k_stride_page % 8))
        return ART_ERR_UNSUPPORTED;
    const size_t need = (size_t)shape->batch * shape->num_kv_heads * mb * sizeof(double);
    double* scores = block_scores;
    if (importance && !scores) {
        if (!workspace || workspace_bytes < need) return ART_ERR_WORKSPACE_TOO_SMALL;
        if ((uintptr_t)workspace % 8) return ART_ERR_INVALID_ARG;
        scores = static_cast<double*>(workspace);
    }
    ListParams P;
    memset(&P, 0, sizeof P);
    P.batch = shape->batch;
    P.num_q_heads = shape->num_q_heads;
    P.num_kv_heads = shape->num_kv_heads;
    P.block_size = shape->block_size;
    P.page_shift = ilog2_exact(shape->page_size);
    P.num_pages = shape->num_pages;
    P.max_pages = shape->max_pages_per_seq;
    P.max_blocks = mb;
    P.max_list = shape->max_blocks_per_list;
    P.sort_n = sn;
    P.ks_page = shape->k_stride_page;
    P.ks_head = shape->k_stride_head;
    P.ks_tok = shape->k_stride_token;
    P.policy = opts->policy;
    P.score_kind = opts->score_kind;
    P.budget = opts->budget;
    P.sink_blocks = opts->sink_blocks;
    P.keep_last = opts->keep_last;
    P.q = static_cast<const uint16_t*>(q);
    P.k = static_cast<const uint16_t*>(k_cache);
    P.page_table = page_table;
    P.seq_lens = seq_lens;
    P.list = block_list;
    P.list_len = block_list_len;
    P.scores = scores;
    const int groups = shape->batch * shape->num_kv_heads;
    if (importance && (int64_t)groups * mb > 0) {
        const int64_t waves = (int64_t)groups * mb;
        if (opts->score_kind == ART_SCORE_KEY_NORM) {
            if (launch_persistent(score_key_norm_kernel, waves, kKeyNormLds, stream, P) != hipSuccess)
                return ART_ERR_HIP;
        } else {
            hipError_t e;
            switch (shape->num_q_heads / shape->num_kv_heads) {
                case 1: e = launch_persistent(score_query_bound_kernel<1>, waves, 0, stream, P); break;
                case 2: e = launch_persistent(score_query_bound_kernel<2>, waves, 0, stream, P); break;
                case 4: e = launch_persistent(score_query_bound_kernel<4>, waves, 0, stream, P); break;
                case 8: e = launch_persistent(score_query_bound_kernel<8>, waves, 0, stream, P); break;
                default: e = launch_persistent(score_query_bound_kernel<16>, waves, 0, stream, P); break;
            }
            if (e != hipSuccess) return ART_ERR_HIP;
        }
    }
    const size_t lds = importance ? (size_t)sn * (sizeof(double) + sizeof(int)) +
                                        (kListThreads / 64 + 1) * sizeof(int)
                                  : 0;
    hipLaunchKernelGGL(select_kernel, dim3((unsigned)groups), dim3(kListThreads), lds, stream, P);
    return hipGetLastError() == hipSuccess ? ART_OK : ART_ERR_HIP;
}

}  // extern "C"
