// Fused aggregate + optimize kernel of the exchange step, for gfx950.
//
// One wave plays the role of one PHub core (paper, section 3.2.4): it walks
// the list of chunks the schedule fixed for it at initialisation, and for
// each element it sums the N workers' gradients
// (section 3.2.2, "tall" aggregation: one worker takes the same chunk
// across all gradient arrays) and immediately runs the optimizer on that
// element (section 3.2.2: the thread that aggregates a chunk also
// optimizes it).  Waves never synchronise with each other.  The partial sum
// never leaves registers, so there is no merge buffer: each gradient byte is
// read once and W and M are read and written once.
//
// Launch shape: one workgroup of kBlockThreads per compute unit, persistent.
// The step is HBM-bound and mixes many read streams with two in-place write
// streams (W and M); on MI355X such a mix reaches the highest bandwidth with
// few waves per CU.
//
// Memory access: a wave walks its full tiles, then its remainders.  A tile
// is 1024 elements of each of the N + 2 arrays: a lane takes 4 float4 of
// each (the wave's 64 lanes cover 4 contiguous 1 KB pieces).  Segments are
// cut on the host into full tiles and a remainder, so the tile loop is
// straight-line code.  The tile's loads go out piece by piece in a sliding
// window that continues into the wave's next tile (see the load window
// below); each piece is optimized and written back as soon as its last
// gradient is in.  Gradients are read once per step and loaded
// non-temporally.  W and M are read and written non-temporally, unless the
// job keeps them in the memory-side cache between steps (RES: cache-
// allocating policy for every W and M access of the launch).
//
// Arithmetic (no MFMA: the work is elementwise and HBM-bound): the sum is a
// left fold in ascending worker index, plain fp32 additions; then four
// fused multiply-adds:
//     d = wd*w + s;  m' = mu*m + d;  u = mu*m' + d (Nesterov) or m';
//     w' = -lr*u + w.
// The file is compiled with -ffp-contract=off and without fast-math, so the
// compiler neither fuses nor reorders beyond the explicit fma calls, and
// subnormals are kept.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <utility>

#include "kernels.hpp"

namespace phub {

typedef float f4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kWavesPerBlock = kBlockThreads / 64;

template <bool NEST>
__device__ __forceinline__ void optimize(float s, float& w, float& m, float nlr, float mu,
                                         float wd) {
    const float d = __builtin_fmaf(wd, w, s);
    const float m1 = __builtin_fmaf(mu, m, d);
    const float u = NEST ? __builtin_fmaf(mu, m1, d) : m1;
    w = __builtin_fmaf(nlr, u, w);
    m = m1;
}

template <bool NEST>
__device__ __forceinline__ void optimize4(const f4& s, f4& w, f4& m, float nlr, float mu,
                                          float wd) {
    const f4 vwd = wd, vmu = mu, vnlr = nlr;
    const f4 d = __builtin_elementwise_fma(vwd, w, s);
    const f4 m1 = __builtin_elementwise_fma(vmu, m, d);
    const f4 u = NEST ? __builtin_elementwise_fma(vmu, m1, d) : m1;
    w = __builtin_elementwise_fma(vnlr, u, w);
    m = m1;
}

// Gradient pointers come from a table in memory, so the compiler cannot tell
// they address global memory and would emit flat loads (which wait on both
// the vector and the LDS counters).  Casting to the global address space
// gives global_load_dwordx4 with the uniform base in SGPRs and a 32-bit
// per-lane offset.
#define PHUB_GLOBAL __attribute__((address_space(1)))

__device__ __forceinline__ f4 load_stream(const float* base, uint32_t byte_off) {
    const PHUB_GLOBAL char* b = (const PHUB_GLOBAL char*)base;
    return __builtin_nontemporal_load((const PHUB_GLOBAL f4*)(b + byte_off));
}

// W and M accesses.  The policy is a template argument resolved with
// `if constexpr`: written as a run-time choice between two loads of the same
// address, the compiler merges the two loads into one and drops the
// non-temporal hint.
template <bool RES>
__device__ __forceinline__ f4 load_wm(const float* base, uint32_t byte_off) {
    const PHUB_GLOBAL f4* a = (const PHUB_GLOBAL f4*)((const PHUB_GLOBAL char*)base + byte_off);
    if constexpr (RES)
        return *a;
    else
        return __builtin_nontemporal_load(a);
}

template <bool RES>
__device__ __forceinline__ void store_wm(float* base, uint32_t byte_off, const f4& v) {
    PHUB_GLOBAL f4* a = (PHUB_GLOBAL f4*)((PHUB_GLOBAL char*)base + byte_off);
    if constexpr (RES)
        *a = v;
    else
        __builtin_nontemporal_store(v, a);
}

// Updated weights written to a worker's model buffer (pushpull): written
// once and not read by the step, so non-temporal.
__device__ __forceinline__ void store_out(float* base, uint32_t byte_off, const f4& v) {
    __builtin_nontemporal_store(v, (PHUB_GLOBAL f4*)((PHUB_GLOBAL char*)base + byte_off));
}

__device__ __forceinline__ float load1(const float* base, int64_t i) {
    return ((const PHUB_GLOBAL float*)base)[i];
}

__device__ __forceinline__ void store1(float* base, int64_t i, float v) {
    ((PHUB_GLOBAL float*)base)[i] = v;
}

__device__ __forceinline__ uint32_t wave_index() {
    return __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6));
}

// The kernel arguments are __restrict__: the schedule and the pointer table
// are never written by the kernel and W/M never alias the gradients, which
// lets the compiler fetch descriptors and pointers with scalar loads.
#define PHUB_KERNEL_ARGS                                                                  \
    const DevTile* __restrict__ tiles, const int32_t* __restrict__ tile_begin,            \
        const DevRem* __restrict__ rems, const int32_t* __restrict__ rem_begin,           \
        const float* const* __restrict__ grads, float* const* __restrict__ outs,          \
        float* __restrict__ weights, float* __restrict__ moments, float lr, float mu,     \
        float wd, int num_workers

// Splits a tile's float4 index into a part folded into the base pointers
// (a multiple of 2^20 float4, 16 MB) and a low part that keeps the per-lane
// 32-bit byte offset far from overflow.
constexpr uint32_t kVecLowMask = (1u << 20) - 1;

// The streams of one full tile: uniform base pointers of the NW gradients,
// of W and of M, and the lane's byte offset of its first float4 from them.
// Lane l takes the float4s at tile float4 index l, l + 64, l + 128 and
// l + 192 (kVecPerLane pieces of 1 KB per wave), so every access is a
// uniform base in SGPRs + 32-bit lane offset + immediate.
template <int NW>
struct TileStreams {
    const float* g[NW];
    float* w;
    float* m;
    uint32_t off;
    uint32_t vhi;  // float4 index folded into the gradient (and output) bases
};

template <int NW>
__device__ __forceinline__ void tile_bases(TileStreams<NW>& s, const DevTile& d, float* weights,
                                           float* moments) {
    const uint32_t vlo = uint32_t(d.vec) & kVecLowMask;
    s.w = weights + d.arena_offset - size_t(vlo) * 4;
    s.m = moments + d.arena_offset - size_t(vlo) * 4;
    s.off = (vlo + (threadIdx.x & 63u)) * 16u;
}

// Streams of a tile from its key's pointer row in memory (scalar loads).
template <int NW>
__device__ __forceinline__ void tile_streams(TileStreams<NW>& s, const DevTile& d,
                                             const float* const* row, float* weights,
                                             float* moments) {
    const uint32_t vhi = uint32_t(d.vec) & ~kVecLowMask;
#pragma unroll
    for (int w = 0; w < NW; ++w) s.g[w] = row[w] + size_t(vhi) * 4;
    s.vhi = vhi;
    tile_bases<NW>(s, d, weights, moments);
}

// A key's pointer row fetched with one vector load, lane w holding worker
// w's pointer (lanes past the row repeat its last entry).  Held this way
// the next tile's row costs two VGPRs instead of 2 * NW SGPRs, which
// matters while the current tile's pointers still occupy SGPRs.
template <int NW>
__device__ __forceinline__ uint64_t load_row(const float* const* row) {
    const uint32_t l = threadIdx.x & 63u;
    const uint32_t i = l < uint32_t(NW) ? l : uint32_t(NW - 1);
    return ((const PHUB_GLOBAL uint64_t*)row)[i];
}

__device__ __forceinline__ const float* lane_pointer(uint64_t row, int w) {
    const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(row)), w));
    const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(row >> 32)), w));
    return reinterpret_cast<const float*>((uint64_t(hi) << 32) | lo);
}

// Streams of a tile from a pointer row held one per lane.
template <int NW>
__device__ __forceinline__ void tile_streams(TileStreams<NW>& s, const DevTile& d, uint64_t row,
                                             float* weights, float* moments) {
    const uint32_t vhi = uint32_t(d.vec) & ~kVecLowMask;
#pragma unroll
    for (int w = 0; w < NW; ++w) s.g[w] = lane_pointer(row, w) + size_t(vhi) * 4;
    s.vhi = vhi;
    tile_bases<NW>(s, d, weights, moments);
}

// Issue order of a tile's loads: for each of the kVecPerLane pieces, W, M,
// then the gradients in worker order; kTileLoads loads per tile.  A wave
// keeps a window of loads in flight beyond the one it waits for, and the
// window runs on into the wave's next tile.  Its depth follows the W/M
// policy (measured on MI355X):
//  - non-temporal W and M: a shallow window (kShallowAhead loads, a few KB
//    per wave) with the W and M reads and writes spread through the tile
//    moves more bytes than a deep one; deep windows flood the memory system
//    with open streams;
//  - W and M held in the memory-side cache: a whole tile ahead (every load
//    of the next tile in flight while this one is consumed), since only the
//    gradient streams then reach HBM.
#ifndef PHUB_LOADS_AHEAD
#define PHUB_LOADS_AHEAD 3
#endif
constexpr int kShallowAhead = PHUB_LOADS_AHEAD;

template <int NW>
constexpr int kTileLoads = kVecPerLane * (NW + 2);

template <int NW, bool RES>
constexpr int kAhead = RES ? kTileLoads<NW> - 1 : kShallowAhead;

template <int NW, bool RES>
constexpr int kRing = kAhead<NW, RES> + 1;

template <int NW, bool RES, int I>
__device__ __forceinline__ f4 tile_load(const TileStreams<NW>& s) {
    constexpr int k = I % (NW + 2);
    constexpr uint32_t o = uint32_t(I / (NW + 2)) * 1024u;
    if constexpr (k == 0)
        return load_wm<RES>(s.w, s.off + o);
    else if constexpr (k == 1)
        return load_wm<RES>(s.m, s.off + o);
    else
        return load_stream(s.g[k - 2], s.off + o);
}

template <int NW, bool RES>
struct TilePipe {
    static constexpr int R = kRing<NW, RES>;
    f4 ring[R];            // loads in flight, load j of a tile in slot j % R
    f4 acc[kVecPerLane];   // running gradient sums
    f4 wv[kVecPerLane];
    f4 mv[kVecPerLane];
};

// Step I of a tile: issue load I + kAhead (of this tile, or of the
// next one if there is one), then consume load I.  After the last gradient
// of a piece, that piece is optimized and written back.  Just before the
// first load of the next tile is issued, the next tile's streams are formed
// from its descriptor and pointer row, which were fetched at the start of
// this tile.
template <int NW, bool NEST, bool RES, bool PULL, int I>
__device__ __forceinline__ void tile_step(TilePipe<NW, RES>& p, const TileStreams<NW>& a,
                                          TileStreams<NW>& b, const DevTile& nd,
                                          uint64_t nrow, uint64_t prow, bool has_next,
                                          float* weights, float* moments, float nlr, float mu,
                                          float wd) {
    constexpr int L = kTileLoads<NW>;
    constexpr int R = kRing<NW, RES>;
    constexpr int J = I + kAhead<NW, RES>;
    if constexpr (J < L) {
        p.ring[J % R] = tile_load<NW, RES, J>(a);
    } else {
        if constexpr (J == L) tile_streams<NW>(b, nd, nrow, weights, moments);
        if (has_next) p.ring[J % R] = tile_load<NW, RES, J - L>(b);
    }
    __builtin_amdgcn_sched_barrier(0);
    const f4 v = p.ring[I % R];
    constexpr int k = I % (NW + 2);
    constexpr int u = I / (NW + 2);
    if constexpr (k == 0)
        p.wv[u] = v;
    else if constexpr (k == 1)
        p.mv[u] = v;
    else if constexpr (k == 2)
        p.acc[u] = v;
    else
        p.acc[u] = p.acc[u] + v;
    // Keep the addition (and so the wait for load I) at this step: the
    // compiler would otherwise sink the additions of the last piece past the
    // next-tile branch to their use, and issue that piece's loads as a burst.
    if constexpr (k >= 3) asm volatile("" : "+v"(p.acc[u]));
    if constexpr (k == NW + 1) {
        optimize4<NEST>(p.acc[u], p.wv[u], p.mv[u], nlr, mu, wd);
        store_wm<RES>(a.w, a.off + u * 1024u, p.wv[u]);
        store_wm<RES>(a.m, a.off + u * 1024u, p.mv[u]);
        if constexpr (PULL) {
            // the piece of w' into every worker's model buffer (pushpull)
#pragma unroll
            for (int w = 0; w < NW; ++w)
                store_out(const_cast<float*>(lane_pointer(prow, w)) + size_t(a.vhi) * 4,
                          a.off + u * 1024u, p.wv[u]);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
}

template <int NW, bool NEST, bool RES, bool PULL, int... I>
__device__ __forceinline__ void tile_steps(std::integer_sequence<int, I...>, TilePipe<NW, RES>& p,
                                           const TileStreams<NW>& a, TileStreams<NW>& b,
                                           const DevTile& nd, uint64_t nrow, uint64_t prow,
                                           bool has_next, float* weights, float* moments,
                                           float nlr, float mu, float wd) {
    (tile_step<NW, NEST, RES, PULL, I>(p, a, b, nd, nrow, prow, has_next, weights, moments, nlr,
                                       mu, wd),
     ...);
}

template <int NW, bool RES, int... I>
__device__ __forceinline__ void tile_prologue(std::integer_sequence<int, I...>, TilePipe<NW, RES>& p,
                                              const TileStreams<NW>& a) {
    ((p.ring[I % kRing<NW, RES>] = tile_load<NW, RES, I>(a)), ...);
}

// The rest of a segment: nvec < 256 float4 then a ragged end of rem < 4
// elements (one per lane).
template <int NW, bool NEST, bool RES, bool PULL>
__device__ __forceinline__ void partial(const float* const* g, float* wb, float* mb,
                                        float* const* out, uint32_t nvec, uint32_t rem,
                                        float nlr, float mu, float wd) {
    const uint32_t lane = threadIdx.x & 63u;
    for (uint32_t v = lane; v < nvec; v += 64u) {
        f4 a[NW];
#pragma unroll
        for (int w = 0; w < NW; ++w) a[w] = load_stream(g[w], v * 16u);
        f4 wv = load_wm<RES>(wb, v * 16u);
        f4 mv = load_wm<RES>(mb, v * 16u);
        f4 s = a[0];
#pragma unroll
        for (int w = 1; w < NW; ++w) s = s + a[w];
        optimize4<NEST>(s, wv, mv, nlr, mu, wd);
        store_wm<RES>(wb, v * 16u, wv);
        store_wm<RES>(mb, v * 16u, mv);
        if constexpr (PULL) {
#pragma unroll
            for (int w = 0; w < NW; ++w) store_out(out[w], v * 16u, wv);
        }
    }
    if (lane < rem) {
        const int64_t i = int64_t(nvec) * 4 + lane;
        float s = load1(g[0], i);
#pragma unroll
        for (int w = 1; w < NW; ++w) s = s + load1(g[w], i);
        float wv = load1(wb, i), mv = load1(mb, i);
        optimize<NEST>(s, wv, mv, nlr, mu, wd);
        store1(wb, i, wv);
        store1(mb, i, mv);
        if constexpr (PULL) {
#pragma unroll
            for (int w = 0; w < NW; ++w) store1(out[w], i, wv);
        }
    }
}

// NW > 0: exactly NW workers.  Each wave first streams its full tiles
// through the load window, then its remainders.  At the start of tile t the
// wave fetches the pointer row of tile t + 1 (one vector load), whose
// descriptor it fetched at the start of tile t - 1, and the descriptor of
// tile t + 2 (a scalar load); both have long arrived when the window
// reaches tile t + 1.
//
// One wave per SIMD (one workgroup of 4 waves per CU).
#define PHUB_ONE_WAVE_PER_SIMD __attribute__((amdgpu_waves_per_eu(1, 1)))

template <int NW, bool NEST, bool RES, bool PULL>
__global__ __launch_bounds__(kBlockThreads) PHUB_ONE_WAVE_PER_SIMD void fused_step_fixed(
    PHUB_KERNEL_ARGS) {
    static_assert(kTileLoads<NW> % kRing<NW, RES> == 0, "the load window must wrap with the tile");
    const uint32_t wave = wave_index();
    const float nlr = -lr;

    const int32_t tb = tile_begin[wave];
    const int32_t te = tile_begin[wave + 1];
    if (tb < te) {
        const int32_t last = te - 1;
        TilePipe<NW, RES> p;
        TileStreams<NW> a, b;
        uint64_t prow = 0;  // pushpull: model-buffer pointer row of the current tile
        {
            const DevTile first = tiles[tb];
            tile_streams<NW>(a, first, grads + int64_t(first.key) * NW, weights, moments);
            if constexpr (PULL) prow = load_row<NW>(outs + int64_t(first.key) * NW);
        }
        DevTile nd = tiles[tb + 1 <= last ? tb + 1 : last];
        tile_prologue<NW, RES>(std::make_integer_sequence<int, kAhead<NW, RES>>{}, p, a);
        for (int32_t t = tb;; ++t) {
            const bool has_next = t < last;
            const uint64_t nrow = load_row<NW>(grads + int64_t(nd.key) * NW);
            uint64_t nprow = 0;
            if constexpr (PULL) nprow = load_row<NW>(outs + int64_t(nd.key) * NW);
            const DevTile nd2 = tiles[t + 2 <= last ? t + 2 : last];
            tile_steps<NW, NEST, RES, PULL>(std::make_integer_sequence<int, kTileLoads<NW>>{}, p,
                                            a, b, nd, nrow, prow, has_next, weights, moments, nlr,
                                            mu, wd);
            if (!has_next) break;
            a = b;
            nd = nd2;
            prow = nprow;
        }
    }

    const int32_t rb = rem_begin[wave];
    const int32_t re = rem_begin[wave + 1];
    for (int32_t r = rb; r < re; ++r) {
        const DevRem rm = rems[r];
        const float* g[NW];
        float* out[NW];
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            g[w] = grads[int64_t(rm.key) * NW + w] + rm.offset;
            out[w] = PULL ? outs[int64_t(rm.key) * NW + w] + rm.offset : nullptr;
        }
        partial<NW, NEST, RES, PULL>(g, weights + rm.arena_offset, moments + rm.arena_offset, out,
                                     uint32_t(rm.count) >> 2, uint32_t(rm.count) & 3u, nlr, mu,
                                     wd);
    }
}

// Any N: workers taken in batches of kBatch, each batch's loads in flight
// together, the running sum carried across batches in worker order.
constexpr int kBatch = 8;

template <bool NEST, bool RES, bool PULL>
__device__ __forceinline__ void run_any(const float* const* kp, float* const* ko, int n,
                                        int64_t offset, float* wb, float* mb, uint32_t nvec,
                                        uint32_t rem, float nlr, float mu, float wd) {
    const uint32_t lane = threadIdx.x & 63u;
    for (uint32_t v = lane; v < nvec; v += 64u) {
        const uint32_t bo = v * 16u;
        f4 s = load_stream(kp[0] + offset, bo);
        for (int w0 = 1; w0 < n; w0 += kBatch) {
            f4 a[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j)
                if (w0 + j < n) a[j] = load_stream(kp[w0 + j] + offset, bo);
#pragma unroll
            for (int j = 0; j < kBatch; ++j)
                if (w0 + j < n) s = s + a[j];
        }
        f4 wv = load_wm<RES>(wb, bo);
        f4 mv = load_wm<RES>(mb, bo);
        optimize4<NEST>(s, wv, mv, nlr, mu, wd);
        store_wm<RES>(wb, bo, wv);
        store_wm<RES>(mb, bo, mv);
        if constexpr (PULL)
            for (int w = 0; w < n; ++w) store_out(ko[w] + offset, bo, wv);
    }
    if (lane < rem) {
        const int64_t i = int64_t(nvec) * 4 + lane;
        float s = load1(kp[0] + offset, i);
        for (int w = 1; w < n; ++w) s = s + load1(kp[w] + offset, i);
        float wv = load1(wb, i), mv = load1(mb, i);
        optimize<NEST>(s, wv, mv, nlr, mu, wd);
        store1(wb, i, wv);
        store1(mb, i, mv);
        if constexpr (PULL)
            for (int w = 0; w < n; ++w) store1(ko[w] + offset, i, wv);
    }
}

template <bool NEST, bool RES, bool PULL>
__global__ __launch_bounds__(kBlockThreads) void fused_step_any(PHUB_KERNEL_ARGS) {
    const uint32_t wave = wave_index();
    const int n = num_workers;
    const float nlr = -lr;
    const int32_t tb = tile_begin[wave];
    const int32_t te = tile_begin[wave + 1];
    for (int32_t t = tb; t < te; ++t) {
        const DevTile tl = tiles[t];
        run_any<NEST, RES, PULL>(grads + int64_t(tl.key) * n, PULL ? outs + int64_t(tl.key) * n : nullptr,
                                 n, int64_t(tl.vec) * 4, weights + tl.arena_offset,
                                 moments + tl.arena_offset, uint32_t(kTileElems / 4), 0u, nlr, mu,
                                 wd);
    }
    const int32_t rb = rem_begin[wave];
    const int32_t re = rem_begin[wave + 1];
    for (int32_t r = rb; r < re; ++r) {
        const DevRem rm = rems[r];
        run_any<NEST, RES, PULL>(grads + int64_t(rm.key) * n, PULL ? outs + int64_t(rm.key) * n : nullptr,
                                 n, rm.offset, weights + rm.arena_offset,
                                 moments + rm.arena_offset, uint32_t(rm.count) >> 2,
                                 uint32_t(rm.count) & 3u, nlr, mu, wd);
    }
}

// Ablation: the unfused ("wide") form of the step, kept to measure what
// fusion saves.  Pass 1 sums the N gradients of every element in worker
// order and writes the sum to a merge buffer laid out like W; pass 2 reads
// the merge buffer, W and M and runs the optimizer.  Same arithmetic, same
// schedule, (N + 6) * 4 bytes per element instead of (N + 4) * 4, and two
// launches.
__device__ __forceinline__ void aggregate_range(const float* const* kp, int n, int64_t offset,
                                                float* out, uint32_t nvec, uint32_t rem) {
    const uint32_t lane = threadIdx.x & 63u;
    for (uint32_t v = lane; v < nvec; v += 64u) {
        const uint32_t bo = v * 16u;
        f4 s = load_stream(kp[0] + offset, bo);
        for (int w0 = 1; w0 < n; w0 += kBatch) {
            f4 a[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j)
                if (w0 + j < n) a[j] = load_stream(kp[w0 + j] + offset, bo);
#pragma unroll
            for (int j = 0; j < kBatch; ++j)
                if (w0 + j < n) s = s + a[j];
        }
        store_out(out, bo, s);
    }
    if (lane < rem) {
        const int64_t i = int64_t(nvec) * 4 + lane;
        float s = load1(kp[0] + offset, i);
        for (int w = 1; w < n; ++w) s = s + load1(kp[w] + offset, i);
        store1(out, i, s);
    }
}

template <bool NEST, bool RES>
__device__ __forceinline__ void optimize_range(const float* sum, float* wb, float* mb,
                                               uint32_t nvec, uint32_t rem, float nlr, float mu,
                                               float wd) {
    const uint32_t lane = threadIdx.x & 63u;
    for (uint32_t v = lane; v < nvec; v += 64u) {
        const uint32_t bo = v * 16u;
        const f4 s = load_stream(sum, bo);
        f4 wv = load_wm<RES>(wb, bo);
        f4 mv = load_wm<RES>(mb, bo);
        optimize4<NEST>(s, wv, mv, nlr, mu, wd);
        store_wm<RES>(wb, bo, wv);
        store_wm<RES>(mb, bo, mv);
    }
    if (lane < rem) {
        const int64_t i = int64_t(nvec) * 4 + lane;
        float wv = load1(wb, i), mv = load1(mb, i);
        optimize<NEST>(load1(sum, i), wv, mv, nlr, mu, wd);
        store1(wb, i, wv);
        store1(mb, i, mv);
    }
}

__global__ __launch_bounds__(kBlockThreads) void aggregate_only(PHUB_KERNEL_ARGS, float* merge) {
    const uint32_t wave = wave_index();
    const int n = num_workers;
    for (int32_t t = tile_begin[wave]; t < tile_begin[wave + 1]; ++t) {
        const DevTile tl = tiles[t];
        aggregate_range(grads + int64_t(tl.key) * n, n, int64_t(tl.vec) * 4,
                        merge + tl.arena_offset, uint32_t(kTileElems / 4), 0u);
    }
    for (int32_t r = rem_begin[wave]; r < rem_begin[wave + 1]; ++r) {
        const DevRem rm = rems[r];
        aggregate_range(grads + int64_t(rm.key) * n, n, rm.offset, merge + rm.arena_offset,
                        uint32_t(rm.count) >> 2, uint32_t(rm.count) & 3u);
    }
}

template <bool NEST, bool RES>
__global__ __launch_bounds__(kBlockThreads) void optimize_only(PHUB_KERNEL_ARGS, float* merge) {
    const uint32_t wave = wave_index();
    const float nlr = -lr;
    for (int32_t t = tile_begin[wave]; t < tile_begin[wave + 1]; ++t) {
        const DevTile tl = tiles[t];
        optimize_range<NEST, RES>(merge + tl.arena_offset, weights + tl.arena_offset,
                                  moments + tl.arena_offset, uint32_t(kTileElems / 4), 0u, nlr,
                                  mu, wd);
    }
    for (int32_t r = rem_begin[wave]; r < rem_begin[wave + 1]; ++r) {
        const DevRem rm = rems[r];
        optimize_range<NEST, RES>(merge + rm.arena_offset, weights + rm.arena_offset,
                                  moments + rm.arena_offset, uint32_t(rm.count) >> 2,
                                  uint32_t(rm.count) & 3u, nlr, mu, wd);
    }
}

#define PHUB_LAUNCH_ARGS                                                                    \
    p.tiles, p.tile_begin, p.rems, p.rem_begin, p.grads, p.outs, p.weights, p.moments, p.lr, \
        p.mu, p.wd, p.num_workers

template <bool NEST, bool RES, bool PULL>
hipError_t launch_any(const StepParams& p, int grid, hipStream_t stream) {
    hipLaunchKernelGGL((fused_step_any<NEST, RES, PULL>), dim3(grid), dim3(kBlockThreads), 0,
                       stream, PHUB_LAUNCH_ARGS);
    return hipGetLastError();
}

template <int NW, bool NEST, bool RES, bool PULL>
hipError_t launch_one(const StepParams& p, int grid, hipStream_t stream) {
    if constexpr (kTileLoads<NW> % kRing<NW, RES> == 0) {
        hipLaunchKernelGGL((fused_step_fixed<NW, NEST, RES, PULL>), dim3(grid),
                           dim3(kBlockThreads), 0, stream, PHUB_LAUNCH_ARGS);
        return hipGetLastError();
    } else {
        return launch_any<NEST, RES, PULL>(p, grid, stream);
    }
}

template <int NW, bool RES>
hipError_t launch_n(const StepParams& p, bool nesterov, int grid, hipStream_t stream) {
    const bool pull = p.outs != nullptr;
    if (nesterov)
        return pull ? launch_one<NW, true, RES, true>(p, grid, stream)
                    : launch_one<NW, true, RES, false>(p, grid, stream);
    return pull ? launch_one<NW, false, RES, true>(p, grid, stream)
                : launch_one<NW, false, RES, false>(p, grid, stream);
}

template <bool RES>
hipError_t launch_res(const StepParams& p, bool nesterov, int grid, hipStream_t stream) {
    switch (p.num_workers) {
        case 1: return launch_n<1, RES>(p, nesterov, grid, stream);
        case 2: return launch_n<2, RES>(p, nesterov, grid, stream);
        case 3: return launch_n<3, RES>(p, nesterov, grid, stream);
        case 4: return launch_n<4, RES>(p, nesterov, grid, stream);
        case 5: return launch_n<5, RES>(p, nesterov, grid, stream);
        case 6: return launch_n<6, RES>(p, nesterov, grid, stream);
        case 7: return launch_n<7, RES>(p, nesterov, grid, stream);
        case 8: return launch_n<8, RES>(p, nesterov, grid, stream);
        case 9: return launch_n<9, RES>(p, nesterov, grid, stream);
        case 10: return launch_n<10, RES>(p, nesterov, grid, stream);
        case 11: return launch_n<11, RES>(p, nesterov, grid, stream);
        case 12: return launch_n<12, RES>(p, nesterov, grid, stream);
        case 13: return launch_n<13, RES>(p, nesterov, grid, stream);
        case 14: return launch_n<14, RES>(p, nesterov, grid, stream);
        case 15: return launch_n<15, RES>(p, nesterov, grid, stream);
        case 16: return launch_n<16, RES>(p, nesterov, grid, stream);
        default: {
            const bool pull = p.outs != nullptr;
            if (nesterov)
                return pull ? launch_any<true, RES, true>(p, grid, stream)
                            : launch_any<true, RES, false>(p, grid, stream);
            return pull ? launch_any<false, RES, true>(p, grid, stream)
                        : launch_any<false, RES, false>(p, grid, stream);
        }
    }
}

template <bool RES>
hipError_t launch_unfused(const StepParams& p, bool nesterov, int grid, hipStream_t stream) {
    hipLaunchKernelGGL(aggregate_only, dim3(grid), dim3(kBlockThreads), 0, stream,
                       PHUB_LAUNCH_ARGS, p.merge);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    if (nesterov)
        hipLaunchKernelGGL((optimize_only<true, RES>), dim3(grid), dim3(kBlockThreads), 0, stream,
                           PHUB_LAUNCH_ARGS, p.merge);
    else
        hipLaunchKernelGGL((optimize_only<false, RES>), dim3(grid), dim3(kBlockThreads), 0, stream,
                           PHUB_LAUNCH_ARGS, p.merge);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_fused_step(const StepParams& p, bool nesterov, bool resident, int grid,
                             hipStream_t stream) {
    if (p.merge)
        return resident ? launch_unfused<true>(p, nesterov, grid, stream)
                        : launch_unfused<false>(p, nesterov, grid, stream);
    return resident ? launch_res<true>(p, nesterov, grid, stream)
                    : launch_res<false>(p, nesterov, grid, stream);
}

}  // namespace phub
