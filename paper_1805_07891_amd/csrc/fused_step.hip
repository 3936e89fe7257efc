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
// read once and each optimizer state array is read and written once.
//
// Optimizers are pluggable (section 3.2.2): momentum SGD (plain or
// Nesterov; state W, M), plain SGD (state W) and Adam (state W, M, V) are
// compile-time policies of the same kernel; the S state arrays stream
// beside the N gradients.
//
// Launch shape: one workgroup of kBlockThreads per compute unit, persistent.
// The step is HBM-bound and mixes many read streams with a few in-place
// write streams (the state); on MI355X such a mix reaches the highest
// bandwidth with few waves per CU.
//
// Memory access: a wave reads its head (its bins and the first descriptor
// of each, WaveHead), then walks its full tiles, then its remainders.  A
// tile is 1024 elements of each of the N + S arrays: a lane takes 4 float4
// of each (the wave's 64 lanes cover 4 contiguous 1 KB pieces).  Segments
// are cut on the host into full tiles and a remainder, so the tile loop is
// straight-line code.  The tile's loads go out piece by piece in a sliding
// window that continues into the wave's next tile (see the load window
// below); each piece is optimized as soon as its last gradient is in, and
// written back at once, or, from enough gradient streams per state stream,
// in bursts of several tiles through LDS, timed by a chip-wide clock so
// that all waves write together (the burst write-back below).  Gradients
// are read once per step and loaded non-temporally.  A wave has two bins:
// the part of the job whose state is read and written non-temporally like
// the gradients, and the part whose state stays in the memory-side cache
// between steps (cache-allocating loads and stores).  Either may be empty.
//
// Arithmetic (no MFMA: the work is elementwise and HBM-bound): the sum is a
// left fold in ascending worker index, plain fp32 additions; then the
// optimizer, e.g. for momentum four fused multiply-adds:
//     d = wd*w + s;  m' = mu*m + d;  u = mu*m' + d (Nesterov) or m';
//     w' = -lr*u + w.
// The file is compiled with -ffp-contract=off and without fast-math, so the
// compiler neither fuses nor reorders beyond the explicit fma calls, and
// subnormals are kept; Adam's square root and division are correctly
// rounded (the division by the compiler's IEEE sequence, the square root
// by sqrt_rn below).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>
#include <utility>

#include "kernels.hpp"

namespace phub {

typedef float f4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kWavesPerBlock = kBlockThreads / 64;

// ------------------------------------------------------------- optimizers

// State arrays of each optimizer, W first.
template <int OPT>
constexpr int kStates = OPT == kOptSgd ? 1 : (OPT == kOptAdam ? 3 : 2);

// Correctly rounded single-precision square root.  The hardware square
// root (with the compiler's denormal scaling) is within one ulp, so the
// correctly rounded root is y, or its neighbour below or above.  The
// midpoints between neighbours have at most 25 significant bits, so their
// squares are exact in double; comparing x with them decides exactly
// (a float's square root is never a midpoint, so there are no ties).
__device__ __forceinline__ float sqrt_rn(float x) {
    const float y = __builtin_sqrtf(x);
    if (!(x > 0.0f) || !(y < __builtin_huge_valf())) return y;  // 0, < 0, NaN, inf
    const uint32_t yb = __builtin_bit_cast(uint32_t, y);
    const float down = __builtin_bit_cast(float, yb - 1u);
    const float up = __builtin_bit_cast(float, yb + 1u);
    const double lo = 0.5 * (double(down) + double(y));
    const double hi = 0.5 * (double(y) + double(up));
    const double xd = double(x);
    if (xd < lo * lo) return down;
    if (xd > hi * hi) return up;
    return y;
}

// One element: st[0] = w, st[1] = m, st[2] = v, updated in place.
template <int OPT>
__device__ __forceinline__ void update(float s, float* st, OptArgs o) {
    if constexpr (OPT == kOptSgd) {
        const float d = __builtin_fmaf(o.wd, st[0], s);
        st[0] = __builtin_fmaf(o.nlr, d, st[0]);
    } else if constexpr (OPT == kOptAdam) {
        const float d = __builtin_fmaf(o.wd, st[0], s);
        const float m = __builtin_fmaf(o.b1, st[1], o.c1 * d);
        const float dd = d * d;
        const float v = __builtin_fmaf(o.b2, st[2], o.c2 * dd);
        const float den = sqrt_rn(v * o.k2) + o.eps;
        const float q = __fdiv_rn(o.k1 * m, den);
        st[0] = st[0] - q;
        st[1] = m;
        st[2] = v;
    } else {
        constexpr bool NEST = OPT == kOptNesterov;
        const float d = __builtin_fmaf(o.wd, st[0], s);
        const float m1 = __builtin_fmaf(o.mu, st[1], d);
        const float u = NEST ? __builtin_fmaf(o.mu, m1, d) : m1;
        st[0] = __builtin_fmaf(o.nlr, u, st[0]);
        st[1] = m1;
    }
}

// Four elements at once (a float4 of each array).
template <int OPT>
__device__ __forceinline__ void update4(const f4& s, f4* st, OptArgs o) {
    if constexpr (OPT == kOptAdam) {
        // the square root and division per component, correctly rounded
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            float e[3] = {st[0][c], st[1][c], st[2][c]};
            update<OPT>(s[c], e, o);
            st[0][c] = e[0];
            st[1][c] = e[1];
            st[2][c] = e[2];
        }
    } else if constexpr (OPT == kOptSgd) {
        const f4 vwd = o.wd, vnlr = o.nlr;
        const f4 d = __builtin_elementwise_fma(vwd, st[0], s);
        st[0] = __builtin_elementwise_fma(vnlr, d, st[0]);
    } else {
        constexpr bool NEST = OPT == kOptNesterov;
        const f4 vwd = o.wd, vmu = o.mu, vnlr = o.nlr;
        const f4 d = __builtin_elementwise_fma(vwd, st[0], s);
        const f4 m1 = __builtin_elementwise_fma(vmu, st[1], d);
        const f4 u = NEST ? __builtin_elementwise_fma(vmu, m1, d) : m1;
        st[0] = __builtin_elementwise_fma(vnlr, u, st[0]);
        st[1] = m1;
    }
}

// --------------------------------------------------------- memory access

// Gradient pointers come from a table in memory, so the compiler cannot tell
// they address global memory and would emit flat loads (which wait on both
// the vector and the LDS counters).  Casting to the global address space
// gives global_load_dwordx4 with the uniform base in SGPRs and a 32-bit
// per-lane offset.
#define PHUB_GLOBAL __attribute__((address_space(1)))
#define PHUB_LDS __attribute__((address_space(3)))

// Gradient loads (and the unfused variant's sum buffer): non-temporal, as
// each gradient byte is read once.  A build with PHUB_GRADIENT_LOADS_CACHED
// set loads them cache-allocating instead: the ablation of caching the
// gradients beside the model (the paper's Table 4).
#ifndef PHUB_GRADIENT_LOADS_CACHED
#define PHUB_GRADIENT_LOADS_CACHED 0
#endif
__device__ __forceinline__ f4 load_stream(const float* base, uint32_t byte_off) {
    const PHUB_GLOBAL char* b = (const PHUB_GLOBAL char*)base;
#if PHUB_GRADIENT_LOADS_CACHED
    return *(const PHUB_GLOBAL f4*)(b + byte_off);
#else
    return __builtin_nontemporal_load((const PHUB_GLOBAL f4*)(b + byte_off));
#endif
}

// State accesses.  The policy is a template argument resolved with
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

// A float4 of stashed state written back in a write phase: a buffer store
// (the compiler tracks it like any other store; the base in SGPRs, a 32-bit
// lane offset) with the cache policy bits of gfx950 given directly:
// non-temporal (2) with the sc1 bit (16).  Measured in the write phases
// against the non-temporal global store: +0.1 to +0.9 points on 8- and
// 16-worker jobs and +0.5 on four tenants; plain (cache-allocating) stores
// were 13-15 points below.  The descriptor covers 2 GB from the base, far
// beyond a tile's offsets (below 17 MB).
constexpr int kBufferWord3 = 0x00020000;  // buffer descriptor's format word on gfx9
constexpr int kWriteBackCachePolicy = 2 | 16;
__device__ __forceinline__ void store_wb(float* base, uint32_t byte_off, const f4& v) {
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc(base, 0, 0x7fffffff, kBufferWord3);
    __builtin_amdgcn_raw_buffer_store_b128(v, r, int(byte_off), 0, kWriteBackCachePolicy);
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
// are never written by the kernel and the state never aliases the
// gradients, which lets the compiler fetch descriptors and pointers with
// scalar loads.
#define PHUB_KERNEL_ARGS                                                                  \
    const DevTile* __restrict__ tiles, const int32_t* __restrict__ tile_begin,            \
        const DevRem* __restrict__ rems, const int32_t* __restrict__ rem_begin,           \
        const WaveHead* __restrict__ heads,                                               \
        const float* const* __restrict__ grads, float* const* __restrict__ outs,          \
        float* __restrict__ weights, float* __restrict__ moments,                         \
        float* __restrict__ second, OptArgs o, int num_workers,                           \
        const DevTile* __restrict__ pool, int32_t pool_count,                             \
        unsigned long long* __restrict__ pool_counters, uint64_t pool_launch

// Splits a tile's float4 index into a part folded into the base pointers
// (a multiple of 2^20 float4, 16 MB) and a low part that keeps the per-lane
// 32-bit byte offset far from overflow.
constexpr uint32_t kVecLowMask = (1u << 20) - 1;

// ------------------------------------------------------------ full tiles

// The streams of one full tile: uniform base pointers of the NW gradients
// and of the S state arrays, and the lane's byte offset of its first float4
// from them.  Lane l takes the float4s at tile float4 index l, l + 64,
// l + 128 and l + 192 (kVecPerLane pieces of 1 KB per wave), so every
// access is a uniform base in SGPRs + 32-bit lane offset + immediate.
template <int NW, int S>
struct TileStreams {
    const float* g[NW];
    float* st[S];
    uint32_t off;
    uint32_t vhi;  // float4 index folded into the gradient (and output) bases
};

template <int NW, int S>
__device__ __forceinline__ void tile_bases(TileStreams<NW, S>& s, const DevTile& d,
                                           float* const* state) {
    const uint32_t vlo = d.vec & kVecLowMask;
#pragma unroll
    for (int i = 0; i < S; ++i) s.st[i] = state[i] + d.arena_offset - size_t(vlo) * 4;
    s.off = (vlo + (threadIdx.x & 63u)) * 16u;
}

// Streams of a tile from its key's pointer row in memory (scalar loads).
template <int NW, int S>
__device__ __forceinline__ void tile_streams(TileStreams<NW, S>& s, const DevTile& d,
                                             const float* const* row, float* const* state) {
    const uint32_t vhi = d.vec & ~kVecLowMask;
#pragma unroll
    for (int w = 0; w < NW; ++w) s.g[w] = row[w] + size_t(vhi) * 4;
    s.vhi = vhi;
    tile_bases<NW, S>(s, d, state);
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
template <int NW, int S>
__device__ __forceinline__ void tile_streams(TileStreams<NW, S>& s, const DevTile& d,
                                             uint64_t row, float* const* state) {
    const uint32_t vhi = d.vec & ~kVecLowMask;
#pragma unroll
    for (int w = 0; w < NW; ++w) s.g[w] = lane_pointer(row, w) + size_t(vhi) * 4;
    s.vhi = vhi;
    tile_bases<NW, S>(s, d, state);
}

// Issue order of a tile's loads: for each of the kVecPerLane pieces, the S
// state arrays (W first), then the gradients in worker order; kTileLoads
// loads per tile.  A wave keeps a window of loads in flight beyond the one
// it waits for, and the window runs on into the wave's next tile.  Load j
// of a tile sits in ring slot j mod R; where the ring R does not divide the
// tile's loads, consecutive tiles take turns (phases) so that every load
// keeps its slot.  The depth follows the state policy (measured on MI355X):
//  - non-temporal state: a ring of 6 loads (five ahead), or 5 or 8 for a
//    few worker counts and optimizers (kRingTable), from a sweep of rings 4
//    to 8 for every worker count and optimizer (fraction of peak with
//    nothing cached, ResNet-269-shaped keys).  Six beats four everywhere
//    (momentum with 16 workers 0.765 against 0.717, plain SGD with 16 0.834
//    against 0.736, Adam with 10 0.731 against 0.673); eight is better for
//    Adam with 3-7 workers (3 workers: 0.752 against 0.684) and plain SGD
//    with 2, 3 or 6; five for momentum with 3 or 8 workers (8: 0.749
//    against 0.737).  Deeper windows flood the memory system with open
//    streams, and loads and stores share one in-order counter, so a load
//    issued after a state store is consumed only once that store has
//    completed;
//  - state held in the memory-side cache: a whole tile ahead (every load of
//    the next tile in flight while this one is consumed), since only the
//    gradient streams then reach HBM.
template <int NW, int S>
constexpr int kTileLoads = kVecPerLane * (NW + S);

// Ring of the non-temporal window, [S - 1][N - 1] (S = 1 plain SGD, 2
// momentum, 3 Adam): 6 unless another ring measured more than half a point
// better (momentum with 8 workers took 5 before its state was written back
// in the write phases below; with them, 6 is 5 points faster on a
// 143.7 M-parameter job).  A ring of 5 must divide the tile's 4 (N + S)
// loads; 6 and 8 take at most three and two phases.
constexpr int kRingTable[3][kMaxFixedWorkers] = {
    {6, 8, 8, 6, 6, 8, 6, 6, 6, 6, 6, 6, 6, 6, 6, 6},
    {6, 6, 5, 6, 6, 6, 6, 6, 6, 6, 6, 6, 6, 6, 6, 6},
    {6, 6, 8, 8, 8, 8, 8, 6, 6, 6, 6, 6, 6, 6, 6, 6},
};

#ifdef PHUB_LOADS_AHEAD
template <int NW, int S>
constexpr int kShallowAhead = PHUB_LOADS_AHEAD;  // a fixed depth, for sweeps
#else
template <int NW, int S>
constexpr int kShallowAhead =
    (NW >= 1 && NW <= kMaxFixedWorkers && S >= 1 && S <= 3 ? kRingTable[S - 1][NW - 1] : 6) - 1;
#endif

constexpr int gcd_int(int a, int b) { return b == 0 ? a : gcd_int(b, a % b); }

// Ring of the resident bin: a whole tile while that fits the registers
// (up to 80 loads, 320 VGPRs); beyond, the largest of 32, 24, 20, 16 loads
// that needs at most three phases (rings of 12 or 24 measured equal to the
// whole tile at 8-16 workers).
constexpr int resident_ring(int loads) {
    if (loads <= 80) return loads;
    for (int r : {32, 24, 20, 16})
        if (r / gcd_int(loads, r) <= 3) return r;
    return 4;
}

template <int NW, int S, bool RES>
constexpr int kAhead = RES ? resident_ring(kTileLoads<NW, S>) - 1 : kShallowAhead<NW, S>;

template <int NW, int S, bool RES>
constexpr int kRing = kAhead<NW, S, RES> + 1;

// Where the ring does not divide the tile's loads, a wave's tiles take
// kPhases turns: load j of a tile in phase h sits in ring slot
// (h L + j) mod R, and after kPhases tiles the slots line up again.
template <int NW, int S, bool RES>
constexpr int kPhases = kRing<NW, S, RES> / gcd_int(kTileLoads<NW, S>, kRing<NW, S, RES>);

// Burst write-back of the streamed bin's state, in chip-wide write phases.
// A few write streams spread evenly through many read streams cost HBM much
// more than the same bytes written in runs.  So, from enough workers per
// state array (burst_write_back), the streamed bin does not write a piece's
// new state as soon as it is computed: the state goes to a stash in LDS,
// and the wave writes the stash back in one run of stores when it finishes
// a piece inside the write window (then the tiles before the current one;
// at a tile's end, the tile too), or when the stash is full (kStashTiles
// tiles), or after its last tile.  The write window is the first part of a
// period of the device's constant-rate wall clock, which every wave of
// every launch on the chip reads alike: the waves write at the same time
// and read at the same time, so HBM sees long runs of writes and long runs
// of reads instead of a steady mix.  The period follows the tile's bytes
// and the stash's size (kWritePeriodNsPerStreamTile: about as many tiles of
// a wave as the stash holds besides the one in progress) and the window is
// about one tile long (kWriteWindowNs).  Measured on MI355X with
// nothing cached, fraction of peak (8 workers, momentum), piece by piece ->
// burst write-back: 143.7 M parameters 0.72 -> 0.815, 61.1 M 0.78 -> 0.816,
// 102 M with 16 workers 0.77 -> 0.84; the same stash flushed only when
// full, 0.73 on the first; flushed on each compute unit's own cycle counter
// (not aligned across the chip), 0.71; looked for only at the end of a tile
// (with the best period and window for that), 1-2.6 points below.
// Each lane reads back only the values it wrote, so the stash needs no
// barrier, and results do not depend on when it is written back.  The
// stash takes the compute unit's 160 KB of LDS (at most 40 KB per wave).
constexpr int kLdsBytes = 160 * 1024;
static_assert(kStashBytesPerWave * kWavesPerBlock <= kLdsBytes, "the stash fits the LDS");

template <int S>
constexpr int kStashTiles = stash_tiles(S);
static_assert(kVecPerLane * 1024 == 4 * 1024, "a tile is 4 KB per array and wave");

// float4 per tile and per wave in the stash (lane l holds entry l of every 64)
template <int S>
constexpr int kStashTileVecs = S * kVecPerLane * 64;

template <int NW, int S, bool RES, bool PULL>
constexpr bool kStash =
    !RES && !PULL && burst_write_back(NW, S) && kStashTiles<S> >= 2;


template <int NW, int S, bool RES, int I>
__device__ __forceinline__ f4 tile_load(const TileStreams<NW, S>& s) {
    constexpr int k = I % (NW + S);
    constexpr uint32_t o = uint32_t(I / (NW + S)) * 1024u;
    if constexpr (k < S)
        return load_wm<RES>(s.st[k], s.off + o);
    else
        return load_stream(s.g[k - S], s.off + o);
}

template <int NW, int S, bool RES>
struct TilePipe {
    static constexpr int R = kRing<NW, S, RES>;
    f4 ring[R];               // loads in flight, load j of a tile in slot j % R
    f4 acc[kVecPerLane];      // running gradient sums
    f4 sv[S][kVecPerLane];    // the state of each piece
};

// Whether the device's wall clock is inside a write window of the burst
// write-back (the same answer for every lane: the clock is a scalar).  The
// low 32 bits of the clock wrap every 43 s at 100 MHz; the wrap shifts the
// phase of the periods once, which costs nothing but a slightly misplaced
// window.
__device__ __forceinline__ bool in_write_window(uint32_t period, uint32_t window) {
    const uint32_t now = uint32_t(wall_clock64());
    return now % period < window;
}

// Writes back the stashed state of the wave's tiles [t0, t1] (streamed
// bin), tile by tile, each tile's S arrays piece by piece; tile t's state
// is in stash slot t mod kStashTiles.  `stash` points at the lane's entry
// of the wave's first stash slot.
template <int NW, int S>
__device__ __forceinline__ void write_stash(const DevTile* __restrict__ tiles, int32_t t0,
                                            int32_t t1, const PHUB_LDS f4* stash,
                                            float* const* state) {
    for (int32_t t = t0; t <= t1; ++t) {
        TileStreams<NW, S> s;
        tile_bases<NW, S>(s, tiles[t], state);
        const PHUB_LDS f4* ts = stash + (t % kStashTiles<S>) * kStashTileVecs<S>;
#pragma unroll
        for (int i = 0; i < S; ++i) {
#pragma unroll
            for (int u = 0; u < kVecPerLane; ++u) {
                const f4 v = ts[(i * kVecPerLane + u) * 64];
                store_wb(s.st[i], s.off + u * 1024u, v);
            }
        }
    }
}

// Where a wave's walk over a list of tiles stands in the burst write-back:
// tile t's state goes to stash slot t mod kStashTiles, and the tiles
// [t_stash, t) before the current one t wait in the stash.
struct TileCursor {
    const DevTile* tiles;
    PHUB_LDS f4* stash;  // the lane's entry of the wave's first slot
    int32_t t;
    int32_t t_stash;
    __device__ bool waiting() const { return t != t_stash; }
    // write back the tiles before the current one
    template <int NW, int S>
    __device__ void write_back_before(float* const* state) {
        write_stash<NW, S>(tiles, t_stash, t - 1, stash, state);
        t_stash = t;
    }
};

// Step I of a tile: issue load I + kAhead (of this tile, or of the next one
// if there is one), then consume load I.  After the last gradient of a
// piece, that piece is optimized and written back.  Just before the first
// load of the next tile is issued, the next tile's streams are formed from
// its descriptor and pointer row, which were fetched at the start of this
// tile.
template <int NW, int OPT, bool RES, bool PULL, int PH, int I, typename Cursor>
__device__ __forceinline__ void tile_step(TilePipe<NW, kStates<OPT>, RES>& p,
                                          const TileStreams<NW, kStates<OPT>>& a,
                                          TileStreams<NW, kStates<OPT>>& b, const DevTile& nd,
                                          uint64_t nrow, uint64_t prow, bool has_next,
                                          float* const* state, OptArgs o,
                                          PHUB_LDS f4* tile_stash, Cursor* cur) {
    constexpr int S = kStates<OPT>;
    constexpr int L = kTileLoads<NW, S>;
    constexpr int R = kRing<NW, S, RES>;
    constexpr int J = I + kAhead<NW, S, RES>;
    constexpr int base = (PH * L) % R;  // slot of this tile's first load
    if constexpr (J < L) {
        p.ring[(base + J) % R] = tile_load<NW, S, RES, J>(a);
    } else {
        if constexpr (J == L) tile_streams<NW, S>(b, nd, nrow, state);
        if (has_next) p.ring[(base + J) % R] = tile_load<NW, S, RES, J - L>(b);
    }
    __builtin_amdgcn_sched_barrier(0);
    const f4 v = p.ring[(base + I) % R];
    constexpr int k = I % (NW + S);
    constexpr int u = I / (NW + S);
    if constexpr (k < S)
        p.sv[k][u] = v;
    else if constexpr (k == S)
        p.acc[u] = v;
    else
        p.acc[u] = p.acc[u] + v;
    // Keep the addition (and so the wait for load I) at this step: the
    // compiler would otherwise sink the additions of the last piece past the
    // next-tile branch to their use, and issue that piece's loads as a burst.
    if constexpr (k > S) asm volatile("" : "+v"(p.acc[u]));
    if constexpr (k == NW + S - 1) {
        f4 st[S];
#pragma unroll
        for (int i = 0; i < S; ++i) st[i] = p.sv[i][u];
        update4<OPT>(p.acc[u], st, o);
        if constexpr (kStash<NW, S, RES, PULL>) {
#pragma unroll
            for (int i = 0; i < S; ++i) tile_stash[(i * kVecPerLane + u) * 64] = st[i];
            // the window opened during this tile: write back the tiles
            // before it now (this tile's pieces stay in its slot), so that
            // the waves' write-backs start within a piece of the window's
            // opening instead of within a tile
            if constexpr (u + 1 < kVecPerLane) {
                if (cur->waiting() && in_write_window(o.wb_period, o.wb_window))
                    cur->template write_back_before<NW, S>(state);
            }
        } else {
#pragma unroll
            for (int i = 0; i < S; ++i) store_wm<RES>(a.st[i], a.off + u * 1024u, st[i]);
        }
        if constexpr (PULL) {
            // the piece of w' into every worker's model buffer (pushpull)
#pragma unroll
            for (int w = 0; w < NW; ++w)
                store_out(const_cast<float*>(lane_pointer(prow, w)) + size_t(a.vhi) * 4,
                          a.off + u * 1024u, st[0]);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
}

template <int NW, int OPT, bool RES, bool PULL, int PH, typename Cursor, int... I>
__device__ __forceinline__ void tile_steps(std::integer_sequence<int, I...>,
                                           TilePipe<NW, kStates<OPT>, RES>& p,
                                           const TileStreams<NW, kStates<OPT>>& a,
                                           TileStreams<NW, kStates<OPT>>& b, const DevTile& nd,
                                           uint64_t nrow, uint64_t prow, bool has_next,
                                           float* const* state, OptArgs o,
                                           PHUB_LDS f4* tile_stash, Cursor* cur) {
    (tile_step<NW, OPT, RES, PULL, PH, I>(p, a, b, nd, nrow, prow, has_next, state, o, tile_stash,
                                          cur),
     ...);
}

template <int NW, int S, bool RES, int... I>
__device__ __forceinline__ void tile_prologue(std::integer_sequence<int, I...>,
                                              TilePipe<NW, S, RES>& p,
                                              const TileStreams<NW, S>& a) {
    ((p.ring[I % kRing<NW, S, RES>] = tile_load<NW, S, RES, I>(a)), ...);
}

// ------------------------------------------------------ the tile pool

// Dynamic schedule (work stealing): the streamed bin's full tiles of a
// launch form one pool, in address order, and every wave takes its next
// tile of the pool from a counter shared with the other waves of its XCD
// (PoolCounters), each counter serving every C-th tile, so that all waves
// still work on neighbouring tiles.  A wave that starts late (its compute
// unit was still held by another tenant's launch) simply takes fewer
// tiles.  A counter is never reset: the host passes each launch the
// counter's value at its start (the base), and every wave stops after
// exactly one take past its tiles.
//
// A take is a vector atomic from lane 0 whose value is read one tile later
// (issue_take, then resolve_take), so that the wait for it falls behind
// loads the wave has issued meanwhile, not in front of them.
__device__ __forceinline__ uint64_t issue_take(unsigned long long* counter) {
    uint64_t v = 0;
    if ((threadIdx.x & 63u) == 0) v = atomicAdd(counter, 1ull);
    return v;
}

// Pool index of a take, or -1 past the pool (or before it: never, unless
// the base is wrong, in which case nothing is read).
__device__ __forceinline__ int32_t resolve_take(uint64_t v, uint64_t base, int32_t count) {
    const uint32_t lo = uint32_t(__builtin_amdgcn_readfirstlane(int(uint32_t(v))));
    const uint32_t hi = uint32_t(__builtin_amdgcn_readfirstlane(int(uint32_t(v >> 32))));
    const int64_t i = int64_t(((uint64_t(hi) << 32) | lo) - base);
    return i >= 0 && i < int64_t(count) ? int32_t(i) : -1;
}

// Writes back the `count` stashed tiles of a pool walk whose oldest sits in
// stash slot `first`, the next ones in the slots after it (mod SLOTS);
// slot k holds pool tile pool[idx[k] * stride].
template <int NW, int S, int SLOTS>
__device__ __forceinline__ void write_stash_slots(const DevTile* __restrict__ pool, int stride,
                                                  const int32_t (&idx)[SLOTS], int first,
                                                  int count, const PHUB_LDS f4* stash,
                                                  float* const* state) {
#pragma unroll
    for (int k = 0; k < SLOTS; ++k) {
        if ((k - first + SLOTS) % SLOTS < count) {
            TileStreams<NW, S> s;
            tile_bases<NW, S>(s, pool[int64_t(idx[k]) * stride], state);
            const PHUB_LDS f4* ts = stash + k * kStashTileVecs<S>;
#pragma unroll
            for (int i = 0; i < S; ++i) {
#pragma unroll
                for (int u = 0; u < kVecPerLane; ++u) {
                    const f4 v = ts[(i * kVecPerLane + u) * 64];
                    store_wb(s.st[i], s.off + u * 1024u, v);
                }
            }
        }
    }
}

// Where a wave's pool walk stands in the burst write-back: its n-th tile
// (counted from 0) goes to stash slot n mod SLOTS, and the tiles
// [first, n) before the current one wait in the stash.
template <int SLOTS>
struct PoolCursor {
    const DevTile* pool;
    int stride;
    PHUB_LDS f4* stash;
    int32_t idx[SLOTS];  // the pool tile held by each slot
    int32_t n;
    int32_t first;
    __device__ bool waiting() const { return n != first; }
    // write back the tiles [first, end)
    template <int NW, int S>
    __device__ void write_back_to(int32_t end, float* const* state) {
        write_stash_slots<NW, S, SLOTS>(pool, stride, idx, first % SLOTS, end - first, stash,
                                        state);
        first = end;
    }
    template <int NW, int S>
    __device__ void write_back_before(float* const* state) {
        write_back_to<NW, S>(n, state);
    }
};

// ------------------------------------------------------------ remainders

// A remainder of a segment: nvec float4 and then rem (< 4) single elements
// per array.  Every lane's loads of a group of up to kVecPerLane float4 per
// array (as many as keep at most 64 loads in flight) and of its single
// element are issued before the first is consumed: a remainder shorter
// than a tile (the schedule's) costs one trip to memory, not one per
// float4 of a lane.
template <int NW, int OPT, bool RES, bool PULL>
__device__ __forceinline__ void partial(const float* const* g, float* const* stb,
                                        float* const* out, uint32_t nvec, uint32_t rem,
                                        OptArgs o) {
    constexpr int S = kStates<OPT>;
    constexpr int kGroup = (NW + S) * kVecPerLane <= 64 ? kVecPerLane
                           : 64 / (NW + S) > 0 ? 64 / (NW + S) : 1;
    const uint32_t lane = threadIdx.x & 63u;
    // the single elements of the last < 4, loaded with the first group
    const int64_t ti = int64_t(nvec) * 4 + lane;
    const bool tail = lane < rem;
    float ta[NW], tst[S];
    bool tail_loaded = false;
    for (uint32_t v0 = 0; v0 < nvec || !tail_loaded; v0 += 64u * kGroup) {
        f4 a[kGroup][NW];
        f4 st[kGroup][S];
#pragma unroll
        for (int j = 0; j < kGroup; ++j) {
            const uint32_t v = v0 + 64u * j + lane;
            if (v < nvec) {
#pragma unroll
                for (int w = 0; w < NW; ++w) a[j][w] = load_stream(g[w], v * 16u);
#pragma unroll
                for (int i = 0; i < S; ++i) st[j][i] = load_wm<RES>(stb[i], v * 16u);
            }
        }
        if (!tail_loaded && tail) {
#pragma unroll
            for (int w = 0; w < NW; ++w) ta[w] = load1(g[w], ti);
#pragma unroll
            for (int k = 0; k < S; ++k) tst[k] = load1(stb[k], ti);
        }
        tail_loaded = true;
#pragma unroll
        for (int j = 0; j < kGroup; ++j) {
            const uint32_t v = v0 + 64u * j + lane;
            if (v < nvec) {
                f4 s = a[j][0];
#pragma unroll
                for (int w = 1; w < NW; ++w) s = s + a[j][w];
                update4<OPT>(s, st[j], o);
#pragma unroll
                for (int i = 0; i < S; ++i) store_wm<RES>(stb[i], v * 16u, st[j][i]);
                if constexpr (PULL) {
#pragma unroll
                    for (int w = 0; w < NW; ++w) store_out(out[w], v * 16u, st[j][0]);
                }
            }
        }
    }
    if (tail) {
        float s = ta[0];
#pragma unroll
        for (int w = 1; w < NW; ++w) s = s + ta[w];
        update<OPT>(s, tst, o);
#pragma unroll
        for (int k = 0; k < S; ++k) store1(stb[k], ti, tst[k]);
        if constexpr (PULL) {
#pragma unroll
            for (int w = 0; w < NW; ++w) store1(out[w], ti, tst[0]);
        }
    }
}

// ---------------------------------------------------------------- kernels

// The full tiles [tb, te) of one bin, NW workers, state policy RES; `first`
// is tiles[tb], which the wave has from its head.  At
// the start of tile t the wave fetches the pointer row of tile t + 1 (one
// vector load), whose descriptor it fetched at the start of tile t - 1, and
// the descriptor of tile t + 2 (a scalar load); both have long arrived when
// the window reaches tile t + 1.
template <int NW, int OPT, bool RES, bool PULL>
__device__ __forceinline__ void walk_tiles(const DevTile* __restrict__ tiles, int32_t tb,
                                           int32_t te, const DevTile& first,
                                           const float* const* __restrict__ grads,
                                           float* const* __restrict__ outs, float* const* state,
                                           OptArgs o, PHUB_LDS f4* stash) {
    constexpr int S = kStates<OPT>;
    constexpr int NPH = kPhases<NW, S, RES>;
    static_assert(NPH >= 1 && NPH <= 3, "the tile loop below unrolls at most three phases");
    if (tb >= te) return;
    const int32_t last = te - 1;
    TilePipe<NW, S, RES> p;
    TileStreams<NW, S> a, b;
    uint64_t prow = 0;  // pushpull: model-buffer pointer row of the current tile
    tile_streams<NW, S>(a, first, grads + int64_t(first.key) * NW, state);
    if constexpr (PULL) prow = load_row<NW>(outs + int64_t(first.key) * NW);
    DevTile nd = tiles[tb + 1 <= last ? tb + 1 : last];
    tile_prologue<NW, S, RES>(std::make_integer_sequence<int, kAhead<NW, S, RES>>{}, p, a);
    TileCursor c{tiles, stash, tb, tb};  // c.t: the current tile
    int32_t& t = c.t;
    // Tile t in ring phase PH; false after the bin's last tile.
    auto one_tile = [&](auto phase) -> bool {
        constexpr int PH = decltype(phase)::value;
        const bool has_next = t < last;
        const uint64_t nrow = load_row<NW>(grads + int64_t(nd.key) * NW);
        uint64_t nprow = 0;
        if constexpr (PULL) nprow = load_row<NW>(outs + int64_t(nd.key) * NW);
        const DevTile nd2 = tiles[t + 2 <= last ? t + 2 : last];
        PHUB_LDS f4* tile_stash = nullptr;  // this tile's slot of the stash
        if constexpr (kStash<NW, S, RES, PULL>)
            tile_stash = stash + (t % kStashTiles<S>) * kStashTileVecs<S>;
        tile_steps<NW, OPT, RES, PULL, PH>(std::make_integer_sequence<int, kTileLoads<NW, S>>{}, p,
                                           a, b, nd, nrow, prow, has_next, state, o, tile_stash,
                                           &c);
        if constexpr (kStash<NW, S, RES, PULL>) {
            if (t - c.t_stash == kStashTiles<S> - 1 || !has_next ||
                in_write_window(o.wb_period, o.wb_window)) {
                write_stash<NW, S>(tiles, c.t_stash, t, stash, state);
                c.t_stash = t + 1;
            }
        }
        if (!has_next) return false;
        a = b;
        nd = nd2;
        prow = nprow;
        ++t;
        return true;
    };
    for (;;) {
        if (!one_tile(std::integral_constant<int, 0>{})) break;
        if constexpr (NPH >= 2)
            if (!one_tile(std::integral_constant<int, 1 % NPH>{})) break;
        if constexpr (NPH >= 3)
            if (!one_tile(std::integral_constant<int, 2 % NPH>{})) break;
    }
}

// The streamed full tiles of a launch taken from its pool (dynamic
// schedule), NW workers: walk_tiles' pipeline, with the next tiles known
// from takes instead of a fixed list.  The wave's counter serves the pool
// tiles pool[i * stride], i < count.  At the start of tile t the wave
// resolves the take of tile t + 2 (issued at the start of tile t - 1),
// fetches that tile's descriptor and issues the take of tile t + 3 (only
// while takes still land in the pool).
template <int NW, int OPT, bool PULL>
__device__ __forceinline__ void walk_pool(const DevTile* __restrict__ pool, int32_t count,
                                          int stride, unsigned long long* counter, uint64_t base,
                                          const float* const* __restrict__ grads,
                                          float* const* __restrict__ outs, float* const* state,
                                          OptArgs o, PHUB_LDS f4* stash) {
    constexpr bool RES = false;
    constexpr int S = kStates<OPT>;
    constexpr int NPH = kPhases<NW, S, RES>;
    static_assert(NPH >= 1 && NPH <= 3, "the tile loop below unrolls at most three phases");
    constexpr bool STASH = kStash<NW, S, RES, PULL>;
    constexpr int SLOTS = STASH ? kStashTiles<S> : 1;
    int32_t cur = resolve_take(issue_take(counter), base, count);
    if (cur < 0) return;
    int32_t n1 = resolve_take(issue_take(counter), base, count);
    bool take2 = n1 >= 0;  // a take of the tile after next is in flight
    uint64_t v2 = take2 ? issue_take(counter) : 0;
    TilePipe<NW, S, RES> p;
    TileStreams<NW, S> a, b;
    uint64_t prow = 0;
    {
        const DevTile first = pool[int64_t(cur) * stride];
        tile_streams<NW, S>(a, first, grads + int64_t(first.key) * NW, state);
        if constexpr (PULL) prow = load_row<NW>(outs + int64_t(first.key) * NW);
    }
    DevTile nd = pool[int64_t(n1 >= 0 ? n1 : cur) * stride];
    tile_prologue<NW, S, RES>(std::make_integer_sequence<int, kAhead<NW, S, RES>>{}, p, a);
    PoolCursor<SLOTS> c{pool, stride, stash, {}, 0, 0};  // burst write-back
    auto one_tile = [&](auto phase) -> bool {
        constexpr int PH = decltype(phase)::value;
        const bool has_next = n1 >= 0;
        const uint64_t nrow = load_row<NW>(grads + int64_t(nd.key) * NW);
        uint64_t nprow = 0;
        if constexpr (PULL) nprow = load_row<NW>(outs + int64_t(nd.key) * NW);
        const int32_t n2 = take2 ? resolve_take(v2, base, count) : -1;
        const bool take3 = n2 >= 0;
        const uint64_t v3 = take3 ? issue_take(counter) : 0;
        const DevTile nd2 = pool[int64_t(n2 >= 0 ? n2 : cur) * stride];
        PHUB_LDS f4* tile_stash = nullptr;  // this tile's slot of the stash
        if constexpr (STASH) {
            const int sl = c.n % SLOTS;
            tile_stash = stash + sl * kStashTileVecs<S>;
#pragma unroll
            for (int k = 0; k < SLOTS; ++k)
                if (k == sl) c.idx[k] = cur;
        }
        tile_steps<NW, OPT, RES, PULL, PH>(std::make_integer_sequence<int, kTileLoads<NW, S>>{}, p,
                                           a, b, nd, nrow, prow, has_next, state, o, tile_stash,
                                           &c);
        if constexpr (STASH) {
            ++c.n;
            if (c.n - c.first == SLOTS || !has_next || in_write_window(o.wb_period, o.wb_window))
                c.template write_back_to<NW, S>(c.n, state);
        }
        if (!has_next) return false;
        a = b;
        nd = nd2;
        prow = nprow;
        cur = n1;
        n1 = n2;
        take2 = take3;
        v2 = v3;
        return true;
    };
    for (;;) {
        if (!one_tile(std::integral_constant<int, 0>{})) break;
        if constexpr (NPH >= 2)
            if (!one_tile(std::integral_constant<int, 1 % NPH>{})) break;
        if constexpr (NPH >= 3)
            if (!one_tile(std::integral_constant<int, 2 % NPH>{})) break;
    }
}

// The remainders [rb, re) of one bin; `first` is rems[rb], which the wave
// has from its head.  The descriptor of the next remainder is fetched while
// this one is processed.
template <int NW, int OPT, bool RES, bool PULL>
__device__ __forceinline__ void walk_rems(const DevRem* __restrict__ rems, int32_t rb, int32_t re,
                                          const DevRem& first,
                                          const float* const* __restrict__ grads,
                                          float* const* __restrict__ outs, float* const* state,
                                          OptArgs o) {
    constexpr int S = kStates<OPT>;
    DevRem rm = first;
    for (int32_t r = rb; r < re; ++r) {
        const DevRem next = rems[r + 1 < re ? r + 1 : r];
        const float* g[NW];
        float* out[NW];
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            g[w] = grads[int64_t(rm.key) * NW + w] + rm.offset;
            out[w] = PULL ? outs[int64_t(rm.key) * NW + w] + rm.offset : nullptr;
        }
        float* stb[S];
#pragma unroll
        for (int i = 0; i < S; ++i) stb[i] = state[i] + rm.arena_offset;
        partial<NW, OPT, RES, PULL>(g, stb, out, uint32_t(rm.count) >> 2,
                                    uint32_t(rm.count) & 3u, o);
        rm = next;
    }
}

// NW > 0: exactly NW workers.  Each wave streams the full tiles of its
// streamed bin, then those of its cache-resident bin, then the remainders
// of both.  All waves thus work in the same phase at almost every moment:
// on MI355X that measured better than mixing the two kinds of traffic
// (odd waves in the other order), and slightly better than the resident
// bin first.  One wave per SIMD (one workgroup of 4 waves per CU).
#define PHUB_ONE_WAVE_PER_SIMD __attribute__((amdgpu_waves_per_eu(1, 1)))

template <int NW, int OPT, bool PULL>
__global__ __launch_bounds__(kBlockThreads) PHUB_ONE_WAVE_PER_SIMD void fused_step_fixed(
    PHUB_KERNEL_ARGS) {
    float* const state[3] = {weights, moments, second};
    const uint32_t wave = wave_index();
    constexpr int S = kStates<OPT>;
    PHUB_LDS f4* stash = nullptr;  // the lane's entry of its wave's stash
    if constexpr (kStash<NW, S, false, PULL>) {
        __shared__ f4 stash_lds[kWavesPerBlock * kStashTiles<S> * kStashTileVecs<S>];
        stash = (PHUB_LDS f4*)stash_lds +
                (threadIdx.x >> 6) * (kStashTiles<S> * kStashTileVecs<S>) + (threadIdx.x & 63u);
    }
    // the wave's bins and the first descriptor of each, read at once
    const WaveHead h = heads[wave];
    if (pool_count > 0) {
        // this workgroup's counter, the pool tiles it serves, and the
        // counter's value at the start of this launch
        const int nc = pool_counter_count(gridDim.x);
        const int c = int(blockIdx.x % uint32_t(nc));
        const int64_t served = pool_counter_tiles(pool_count, c, nc);
        const uint64_t per_launch =
            uint64_t(served) + uint64_t(kWavesPerBlock) * uint64_t(pool_counter_groups(gridDim.x, c, nc));
        walk_pool<NW, OPT, PULL>(pool + c, int32_t(served), nc,
                                 pool_counters + c * kPoolCounterStride,
                                 pool_launch * per_launch, grads, outs, state, o, stash);
    } else {
        walk_tiles<NW, OPT, false, PULL>(tiles, h.tiles_streamed[0], h.tiles_streamed[1],
                                         h.first_streamed, grads, outs, state, o, stash);
    }
    walk_tiles<NW, OPT, true, PULL>(tiles, h.tiles_resident[0], h.tiles_resident[1],
                                    h.first_resident, grads, outs, state, o, stash);
    walk_rems<NW, OPT, true, PULL>(rems, h.rems_resident[0], h.rems_resident[1],
                                   h.first_rem_resident, grads, outs, state, o);
    walk_rems<NW, OPT, false, PULL>(rems, h.rems_streamed[0], h.rems_streamed[1],
                                    h.first_rem_streamed, grads, outs, state, o);
}

// Any N: workers taken in batches of kBatch, each batch's loads in flight
// together, the running sum carried across batches in worker order.
constexpr int kBatch = 8;

__device__ __forceinline__ f4 sum_any(const float* const* kp, int n, int64_t offset,
                                      uint32_t bo) {
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
    return s;
}

// The same over kVecPerLane float4 per lane at once (1 KB apart): every
// batch keeps kBatch * kVecPerLane loads in flight.
__device__ __forceinline__ void sum_any_pieces(const float* const* kp, int n, int64_t offset,
                                               uint32_t bo, f4* s) {
#pragma unroll
    for (int u = 0; u < kVecPerLane; ++u) s[u] = load_stream(kp[0] + offset, bo + u * 1024u);
    for (int w0 = 1; w0 < n; w0 += kBatch) {
        f4 a[kBatch][kVecPerLane];
#pragma unroll
        for (int j = 0; j < kBatch; ++j)
            if (w0 + j < n) {
#pragma unroll
                for (int u = 0; u < kVecPerLane; ++u)
                    a[j][u] = load_stream(kp[w0 + j] + offset, bo + u * 1024u);
            }
#pragma unroll
        for (int j = 0; j < kBatch; ++j)
            if (w0 + j < n) {
#pragma unroll
                for (int u = 0; u < kVecPerLane; ++u) s[u] = s[u] + a[j][u];
            }
    }
}

template <int OPT, bool RES, bool PULL>
__device__ __forceinline__ void run_any(const float* const* kp, float* const* ko, int n,
                                        int64_t offset, float* const* stb, uint32_t nvec,
                                        uint32_t rem, OptArgs o) {
    constexpr int S = kStates<OPT>;
    const uint32_t lane = threadIdx.x & 63u;
    // whole groups of kVecPerLane * 64 float4 (a full tile is one), then the rest
    const uint32_t nfull = nvec / (64u * kVecPerLane) * (64u * kVecPerLane);
    for (uint32_t v = lane; v < nfull; v += 64u * kVecPerLane) {
        const uint32_t bo = v * 16u;
        f4 sum[kVecPerLane];
        sum_any_pieces(kp, n, offset, bo, sum);
        f4 st[kVecPerLane][S];
#pragma unroll
        for (int u = 0; u < kVecPerLane; ++u)
#pragma unroll
            for (int i = 0; i < S; ++i) st[u][i] = load_wm<RES>(stb[i], bo + u * 1024u);
#pragma unroll
        for (int u = 0; u < kVecPerLane; ++u) {
            update4<OPT>(sum[u], st[u], o);
#pragma unroll
            for (int i = 0; i < S; ++i) store_wm<RES>(stb[i], bo + u * 1024u, st[u][i]);
            if constexpr (PULL)
                for (int w = 0; w < n; ++w) store_out(ko[w] + offset, bo + u * 1024u, st[u][0]);
        }
    }
    for (uint32_t v = nfull + lane; v < nvec; v += 64u) {
        const uint32_t bo = v * 16u;
        const f4 s = sum_any(kp, n, offset, bo);
        f4 st[S];
#pragma unroll
        for (int i = 0; i < S; ++i) st[i] = load_wm<RES>(stb[i], bo);
        update4<OPT>(s, st, o);
#pragma unroll
        for (int i = 0; i < S; ++i) store_wm<RES>(stb[i], bo, st[i]);
        if constexpr (PULL)
            for (int w = 0; w < n; ++w) store_out(ko[w] + offset, bo, st[0]);
    }
    if (lane < rem) {
        const int64_t i = int64_t(nvec) * 4 + lane;
        float s = load1(kp[0] + offset, i);
        for (int w = 1; w < n; ++w) s = s + load1(kp[w] + offset, i);
        float st[S];
#pragma unroll
        for (int k = 0; k < S; ++k) st[k] = load1(stb[k], i);
        update<OPT>(s, st, o);
#pragma unroll
        for (int k = 0; k < S; ++k) store1(stb[k], i, st[k]);
        if constexpr (PULL)
            for (int w = 0; w < n; ++w) store1(ko[w] + offset, i, st[0]);
    }
}

// One bin of the any-N kernel: full tiles [tb, te), then remainders [rb, re).
template <int OPT, bool RES, bool PULL>
__device__ __forceinline__ void any_bin(const DevTile* __restrict__ tiles, int32_t tb, int32_t te,
                                        const DevRem* __restrict__ rems, int32_t rb, int32_t re,
                                        const float* const* __restrict__ grads,
                                        float* const* __restrict__ outs, float* const* state,
                                        int n, OptArgs o) {
    constexpr int S = kStates<OPT>;
    for (int32_t t = tb; t < te; ++t) {
        const DevTile tl = tiles[t];
        float* stb[S];
#pragma unroll
        for (int i = 0; i < S; ++i) stb[i] = state[i] + tl.arena_offset;
        run_any<OPT, RES, PULL>(grads + int64_t(tl.key) * n,
                                PULL ? outs + int64_t(tl.key) * n : nullptr, n,
                                int64_t(tl.vec) * 4, stb, uint32_t(kTileElems / 4), 0u, o);
    }
    for (int32_t r = rb; r < re; ++r) {
        const DevRem rm = rems[r];
        float* stb[S];
#pragma unroll
        for (int i = 0; i < S; ++i) stb[i] = state[i] + rm.arena_offset;
        run_any<OPT, RES, PULL>(grads + int64_t(rm.key) * n,
                                PULL ? outs + int64_t(rm.key) * n : nullptr, n, rm.offset, stb,
                                uint32_t(rm.count) >> 2, uint32_t(rm.count) & 3u, o);
    }
}

template <int OPT, bool PULL>
__global__ __launch_bounds__(kBlockThreads) void fused_step_any(PHUB_KERNEL_ARGS) {
    float* const state[3] = {weights, moments, second};
    const uint32_t wave = wave_index();
    const uint32_t bins = gridDim.x * kWavesPerBlock;
    any_bin<OPT, false, PULL>(tiles, tile_begin[bins + wave], tile_begin[bins + wave + 1], rems,
                              rem_begin[bins + wave], rem_begin[bins + wave + 1], grads, outs,
                              state, num_workers, o);
    any_bin<OPT, true, PULL>(tiles, tile_begin[wave], tile_begin[wave + 1], rems, rem_begin[wave],
                             rem_begin[wave + 1], grads, outs, state, num_workers, o);
}

// Ablation: the unfused ("wide") form of the step, kept to measure what
// fusion saves.  Pass 1 sums the N gradients of every element in worker
// order and writes the sum to a merge buffer laid out like W; pass 2 reads
// the merge buffer and the state and runs the optimizer.  Same arithmetic,
// same schedule, (N + 2 S + 2) * 4 bytes per element instead of
// (N + 2 S) * 4, and two launches.
__device__ __forceinline__ void aggregate_range(const float* const* kp, int n, int64_t offset,
                                                float* out, uint32_t nvec, uint32_t rem) {
    const uint32_t lane = threadIdx.x & 63u;
    for (uint32_t v = lane; v < nvec; v += 64u)
        store_out(out, v * 16u, sum_any(kp, n, offset, v * 16u));
    if (lane < rem) {
        const int64_t i = int64_t(nvec) * 4 + lane;
        float s = load1(kp[0] + offset, i);
        for (int w = 1; w < n; ++w) s = s + load1(kp[w] + offset, i);
        store1(out, i, s);
    }
}

template <int OPT, bool RES>
__device__ __forceinline__ void optimize_range(const float* sum, float* const* stb, uint32_t nvec,
                                               uint32_t rem, OptArgs o) {
    constexpr int S = kStates<OPT>;
    const uint32_t lane = threadIdx.x & 63u;
    for (uint32_t v = lane; v < nvec; v += 64u) {
        const uint32_t bo = v * 16u;
        const f4 s = load_stream(sum, bo);
        f4 st[S];
#pragma unroll
        for (int i = 0; i < S; ++i) st[i] = load_wm<RES>(stb[i], bo);
        update4<OPT>(s, st, o);
#pragma unroll
        for (int i = 0; i < S; ++i) store_wm<RES>(stb[i], bo, st[i]);
    }
    if (lane < rem) {
        const int64_t i = int64_t(nvec) * 4 + lane;
        float st[S];
#pragma unroll
        for (int k = 0; k < S; ++k) st[k] = load1(stb[k], i);
        update<OPT>(load1(sum, i), st, o);
#pragma unroll
        for (int k = 0; k < S; ++k) store1(stb[k], i, st[k]);
    }
}

__global__ __launch_bounds__(kBlockThreads) void aggregate_only(PHUB_KERNEL_ARGS, float* merge) {
    const uint32_t wave = wave_index();
    const uint32_t bins = gridDim.x * kWavesPerBlock;
    const int n = num_workers;
    for (uint32_t bin : {wave, bins + wave}) {
        for (int32_t t = tile_begin[bin]; t < tile_begin[bin + 1]; ++t) {
            const DevTile tl = tiles[t];
            aggregate_range(grads + int64_t(tl.key) * n, n, int64_t(tl.vec) * 4,
                            merge + tl.arena_offset, uint32_t(kTileElems / 4), 0u);
        }
        for (int32_t r = rem_begin[bin]; r < rem_begin[bin + 1]; ++r) {
            const DevRem rm = rems[r];
            aggregate_range(grads + int64_t(rm.key) * n, n, rm.offset, merge + rm.arena_offset,
                            uint32_t(rm.count) >> 2, uint32_t(rm.count) & 3u);
        }
    }
}

template <int OPT, bool RES>
__device__ __forceinline__ void optimize_bin(const DevTile* __restrict__ tiles, int32_t tb,
                                             int32_t te, const DevRem* __restrict__ rems,
                                             int32_t rb, int32_t re, const float* merge,
                                             float* const* state, OptArgs o) {
    constexpr int S = kStates<OPT>;
    for (int32_t t = tb; t < te; ++t) {
        const DevTile tl = tiles[t];
        float* stb[S];
#pragma unroll
        for (int i = 0; i < S; ++i) stb[i] = state[i] + tl.arena_offset;
        optimize_range<OPT, RES>(merge + tl.arena_offset, stb, uint32_t(kTileElems / 4), 0u, o);
    }
    for (int32_t r = rb; r < re; ++r) {
        const DevRem rm = rems[r];
        float* stb[S];
#pragma unroll
        for (int i = 0; i < S; ++i) stb[i] = state[i] + rm.arena_offset;
        optimize_range<OPT, RES>(merge + rm.arena_offset, stb, uint32_t(rm.count) >> 2,
                                 uint32_t(rm.count) & 3u, o);
    }
}

template <int OPT>
__global__ __launch_bounds__(kBlockThreads) void optimize_only(PHUB_KERNEL_ARGS, float* merge) {
    float* const state[3] = {weights, moments, second};
    const uint32_t wave = wave_index();
    const uint32_t bins = gridDim.x * kWavesPerBlock;
    optimize_bin<OPT, true>(tiles, tile_begin[wave], tile_begin[wave + 1], rems, rem_begin[wave],
                            rem_begin[wave + 1], merge, state, o);
    optimize_bin<OPT, false>(tiles, tile_begin[bins + wave], tile_begin[bins + wave + 1], rems,
                             rem_begin[bins + wave], rem_begin[bins + wave + 1], merge, state, o);
}

// -------------------------------------------------------------- launchers

#define PHUB_LAUNCH_ARGS                                                                     \
    p.tiles, p.tile_begin, p.rems, p.rem_begin, p.heads, p.grads, p.outs, p.weights,         \
        p.moments,                                                                           \
        p.second, p.opt, p.num_workers, p.pool, p.pool_count, p.pool_counters, p.pool_launch

template <int OPT, bool PULL>
hipError_t launch_any(const StepParams& p, int grid, hipStream_t stream) {
    hipLaunchKernelGGL((fused_step_any<OPT, PULL>), dim3(grid), dim3(kBlockThreads), 0, stream,
                       PHUB_LAUNCH_ARGS);
    return hipGetLastError();
}

template <int NW, int OPT, bool PULL>
hipError_t launch_one(const StepParams& p, int grid, hipStream_t stream) {
    constexpr int S = kStates<OPT>;
    if constexpr (kPhases<NW, S, true> <= 3 && kPhases<NW, S, false> <= 3) {
        hipLaunchKernelGGL((fused_step_fixed<NW, OPT, PULL>), dim3(grid), dim3(kBlockThreads), 0,
                           stream, PHUB_LAUNCH_ARGS);
        return hipGetLastError();
    } else {
        return launch_any<OPT, PULL>(p, grid, stream);
    }
}

template <int OPT, bool PULL>
hipError_t launch_pull(const StepParams& p, int grid, hipStream_t stream) {
    static_assert(kMaxFixedWorkers == 16, "one case per fixed worker count");
    static_assert(has_fixed_kernel(20) && has_fixed_kernel(24) && has_fixed_kernel(32),
                  "the larger counts below");
    switch (p.num_workers) {
        case 1: return launch_one<1, OPT, PULL>(p, grid, stream);
        case 2: return launch_one<2, OPT, PULL>(p, grid, stream);
        case 3: return launch_one<3, OPT, PULL>(p, grid, stream);
        case 4: return launch_one<4, OPT, PULL>(p, grid, stream);
        case 5: return launch_one<5, OPT, PULL>(p, grid, stream);
        case 6: return launch_one<6, OPT, PULL>(p, grid, stream);
        case 7: return launch_one<7, OPT, PULL>(p, grid, stream);
        case 8: return launch_one<8, OPT, PULL>(p, grid, stream);
        case 9: return launch_one<9, OPT, PULL>(p, grid, stream);
        case 10: return launch_one<10, OPT, PULL>(p, grid, stream);
        case 11: return launch_one<11, OPT, PULL>(p, grid, stream);
        case 12: return launch_one<12, OPT, PULL>(p, grid, stream);
        case 13: return launch_one<13, OPT, PULL>(p, grid, stream);
        case 14: return launch_one<14, OPT, PULL>(p, grid, stream);
        case 15: return launch_one<15, OPT, PULL>(p, grid, stream);
        case 16: return launch_one<16, OPT, PULL>(p, grid, stream);
        case 20: return launch_one<20, OPT, PULL>(p, grid, stream);
        case 24: return launch_one<24, OPT, PULL>(p, grid, stream);
        case 32: return launch_one<32, OPT, PULL>(p, grid, stream);
        default: return launch_any<OPT, PULL>(p, grid, stream);
    }
}

template <int OPT>
hipError_t launch_unfused(const StepParams& p, int grid, hipStream_t stream) {
    hipLaunchKernelGGL(aggregate_only, dim3(grid), dim3(kBlockThreads), 0, stream,
                       PHUB_LAUNCH_ARGS, p.merge);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    hipLaunchKernelGGL((optimize_only<OPT>), dim3(grid), dim3(kBlockThreads), 0, stream,
                       PHUB_LAUNCH_ARGS, p.merge);
    return hipGetLastError();
}

template <int OPT>
hipError_t launch_opt(const StepParams& p, int grid, hipStream_t stream) {
    if (p.merge) return launch_unfused<OPT>(p, grid, stream);
    return p.outs ? launch_pull<OPT, true>(p, grid, stream)
                  : launch_pull<OPT, false>(p, grid, stream);
}

}  // namespace

namespace {

template <int NW, int S>
constexpr bool fixed_launchable() {
    return kPhases<NW, S, true> <= 3 && kPhases<NW, S, false> <= 3;
}

template <int S>
bool fixed_launchable_n(int n) {
    switch (n) {
        case 1: return fixed_launchable<1, S>();
        case 2: return fixed_launchable<2, S>();
        case 3: return fixed_launchable<3, S>();
        case 4: return fixed_launchable<4, S>();
        case 5: return fixed_launchable<5, S>();
        case 6: return fixed_launchable<6, S>();
        case 7: return fixed_launchable<7, S>();
        case 8: return fixed_launchable<8, S>();
        case 9: return fixed_launchable<9, S>();
        case 10: return fixed_launchable<10, S>();
        case 11: return fixed_launchable<11, S>();
        case 12: return fixed_launchable<12, S>();
        case 13: return fixed_launchable<13, S>();
        case 14: return fixed_launchable<14, S>();
        case 15: return fixed_launchable<15, S>();
        case 16: return fixed_launchable<16, S>();
        case 20: return fixed_launchable<20, S>();
        case 24: return fixed_launchable<24, S>();
        case 32: return fixed_launchable<32, S>();
        default: return false;
    }
}

}  // namespace

bool takes_tile_pool(int num_workers, int optimizer) {
    switch (optimizer) {
        case kOptMomentum:
        case kOptNesterov: return fixed_launchable_n<2>(num_workers);
        case kOptSgd: return fixed_launchable_n<1>(num_workers);
        case kOptAdam: return fixed_launchable_n<3>(num_workers);
        default: return false;
    }
}

hipError_t launch_fused_step(const StepParams& p, int optimizer, int grid, hipStream_t stream) {
    if (p.pool_count > 0 && (p.merge || !takes_tile_pool(p.num_workers, optimizer)))
        return hipErrorInvalidValue;  // only the fixed-N fused kernels walk a pool
    if (!p.merge && !p.heads) return hipErrorInvalidValue;  // the fixed-N kernels read them
    switch (optimizer) {
        case kOptMomentum: return launch_opt<kOptMomentum>(p, grid, stream);
        case kOptNesterov: return launch_opt<kOptNesterov>(p, grid, stream);
        case kOptSgd: return launch_opt<kOptSgd>(p, grid, stream);
        case kOptAdam: return launch_opt<kOptAdam>(p, grid, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace phub
