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
// few waves per CU, each keeping many bytes in flight, rather than with many
// small workgroups.
//
// Memory access: a wave's hot loop moves one tile per iteration, 1024
// elements of each of the N + 2 arrays: a lane loads 4 float4 of each
// (the wave's 64 lanes cover 4 contiguous 1 KB pieces), all 4 * N gradient
// loads in flight before the first addition.  Segments are cut on the host
// into full tiles and a remainder, so the hot loop is straight-line code.
// Gradients are read once per step and loaded non-temporally.  W and M are
// read and written non-temporally, unless the job asks for them to stay in
// the memory-side cache between steps (RES: default, cache-allocating
// policy for every W and M access of the launch).  Tile descriptors and
// per-key gradient pointers are uniform per wave and come through scalar
// loads, prefetched two tiles ahead.
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

__device__ __forceinline__ f4 load_wm(const float* base, uint32_t byte_off, bool resident) {
    const PHUB_GLOBAL f4* a = (const PHUB_GLOBAL f4*)((const PHUB_GLOBAL char*)base + byte_off);
    return resident ? *a : __builtin_nontemporal_load(a);
}

__device__ __forceinline__ void store_wm(float* base, uint32_t byte_off, const f4& v, bool resident) {
    PHUB_GLOBAL f4* a = (PHUB_GLOBAL f4*)((PHUB_GLOBAL char*)base + byte_off);
    if (resident)
        *a = v;
    else
        __builtin_nontemporal_store(v, a);
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
        const float* const* __restrict__ grads, float* __restrict__ weights,              \
        float* __restrict__ moments, float lr, float mu, float wd, int num_workers

// One full tile: kVecPerLane float4 per lane of each array.  g[w], wb and
// mb are uniform base pointers; the tile starts at float4 index `vec` from
// them, and lane l takes the float4s at vec + l, + 64, + 128 and + 192.  The
// per-lane byte offset is formed inside the loop from the tile's (uniform)
// index, so that the compiler addresses every load and store as uniform
// base + 32-bit lane offset + immediate.  All NW * kVecPerLane gradient
// loads and the W and M loads are issued before the first addition.
template <int NW, bool NEST, bool RES>
__device__ __forceinline__ void full_tile(const float* const* g, float* wb, float* mb,
                                          uint32_t vec, float nlr, float mu, float wd) {
    constexpr int U = kVecPerLane;
    const uint32_t off = (vec + (threadIdx.x & 63u)) * 16u;
    f4 a[U][NW];
    f4 wv[U], mv[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int w = 0; w < NW; ++w) a[u][w] = load_stream(g[w], off + u * 1024u);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        wv[u] = load_wm(wb, off + u * 1024u, RES);
        mv[u] = load_wm(mb, off + u * 1024u, RES);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        f4 s = a[u][0];
#pragma unroll
        for (int w = 1; w < NW; ++w) s = s + a[u][w];
        optimize4<NEST>(s, wv[u], mv[u], nlr, mu, wd);
        store_wm(wb, off + u * 1024u, wv[u], RES);
        store_wm(mb, off + u * 1024u, mv[u], RES);
    }
}

// The rest of a segment: nvec < 256 float4 then a ragged end of rem < 4
// elements (one per lane).
template <int NW, bool NEST, bool RES>
__device__ __forceinline__ void partial(const float* const* g, float* wb, float* mb,
                                        uint32_t nvec, uint32_t rem, float nlr, float mu,
                                        float wd) {
    const uint32_t lane = threadIdx.x & 63u;
    for (uint32_t v = lane; v < nvec; v += 64u) {
        f4 a[NW];
#pragma unroll
        for (int w = 0; w < NW; ++w) a[w] = load_stream(g[w], v * 16u);
        f4 wv = load_wm(wb, v * 16u, RES);
        f4 mv = load_wm(mb, v * 16u, RES);
        f4 s = a[0];
#pragma unroll
        for (int w = 1; w < NW; ++w) s = s + a[w];
        optimize4<NEST>(s, wv, mv, nlr, mu, wd);
        store_wm(wb, v * 16u, wv, RES);
        store_wm(mb, v * 16u, mv, RES);
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
    }
}

// Scalar loads return out of order, so the compiler waits for all of them
// (lgkmcnt(0)) before it uses any.  `settle` uses values whose loads were
// issued one tile earlier, so that this single wait happens before the next
// prefetches are issued; the scheduling barriers keep the compiler from
// moving the new scalar loads above it (they would then be waited on too).
__device__ __forceinline__ void settle32(uint32_t v) { asm volatile("" ::"s"(v)); }
__device__ __forceinline__ void settle64(const void* p) { asm volatile("" ::"s"(p)); }

__device__ __forceinline__ void settle_tile(const DevTile& t) {
    settle64(reinterpret_cast<const void*>(t.arena_offset));
    settle32(uint32_t(t.key));
    settle32(uint32_t(t.vec));
}

// NW > 0: exactly NW workers.  Each wave first streams its full tiles, with
// a two-deep prefetch (while tile i streams, the descriptor of tile i + 2
// and the gradient pointers of tile i + 1 are on their way), then its
// remainders.
// Splits a tile's float4 index into a part folded into the base pointers
// (a multiple of 2^20 float4, 16 MB) and a low part that keeps the per-lane
// 32-bit byte offset far from overflow.
constexpr uint32_t kVecLowMask = (1u << 20) - 1;

// One wave per SIMD (one workgroup of 4 waves per CU): the compiler may use
// the whole register file for loads in flight instead of trading them for
// occupancy.
#define PHUB_ONE_WAVE_PER_SIMD __attribute__((amdgpu_waves_per_eu(1, 1)))

template <int NW, bool NEST, bool RES>
__global__ __launch_bounds__(kBlockThreads) PHUB_ONE_WAVE_PER_SIMD void fused_step_fixed(
    PHUB_KERNEL_ARGS) {
    const uint32_t wave = wave_index();
    const float nlr = -lr;

    const int32_t tb = tile_begin[wave];
    const int32_t te = tile_begin[wave + 1];
    if (tb < te) {
        const int32_t last = te - 1;
        DevTile cur = tiles[tb];
        const float* gc[NW];
#pragma unroll
        for (int w = 0; w < NW; ++w) gc[w] = grads[int64_t(cur.key) * NW + w];
        DevTile nxt = tiles[tb + 1 <= last ? tb + 1 : last];
        for (int32_t t = tb; t <= last; ++t) {
            settle_tile(cur);
            settle_tile(nxt);
#pragma unroll
            for (int w = 0; w < NW; ++w) settle64(gc[w]);
            __builtin_amdgcn_sched_barrier(0);
            const float* gn[NW];
#pragma unroll
            for (int w = 0; w < NW; ++w) gn[w] = grads[int64_t(nxt.key) * NW + w];
            const DevTile nxt2 = tiles[t + 2 <= last ? t + 2 : last];
            __builtin_amdgcn_sched_barrier(0);

            const uint32_t vhi = uint32_t(cur.vec) & ~kVecLowMask;
            const uint32_t vlo = uint32_t(cur.vec) & kVecLowMask;
            const float* g[NW];
#pragma unroll
            for (int w = 0; w < NW; ++w) g[w] = gc[w] + size_t(vhi) * 4;
            full_tile<NW, NEST, RES>(g, weights + cur.arena_offset - size_t(vlo) * 4,
                                     moments + cur.arena_offset - size_t(vlo) * 4, vlo, nlr, mu,
                                     wd);
            __builtin_amdgcn_sched_barrier(0);
            cur = nxt;
#pragma unroll
            for (int w = 0; w < NW; ++w) gc[w] = gn[w];
            nxt = nxt2;
        }
    }

    const int32_t rb = rem_begin[wave];
    const int32_t re = rem_begin[wave + 1];
    for (int32_t r = rb; r < re; ++r) {
        const DevRem rm = rems[r];
        const float* g[NW];
#pragma unroll
        for (int w = 0; w < NW; ++w) g[w] = grads[int64_t(rm.key) * NW + w] + rm.offset;
        partial<NW, NEST, RES>(g, weights + rm.arena_offset, moments + rm.arena_offset,
                               uint32_t(rm.count) >> 2, uint32_t(rm.count) & 3u, nlr, mu, wd);
    }
}

// Any N: workers taken in batches of kBatch, each batch's loads in flight
// together, the running sum carried across batches in worker order.
constexpr int kBatch = 8;

template <bool NEST, bool RES>
__device__ __forceinline__ void run_any(const float* const* kp, int n, int64_t offset, float* wb,
                                        float* mb, uint32_t nvec, uint32_t rem, float nlr,
                                        float mu, float wd) {
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
        f4 wv = load_wm(wb, bo, RES);
        f4 mv = load_wm(mb, bo, RES);
        optimize4<NEST>(s, wv, mv, nlr, mu, wd);
        store_wm(wb, bo, wv, RES);
        store_wm(mb, bo, mv, RES);
    }
    if (lane < rem) {
        const int64_t i = int64_t(nvec) * 4 + lane;
        float s = load1(kp[0] + offset, i);
        for (int w = 1; w < n; ++w) s = s + load1(kp[w] + offset, i);
        float wv = load1(wb, i), mv = load1(mb, i);
        optimize<NEST>(s, wv, mv, nlr, mu, wd);
        store1(wb, i, wv);
        store1(mb, i, mv);
    }
}

template <bool NEST, bool RES>
__global__ __launch_bounds__(kBlockThreads) void fused_step_any(PHUB_KERNEL_ARGS) {
    const uint32_t wave = wave_index();
    const int n = num_workers;
    const float nlr = -lr;
    const int32_t tb = tile_begin[wave];
    const int32_t te = tile_begin[wave + 1];
    for (int32_t t = tb; t < te; ++t) {
        const DevTile tl = tiles[t];
        run_any<NEST, RES>(grads + int64_t(tl.key) * n, n, int64_t(tl.vec) * 4,
                           weights + tl.arena_offset, moments + tl.arena_offset,
                           uint32_t(kTileElems / 4), 0u, nlr, mu, wd);
    }
    const int32_t rb = rem_begin[wave];
    const int32_t re = rem_begin[wave + 1];
    for (int32_t r = rb; r < re; ++r) {
        const DevRem rm = rems[r];
        run_any<NEST, RES>(grads + int64_t(rm.key) * n, n, rm.offset, weights + rm.arena_offset,
                           moments + rm.arena_offset, uint32_t(rm.count) >> 2,
                           uint32_t(rm.count) & 3u, nlr, mu, wd);
    }
}

#define PHUB_LAUNCH_ARGS                                                                    \
    p.tiles, p.tile_begin, p.rems, p.rem_begin, p.grads, p.weights, p.moments, p.lr, p.mu, \
        p.wd, p.num_workers

template <int NW, bool RES>
hipError_t launch_n(const StepParams& p, bool nesterov, int grid, hipStream_t stream) {
    if (nesterov)
        hipLaunchKernelGGL((fused_step_fixed<NW, true, RES>), dim3(grid), dim3(kBlockThreads), 0,
                           stream, PHUB_LAUNCH_ARGS);
    else
        hipLaunchKernelGGL((fused_step_fixed<NW, false, RES>), dim3(grid), dim3(kBlockThreads), 0,
                           stream, PHUB_LAUNCH_ARGS);
    return hipGetLastError();
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
        default:
            if (nesterov)
                hipLaunchKernelGGL((fused_step_any<true, RES>), dim3(grid), dim3(kBlockThreads), 0,
                                   stream, PHUB_LAUNCH_ARGS);
            else
                hipLaunchKernelGGL((fused_step_any<false, RES>), dim3(grid), dim3(kBlockThreads), 0,
                                   stream, PHUB_LAUNCH_ARGS);
            return hipGetLastError();
    }
}

}  // namespace

hipError_t launch_fused_step(const StepParams& p, bool nesterov, bool resident, int grid,
                             hipStream_t stream) {
    return resident ? launch_res<true>(p, nesterov, grid, stream)
                    : launch_res<false>(p, nesterov, grid, stream);
}

}  // namespace phub
