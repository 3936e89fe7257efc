// Fused aggregate + optimize kernel of the exchange step, for gfx950.
//
// One wave plays the role of one PHub core (paper, section 3.2.4): it walks
// the list of segments (runs of chunks) the schedule fixed for it at
// initialisation, and for each element it sums the N workers' gradients
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
// Memory access: a lane handles U float4 of each array per iteration, the
// wave's 64 lanes covering U contiguous 1 KB pieces of each of the N + 2
// arrays, all N * U gradient loads in flight before the first addition.
// Gradients are read once per step and loaded non-temporally.  W and M are
// read and written non-temporally, except a leading part of the arenas
// (resident_elems) that uses the default policy so that it can stay in the
// memory-side cache between steps.  Segment descriptors and per-key
// gradient pointers are uniform per wave and come through scalar loads.
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

// float4 per lane per array and iteration: all N * U gradient loads of a
// lane are live at once (up to 16 * 4 * 4 = 256 VGPRs of data at N = 16,
// within the 512 a lane may use at one wave per SIMD).
template <int NW>
constexpr int vec_per_lane() {
#if defined(PHUB_VEC_PER_LANE) && PHUB_VEC_PER_LANE > 0
    return PHUB_VEC_PER_LANE;
#else
    return 4;
#endif
}

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
#define PHUB_KERNEL_ARGS                                                            \
    const DevSegment* __restrict__ segments, const int64_t* __restrict__ bin_begin, \
        const float* const* __restrict__ grads, float* __restrict__ weights,        \
        float* __restrict__ moments, float lr, float mu, float wd, int num_workers, \
        int64_t resident_elems

// One segment, exactly NW workers, processed by the calling wave alone.
template <int NW, int U, bool NEST, bool RES>
__device__ __forceinline__ void segment_fixed(const float* const* g, float* wb, float* mb,
                                              uint32_t nvec, float nlr, float mu, float wd) {
    const uint32_t lane = threadIdx.x & 63u;
    for (uint32_t base = 0; base < nvec; base += 64u * U) {
        f4 a[U][NW];
        f4 wv[U], mv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t v = base + u * 64u + lane;
            if (v < nvec) {
#pragma unroll
                for (int w = 0; w < NW; ++w) a[u][w] = load_stream(g[w], v * 16u);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t v = base + u * 64u + lane;
            if (v < nvec) {
                wv[u] = load_wm(wb, v * 16u, RES);
                mv[u] = load_wm(mb, v * 16u, RES);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t v = base + u * 64u + lane;
            if (v < nvec) {
                f4 s = a[u][0];
#pragma unroll
                for (int w = 1; w < NW; ++w) s = s + a[u][w];
                optimize4<NEST>(s, wv[u], mv[u], nlr, mu, wd);
                store_wm(wb, v * 16u, wv[u], RES);
                store_wm(mb, v * 16u, mv[u], RES);
            }
        }
    }
}

// NW > 0: exactly NW workers.
template <int NW, bool NEST>
__global__ __launch_bounds__(kBlockThreads) void fused_step_fixed(PHUB_KERNEL_ARGS) {
    const uint32_t wave = wave_index();
    const int64_t sb = bin_begin[wave];
    const int64_t se = bin_begin[wave + 1];
    const uint32_t lane = threadIdx.x & 63u;
    const float nlr = -lr;
    for (int64_t si = sb; si < se; ++si) {
        const DevSegment sg = segments[si];
        const float* const* kp = grads + int64_t(sg.key) * NW;
        const float* g[NW];
#pragma unroll
        for (int w = 0; w < NW; ++w) g[w] = kp[w] + sg.offset;
        float* wb = weights + sg.arena_offset;
        float* mb = moments + sg.arena_offset;

        const uint32_t nvec = uint32_t(sg.count) >> 2;
        if (sg.arena_offset + sg.count <= resident_elems)
            segment_fixed<NW, vec_per_lane<NW>(), NEST, true>(g, wb, mb, nvec, nlr, mu, wd);
        else
            segment_fixed<NW, vec_per_lane<NW>(), NEST, false>(g, wb, mb, nvec, nlr, mu, wd);
        // ragged end of a key: fewer than 4 elements, one per lane
        const uint32_t rem = uint32_t(sg.count) & 3u;
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
}

// Any N: workers taken in batches of kBatch, each batch's loads in flight
// together, the running sum carried across batches in worker order.
constexpr int kBatch = 8;

template <bool NEST>
__global__ __launch_bounds__(kBlockThreads) void fused_step_any(PHUB_KERNEL_ARGS) {
    const uint32_t wave = wave_index();
    const int64_t sb = bin_begin[wave];
    const int64_t se = bin_begin[wave + 1];
    const uint32_t lane = threadIdx.x & 63u;
    const int n = num_workers;
    const float nlr = -lr;
    for (int64_t si = sb; si < se; ++si) {
        const DevSegment sg = segments[si];
        const float* const* kp = grads + int64_t(sg.key) * n;
        float* wb = weights + sg.arena_offset;
        float* mb = moments + sg.arena_offset;
        const bool res = sg.arena_offset + sg.count <= resident_elems;
        const uint32_t nvec = uint32_t(sg.count) >> 2;
        for (uint32_t v = lane; v < nvec; v += 64u) {
            const uint32_t bo = v * 16u;
            f4 s = load_stream(kp[0] + sg.offset, bo);
            for (int w0 = 1; w0 < n; w0 += kBatch) {
                f4 a[kBatch];
#pragma unroll
                for (int j = 0; j < kBatch; ++j)
                    if (w0 + j < n) a[j] = load_stream(kp[w0 + j] + sg.offset, bo);
#pragma unroll
                for (int j = 0; j < kBatch; ++j)
                    if (w0 + j < n) s = s + a[j];
            }
            f4 wv = load_wm(wb, bo, res);
            f4 mv = load_wm(mb, bo, res);
            optimize4<NEST>(s, wv, mv, nlr, mu, wd);
            store_wm(wb, bo, wv, res);
            store_wm(mb, bo, mv, res);
        }
        const uint32_t rem = uint32_t(sg.count) & 3u;
        if (lane < rem) {
            const int64_t i = int64_t(nvec) * 4 + lane;
            float s = load1(kp[0] + sg.offset, i);
            for (int w = 1; w < n; ++w) s = s + load1(kp[w] + sg.offset, i);
            float wv = load1(wb, i), mv = load1(mb, i);
            optimize<NEST>(s, wv, mv, nlr, mu, wd);
            store1(wb, i, wv);
            store1(mb, i, mv);
        }
    }
}

#define PHUB_LAUNCH_ARGS                                                                     \
    p.segments, p.bin_begin, p.grads, p.weights, p.moments, p.lr, p.mu, p.wd, p.num_workers, \
        p.resident_elems

template <int NW>
hipError_t launch_n(const StepParams& p, bool nesterov, int grid, hipStream_t stream) {
    if (nesterov)
        hipLaunchKernelGGL((fused_step_fixed<NW, true>), dim3(grid), dim3(kBlockThreads), 0, stream,
                           PHUB_LAUNCH_ARGS);
    else
        hipLaunchKernelGGL((fused_step_fixed<NW, false>), dim3(grid), dim3(kBlockThreads), 0,
                           stream, PHUB_LAUNCH_ARGS);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_fused_step(const StepParams& p, bool nesterov, int grid, hipStream_t stream) {
    switch (p.num_workers) {
        case 1: return launch_n<1>(p, nesterov, grid, stream);
        case 2: return launch_n<2>(p, nesterov, grid, stream);
        case 3: return launch_n<3>(p, nesterov, grid, stream);
        case 4: return launch_n<4>(p, nesterov, grid, stream);
        case 5: return launch_n<5>(p, nesterov, grid, stream);
        case 6: return launch_n<6>(p, nesterov, grid, stream);
        case 7: return launch_n<7>(p, nesterov, grid, stream);
        case 8: return launch_n<8>(p, nesterov, grid, stream);
        case 9: return launch_n<9>(p, nesterov, grid, stream);
        case 10: return launch_n<10>(p, nesterov, grid, stream);
        case 11: return launch_n<11>(p, nesterov, grid, stream);
        case 12: return launch_n<12>(p, nesterov, grid, stream);
        case 13: return launch_n<13>(p, nesterov, grid, stream);
        case 14: return launch_n<14>(p, nesterov, grid, stream);
        case 15: return launch_n<15>(p, nesterov, grid, stream);
        case 16: return launch_n<16>(p, nesterov, grid, stream);
        default:
            if (nesterov)
                hipLaunchKernelGGL((fused_step_any<true>), dim3(grid), dim3(kBlockThreads), 0,
                                   stream, PHUB_LAUNCH_ARGS);
            else
                hipLaunchKernelGGL((fused_step_any<false>), dim3(grid), dim3(kBlockThreads), 0,
                                   stream, PHUB_LAUNCH_ARGS);
            return hipGetLastError();
    }
}

}  // namespace phub
