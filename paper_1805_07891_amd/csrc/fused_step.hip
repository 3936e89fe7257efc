// Fused aggregate + optimize kernel of the exchange step, for gfx950.
//
// One workgroup plays the role of one PHub core (paper, section 3.2.4): it
// walks the segments the schedule gave it, and for each element of a
// segment it sums the N workers' gradients (section 3.2.2, "tall"
// aggregation: one worker of the GPU takes the same chunk across all
// gradient arrays) and immediately runs the optimizer on that element
// (section 3.2.2: the thread that aggregates a chunk also optimizes it).
// The partial sum never leaves registers, so there is no merge buffer:
// each gradient byte is read once and W and M are read and written once.
//
// Memory access: a lane handles 4 consecutive fp32 values (16-byte loads);
// consecutive lanes take consecutive 16-byte pieces, so a wave reads 1 KB
// of each of the N + 2 arrays with fully coalesced dwordx4 loads.  All N
// gradient loads of a lane are issued before the first addition.  Gradients
// are read once per step and are loaded non-temporally; W and M use the
// default policy.  Segment descriptors and per-key gradient pointers are
// uniform across the workgroup and come through scalar loads.
//
// Arithmetic (no MFMA: the work is elementwise and HBM-bound): the sum is a
// left fold in ascending worker index, plain fp32 additions; then four
// fused multiply-adds:
//     d = wd*w + s;  m' = mu*m + d;  u = mu*m' + d (Nesterov) or m';
//     w' = -lr*u + w.
// The file is compiled with -ffp-contract=off and without fast-math, so the
// compiler neither fuses nor reorders beyond the explicit fmaf calls, and
// subnormals are kept.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.hpp"

namespace phub {

typedef float f4 __attribute__((ext_vector_type(4)));

namespace {

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

__device__ __forceinline__ f4 load_keep(const float* base, uint32_t byte_off) {
    const PHUB_GLOBAL char* b = (const PHUB_GLOBAL char*)base;
    return *(const PHUB_GLOBAL f4*)(b + byte_off);
}

__device__ __forceinline__ void store_keep(float* base, uint32_t byte_off, const f4& v) {
    PHUB_GLOBAL char* b = (PHUB_GLOBAL char*)base;
    *(PHUB_GLOBAL f4*)(b + byte_off) = v;
}

__device__ __forceinline__ float load1(const float* base, int64_t i) {
    return ((const PHUB_GLOBAL float*)base)[i];
}

__device__ __forceinline__ void store1(float* base, int64_t i, float v) {
    ((PHUB_GLOBAL float*)base)[i] = v;
}

// The kernel arguments are __restrict__: the schedule and the pointer table
// are never written by the kernel and W/M never alias the gradients, which
// lets the compiler fetch descriptors and pointers with scalar loads.
#define PHUB_KERNEL_ARGS                                                              \
    const DevSegment* __restrict__ segments, const int64_t* __restrict__ group_begin, \
        const float* const* __restrict__ grads, float* __restrict__ weights,          \
        float* __restrict__ moments, float lr, float mu, float wd, int num_workers

// NW > 0: exactly NW workers, all loads of a lane in flight together.
template <int NW, bool NEST>
__global__ __launch_bounds__(kMaxBlockThreads) void fused_step_fixed(PHUB_KERNEL_ARGS) {
    const int64_t sb = group_begin[blockIdx.x];
    const int64_t se = group_begin[blockIdx.x + 1];
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
        for (uint32_t v = threadIdx.x; v < nvec; v += blockDim.x) {
            const uint32_t bo = v * 16u;
            f4 a[NW];
#pragma unroll
            for (int w = 0; w < NW; ++w) a[w] = load_stream(g[w], bo);
            f4 wv = load_keep(wb, bo);
            f4 mv = load_keep(mb, bo);
            f4 s = a[0];
#pragma unroll
            for (int w = 1; w < NW; ++w) s = s + a[w];
            optimize4<NEST>(s, wv, mv, nlr, mu, wd);
            store_keep(wb, bo, wv);
            store_keep(mb, bo, mv);
        }
        // ragged end of a key: fewer than 4 elements, one per lane
        const uint32_t rem = uint32_t(sg.count) & 3u;
        if (threadIdx.x < rem) {
            const int64_t i = int64_t(nvec) * 4 + threadIdx.x;
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
__global__ __launch_bounds__(kMaxBlockThreads) void fused_step_any(PHUB_KERNEL_ARGS) {
    const int64_t sb = group_begin[blockIdx.x];
    const int64_t se = group_begin[blockIdx.x + 1];
    const int n = num_workers;
    const float nlr = -lr;
    for (int64_t si = sb; si < se; ++si) {
        const DevSegment sg = segments[si];
        const float* const* kp = grads + int64_t(sg.key) * n;
        float* wb = weights + sg.arena_offset;
        float* mb = moments + sg.arena_offset;
        const uint32_t nvec = uint32_t(sg.count) >> 2;
        for (uint32_t v = threadIdx.x; v < nvec; v += blockDim.x) {
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
            f4 wv = load_keep(wb, bo);
            f4 mv = load_keep(mb, bo);
            optimize4<NEST>(s, wv, mv, nlr, mu, wd);
            store_keep(wb, bo, wv);
            store_keep(mb, bo, mv);
        }
        const uint32_t rem = uint32_t(sg.count) & 3u;
        if (threadIdx.x < rem) {
            const int64_t i = int64_t(nvec) * 4 + threadIdx.x;
            float s = load1(kp[0] + sg.offset, i);
            for (int w = 1; w < n; ++w) s = s + load1(kp[w] + sg.offset, i);
            float wv = load1(wb, i), mv = load1(mb, i);
            optimize<NEST>(s, wv, mv, nlr, mu, wd);
            store1(wb, i, wv);
            store1(mb, i, mv);
        }
    }
}

#define PHUB_LAUNCH_ARGS                                                                       \
    p.segments, p.group_begin, p.grads, p.weights, p.moments, p.lr, p.mu, p.wd, p.num_workers

template <int NW>
hipError_t launch_n(const StepParams& p, bool nesterov, int grid, int block, hipStream_t stream) {
    if (nesterov)
        hipLaunchKernelGGL((fused_step_fixed<NW, true>), dim3(grid), dim3(block), 0, stream,
                           PHUB_LAUNCH_ARGS);
    else
        hipLaunchKernelGGL((fused_step_fixed<NW, false>), dim3(grid), dim3(block), 0, stream,
                           PHUB_LAUNCH_ARGS);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_fused_step(const StepParams& p, bool nesterov, int grid, int block,
                             hipStream_t stream) {
    switch (p.num_workers) {
        case 1: return launch_n<1>(p, nesterov, grid, block, stream);
        case 2: return launch_n<2>(p, nesterov, grid, block, stream);
        case 3: return launch_n<3>(p, nesterov, grid, block, stream);
        case 4: return launch_n<4>(p, nesterov, grid, block, stream);
        case 5: return launch_n<5>(p, nesterov, grid, block, stream);
        case 6: return launch_n<6>(p, nesterov, grid, block, stream);
        case 7: return launch_n<7>(p, nesterov, grid, block, stream);
        case 8: return launch_n<8>(p, nesterov, grid, block, stream);
        case 9: return launch_n<9>(p, nesterov, grid, block, stream);
        case 10: return launch_n<10>(p, nesterov, grid, block, stream);
        case 11: return launch_n<11>(p, nesterov, grid, block, stream);
        case 12: return launch_n<12>(p, nesterov, grid, block, stream);
        case 13: return launch_n<13>(p, nesterov, grid, block, stream);
        case 14: return launch_n<14>(p, nesterov, grid, block, stream);
        case 15: return launch_n<15>(p, nesterov, grid, block, stream);
        case 16: return launch_n<16>(p, nesterov, grid, block, stream);
        default:
            if (nesterov)
                hipLaunchKernelGGL((fused_step_any<true>), dim3(grid), dim3(block), 0, stream,
                               PHUB_LAUNCH_ARGS);
            else
                hipLaunchKernelGGL((fused_step_any<false>), dim3(grid), dim3(block), 0, stream,
                               PHUB_LAUNCH_ARGS);
            return hipGetLastError();
    }
}

}  // namespace phub
