// Bandwidth probes, timed beside the exchange step to give measured HBM
// ceilings of the same buffers on the same device in the same run.  They do
// none of the step's arithmetic:
//   - read: a read-only non-temporal stream over a set of buffers; the only
//     result is a per-wave value stored only if it equals a caller-chosen
//     sentinel, so that the loads cannot be removed;
//   - write: a write-only non-temporal stream of a constant;
//   - mixed: the step's traffic without its arithmetic: some buffers read
//     only, others read and written back in place (the values read), tile by
//     tile, each tile written back as soon as it is read (a plain mix of
//     read and write streams, with no timing of the writes).
//
// Layout: one workgroup of 256 threads per compute unit; each wave takes
// tiles of 2048 elements (8 KB per stream: every lane holds 8 float4 loads
// in flight), tile t (of stream s, for read and write) at wave
// (s * tiles + t) mod waves.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "phub_probe.h"

typedef float f4 __attribute__((ext_vector_type(4)));

#define PROBE_GLOBAL __attribute__((address_space(1)))

namespace {

constexpr int kMaxStreams = 64;
constexpr int kThreads = 256;
constexpr int kPieces = 8;                    // float4 per lane per tile
constexpr int64_t kTileElems = 64 * 4 * kPieces;

struct Streams {
    const float* p[kMaxStreams];
};

__global__ __launch_bounds__(kThreads) void probe_read(Streams s, int nstreams, int64_t tiles,
                                                       float sentinel, float* sink) {
    const uint32_t waves = gridDim.x * (kThreads / 64);
    const uint32_t wave =
        __builtin_amdgcn_readfirstlane(blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6));
    const uint32_t lane = threadIdx.x & 63u;
    f4 acc = 0.0f;
    const int64_t total = tiles * nstreams;
    for (int64_t i = wave; i < total; i += waves) {
        const int sid = int(i / tiles);
        const int64_t t = i - int64_t(sid) * tiles;
        const PROBE_GLOBAL f4* b =
            (const PROBE_GLOBAL f4*)(s.p[sid]) + t * (kTileElems / 4) + lane;
        f4 v[kPieces];
#pragma unroll
        for (int u = 0; u < kPieces; ++u) v[u] = __builtin_nontemporal_load(b + u * 64);
#pragma unroll
        for (int u = 0; u < kPieces; ++u) acc += v[u];
    }
    const float r = acc.x + acc.y + acc.z + acc.w;
    if (r == sentinel) sink[blockIdx.x * kThreads + threadIdx.x] = r;
}

__global__ __launch_bounds__(kThreads) void probe_write(Streams s, int nstreams, int64_t tiles,
                                                        float value) {
    const uint32_t waves = gridDim.x * (kThreads / 64);
    const uint32_t wave =
        __builtin_amdgcn_readfirstlane(blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6));
    const uint32_t lane = threadIdx.x & 63u;
    const f4 v = value;
    const int64_t total = tiles * nstreams;
    for (int64_t i = wave; i < total; i += waves) {
        const int sid = int(i / tiles);
        const int64_t t = i - int64_t(sid) * tiles;
        PROBE_GLOBAL f4* b = (PROBE_GLOBAL f4*)(s.p[sid]) + t * (kTileElems / 4) + lane;
#pragma unroll
        for (int u = 0; u < kPieces; ++u) __builtin_nontemporal_store(v, b + u * 64);
    }
}

// Streams [0, nread) are read; streams [nread, nread + nrw) are read and
// written back.  Tile t of every stream is handled by wave t mod waves.
__global__ __launch_bounds__(kThreads) void probe_mixed(Streams s, int nread, int nrw,
                                                        int64_t tiles, float sentinel,
                                                        float* sink) {
    const uint32_t waves = gridDim.x * (kThreads / 64);
    const uint32_t wave =
        __builtin_amdgcn_readfirstlane(blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6));
    const uint32_t lane = threadIdx.x & 63u;
    f4 acc = 0.0f;
    for (int64_t t = wave; t < tiles; t += waves) {
        const int64_t base = t * (kTileElems / 4) + lane;
        for (int sid = 0; sid < nread + nrw; ++sid) {
            PROBE_GLOBAL f4* b = (PROBE_GLOBAL f4*)(s.p[sid]) + base;
            f4 v[kPieces];
#pragma unroll
            for (int u = 0; u < kPieces; ++u) v[u] = __builtin_nontemporal_load(b + u * 64);
            if (sid < nread) {
#pragma unroll
                for (int u = 0; u < kPieces; ++u) acc += v[u];
            } else {
                // hide from the compiler that the values are unchanged, or it
                // drops the stores (and then the loads) as no-ops
#pragma unroll
                for (int u = 0; u < kPieces; ++u) asm volatile("" : "+v"(v[u]));
#pragma unroll
                for (int u = 0; u < kPieces; ++u) __builtin_nontemporal_store(v[u], b + u * 64);
            }
        }
    }
    const float r = acc.x + acc.y + acc.z + acc.w;
    if (r == sentinel) sink[blockIdx.x * kThreads + threadIdx.x] = r;
}

bool load_streams(const float* const* streams, int n, Streams* s) {
    if (!streams || n < 1 || n > kMaxStreams) return false;
    for (int i = 0; i < n; ++i) {
        if (!streams[i] || reinterpret_cast<uintptr_t>(streams[i]) % 16 != 0) return false;
        s->p[i] = streams[i];
    }
    for (int i = n; i < kMaxStreams; ++i) s->p[i] = nullptr;
    return true;
}

}  // namespace

extern "C" {

// Reads elems_each floats (a multiple of 2048; each buffer 16-byte aligned)
// from each of nstreams device buffers (host array of device pointers,
// 1..64 entries), once, on hip_stream, with `grid` workgroups of 256
// threads.  sink: device buffer of grid * 256 floats, written only where a
// lane's sum equals `sentinel`.  Returns 0, -1 for bad arguments, or the HIP
// error code of the launch.
int phub_probe_read(const float* const* streams, int nstreams, int64_t elems_each, int grid,
                    float sentinel, float* sink, void* hip_stream) {
    Streams s;
    if (!load_streams(streams, nstreams, &s) || elems_each < 0 || elems_each % kTileElems != 0 ||
        grid < 1 || !sink)
        return -1;
    hipLaunchKernelGGL(probe_read, dim3(grid), dim3(kThreads), 0, (hipStream_t)hip_stream, s,
                       nstreams, elems_each / kTileElems, sentinel, sink);
    return int(hipGetLastError());
}

int phub_probe_write(float* const* streams, int nstreams, int64_t elems_each, int grid,
                     float value, void* hip_stream) {
    Streams s;
    if (!load_streams(const_cast<const float* const*>(streams), nstreams, &s) || elems_each < 0 ||
        elems_each % kTileElems != 0 || grid < 1)
        return -1;
    hipLaunchKernelGGL(probe_write, dim3(grid), dim3(kThreads), 0, (hipStream_t)hip_stream, s,
                       nstreams, elems_each / kTileElems, value);
    return int(hipGetLastError());
}

int phub_probe_mixed(const float* const* read_streams, int nread, float* const* rw_streams,
                     int nrw, int64_t elems_each, int grid, float sentinel, float* sink,
                     void* hip_stream) {
    if (nread < 0 || nrw < 0 || nread + nrw < 1 || nread + nrw > kMaxStreams ||
        elems_each < 0 || elems_each % kTileElems != 0 || grid < 1 || !sink)
        return -1;
    Streams s;
    for (int i = 0; i < kMaxStreams; ++i) s.p[i] = nullptr;
    for (int i = 0; i < nread + nrw; ++i) {
        const float* p = i < nread ? (read_streams ? read_streams[i] : nullptr)
                                   : (rw_streams ? rw_streams[i - nread] : nullptr);
        if (!p || reinterpret_cast<uintptr_t>(p) % 16 != 0) return -1;
        s.p[i] = p;
    }
    hipLaunchKernelGGL(probe_mixed, dim3(grid), dim3(kThreads), 0, (hipStream_t)hip_stream, s,
                       nread, nrw, elems_each / kTileElems, sentinel, sink);
    return int(hipGetLastError());
}

int phub_probe_tile_elems(void) { return int(kTileElems); }

}  // extern "C"
