// Bandwidth probe: a read-only, non-temporal stream over a set of device
// buffers, timed beside the exchange step to give the measured HBM read
// ceiling of the same buffers on the same device in the same run.  It does
// none of the step's arithmetic; the only result is a per-wave value that is
// stored only if it equals a caller-chosen sentinel, so that the loads
// cannot be removed.
//
// Layout: one workgroup of 256 threads per compute unit; each wave reads
// tiles of 2048 elements (8 KB: every lane holds 8 float4 loads in flight),
// tile t of stream s at wave (s * tiles + t) mod waves.
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
    if (!streams || nstreams < 1 || nstreams > kMaxStreams || elems_each < 0 ||
        elems_each % kTileElems != 0 || grid < 1 || !sink)
        return -1;
    Streams s;
    for (int i = 0; i < nstreams; ++i) {
        if (!streams[i] || reinterpret_cast<uintptr_t>(streams[i]) % 16 != 0) return -1;
        s.p[i] = streams[i];
    }
    for (int i = nstreams; i < kMaxStreams; ++i) s.p[i] = nullptr;
    hipLaunchKernelGGL(probe_read, dim3(grid), dim3(kThreads), 0, (hipStream_t)hip_stream, s,
                       nstreams, elems_each / kTileElems, sentinel, sink);
    return int(hipGetLastError());
}

int phub_probe_tile_elems(void) { return int(kTileElems); }

}  // extern "C"
