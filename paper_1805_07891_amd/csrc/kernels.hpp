// Device-side data of the exchange step and its launcher.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

namespace phub {

// Upper bound on threads per workgroup the kernels are compiled for.
constexpr int kMaxBlockThreads = 1024;

// One scheduled segment as the kernel reads it (32 bytes).
struct DevSegment {
    int64_t arena_offset;  // first element's index in the W and M arenas
    int64_t offset;        // first element's index within the key
    int32_t key;
    int32_t count;         // elements, >= 1
    int64_t pad;
};
static_assert(sizeof(DevSegment) == 32, "DevSegment layout");

struct StepParams {
    const DevSegment* segments;   // grouped by workgroup
    const int64_t* group_begin;   // workgroup g owns [group_begin[g], group_begin[g+1])
    const float* const* grads;    // [key * num_workers + worker], 16-byte aligned
    float* weights;               // W arena
    float* moments;               // M arena
    float lr;
    float mu;
    float wd;
    int num_workers;
};

// Enqueues one fused aggregate + optimize pass over the whole schedule.
hipError_t launch_fused_step(const StepParams& p, bool nesterov, int grid, int block,
                             hipStream_t stream);

}  // namespace phub
