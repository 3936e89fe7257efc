// Device-side data of the exchange step and its launcher.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

namespace phub {

#ifndef PHUB_BLOCK_THREADS
#define PHUB_BLOCK_THREADS 256
#endif

// Threads per workgroup; the kernels are compiled for exactly this size so
// that the register budget per lane follows from it.
constexpr int kBlockThreads = PHUB_BLOCK_THREADS;
static_assert(kBlockThreads >= 64 && kBlockThreads <= 1024 && kBlockThreads % 64 == 0,
              "block size must be a multiple of the wave size");

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
    const DevSegment* segments;   // grouped by bin (one bin per wave)
    const int64_t* bin_begin;     // wave w owns [bin_begin[w], bin_begin[w+1]); one entry per
                                  // wave of the grid, plus one
    const float* const* grads;    // [key * num_workers + worker], 16-byte aligned
    float* weights;               // W arena
    float* moments;               // M arena
    float lr;
    float mu;
    float wd;
    int num_workers;
    int64_t resident_elems;  // W/M elements [0, resident_elems) use cache-allocating accesses
};

// Enqueues one fused aggregate + optimize pass over the whole schedule:
// `grid` workgroups of kBlockThreads threads.
hipError_t launch_fused_step(const StepParams& p, bool nesterov, int grid, hipStream_t stream);

}  // namespace phub
