// Device-side data of the exchange step and its launcher.
#pragma once

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdint>
#include <string>
#include <vector>

#include "plan.hpp"

namespace phub {

#ifndef PHUB_BLOCK_THREADS
#define PHUB_BLOCK_THREADS 256
#endif

// Threads per workgroup; the kernels are compiled for exactly this size so
// that the register budget per lane follows from it.
constexpr int kBlockThreads = PHUB_BLOCK_THREADS;
static_assert(kBlockThreads >= 64 && kBlockThreads <= 1024 && kBlockThreads % 64 == 0,
              "block size must be a multiple of the wave size");

// A tile is what one wave moves per iteration of its hot loop: 4 float4 per
// lane of each array, i.e. 1024 elements (4 KB) of every gradient, of W and
// of M.
constexpr int kVecPerLane = 4;
constexpr int64_t kTileElems = 64 * 4 * kVecPerLane;

// Largest key the device descriptors address: a tile's float4 index is 32
// bits.
constexpr int64_t kMaxDeviceKeyElems = int64_t(1) << 34;

// One full tile (16 bytes): kTileElems elements of a key starting at
// element 4 * vec (keys therefore hold fewer than kMaxDeviceKeyElems).
struct DevTile {
    int64_t arena_offset;  // index of the tile's first element in the W and M arenas
    int32_t key;           // the key's row in the gradient pointer table
    uint32_t vec;          // index of the tile's first float4 within the key
};
static_assert(sizeof(DevTile) == 16, "DevTile layout");

// The rest of a segment after its full tiles (32 bytes): fewer than
// kTileElems elements, possibly with a ragged end of up to 3 elements.
struct DevRem {
    int64_t arena_offset;  // index of the first element in the W and M arenas
    int64_t offset;        // index of the first element within the key (multiple of 4)
    int32_t key;           // the key's row in the gradient pointer table
    int32_t count;         // elements, 1 .. kTileElems - 1
    int64_t pad;
};
static_assert(sizeof(DevRem) == 32, "DevRem layout");

// The start of one wave's work in a launch of the fixed-N kernels (128
// bytes), read with one burst of scalar loads at the start of the launch:
// the wave's four bins (as offsets into the tile and remainder tables) and
// the first descriptor of each (zeros where the bin is empty).  Without it
// the first data load of a wave waits for the bin offsets, then for the
// first descriptor, then for the descriptor's pointer row; with it, only
// for the pointer row (one trip to memory less; about 0.4 us of a small
// job's launch on MI355X).
struct WaveHead {
    int32_t tiles_resident[2];   // [begin, end) into the tile table
    int32_t tiles_streamed[2];
    int32_t rems_resident[2];    // [begin, end) into the remainder table
    int32_t rems_streamed[2];
    DevTile first_resident;
    DevTile first_streamed;
    DevRem first_rem_resident;
    DevRem first_rem_streamed;
};
static_assert(sizeof(WaveHead) == 128, "WaveHead layout");

// Optimizers of the fused pass (pluggable, paper section 3.2.2).
enum OptKind : int {
    kOptMomentum = 0,  // SGD with momentum (state W, M)
    kOptNesterov = 1,  // SGD with Nesterov momentum (state W, M)
    kOptSgd = 2,       // plain SGD (state W)
    kOptAdam = 3,      // Adam with bias correction (state W, M, V)
};

// Worker counts 1 .. kMaxFixedWorkers, and 20, 24 and 32, have a
// compile-time kernel each; other counts take the any-N kernel.
constexpr int kMaxFixedWorkers = 16;

constexpr bool has_fixed_kernel(int num_workers) {
    return (num_workers >= 1 && num_workers <= kMaxFixedWorkers) || num_workers == 20 ||
           num_workers == 24 || num_workers == 32;
}

// Whether a fixed-N fused pass (without pushpull) writes the streamed bin's
// state back in bursts through LDS, in the chip-wide write phases below:
// from 6 workers for momentum and plain SGD, from 14 for Adam (measured on
// MI355X with nothing cached, against piece-by-piece write-back: momentum
// with 6-16 workers +0.7 to +4.5 points, plain SGD with 6-16 up to +0.8,
// Adam with 14 and 16 +2.7 and +1.7; with fewer workers 1.5 to 15 points
// slower).  num_states: 1 plain SGD, 2 momentum, 3 Adam.
constexpr int kBurstMinWorkers[3] = {6, 6, 14};

constexpr bool burst_write_back(int num_workers, int num_states) {
    return has_fixed_kernel(num_workers) && num_states >= 1 && num_states <= 3 &&
           num_workers >= kBurstMinWorkers[num_states - 1];
}

// The burst write-back's stash: LDS per wave (the compute unit's 160 KB
// over its four waves), and how many tiles of state it holds for a job
// with num_states state arrays (a tile is 4 KB per array and wave).
constexpr int kStashBytesPerWave = 40 * 1024;
constexpr int stash_tiles(int num_states) {
    return num_states >= 1 ? kStashBytesPerWave / (num_states * 4 * 1024) : 0;
}

// Chip-wide write phases of the burst write-back.  Every wave of every
// launch reads the same constant-rate wall clock; the clock's time is cut
// into periods, and the first part of each period (the write window) is
// when waves write back their stashed state.  A period is about as many
// tiles of a wave's reads as the stash holds besides the tile in progress
// (4 of momentum's 5, 9 of plain SGD's 10, 2 of Adam's 3), at
// kWritePeriodNsPerStreamTile per element stream of a tile (N + 2 S
// streams: gradients, state read, state written) and stashed tile; the
// window is about one tile (kWriteWindowNs).  The host converts both to
// clock ticks.  Swept on MI355X with momentum at 8 and 16 workers: 550-700
// ns per stream and tile and 6-10 us windows lie within a point of each
// other, 800 ns with a 15.4 us window 1-2.6 points below; a period of
// four tiles for every optimizer measured 1.5-2.7 points below this for
// plain SGD at 8 workers and 1.8 below for Adam at 16.
constexpr int64_t kWritePeriodNsPerStreamTile = 650;
constexpr int64_t kWriteWindowNs = 8000;

// Write-phase period and window of the burst write-back in ticks of a wall
// clock running at clock_khz, for a job with num_workers gradients and
// num_states state arrays.
inline void write_phase_ticks(int num_workers, int num_states, int64_t clock_khz,
                              uint32_t* period, uint32_t* window) {
    const int64_t streams = num_workers + 2 * int64_t(num_states);
    const int64_t tiles = std::max<int64_t>(stash_tiles(num_states) - 1, 1);
    const int64_t p = kWritePeriodNsPerStreamTile * streams * tiles * clock_khz / 1000000;
    const int64_t w = kWriteWindowNs * clock_khz / 1000000;
    *period = uint32_t(std::min<int64_t>(std::max<int64_t>(p, 2), INT32_MAX));
    *window = uint32_t(std::min<int64_t>(std::max<int64_t>(w, 1), *period - 1));
}

// Counters of the dynamic schedule.  The waves of workgroup g take from
// counter g mod C (C = the launch's counters: kMaxPoolCounters, or fewer
// for a grid of fewer workgroups; one per XCD of MI355X, whose workgroups
// go to the XCDs in turn), counter c serving pool tiles c, c + C, c + 2 C,
// ...  Each readiness group has its own counters, each on its own 256-byte
// line, never reset: every launch of the group adds the same amount to
// counter c (the tiles it serves plus the waves that take from it, each
// wave taking once past its tiles), so the counter's value at the start of
// the group's launch number L (from 0) is L times that amount.
constexpr int kMaxPoolCounters = 8;
constexpr int kPoolCounterStride = 32;  // unsigned long long: 256 bytes

// Counters a launch of `grid` workgroups uses.
constexpr int pool_counter_count(int64_t grid) {
    return grid < kMaxPoolCounters ? int(grid) : kMaxPoolCounters;
}

// Tiles of a pool of `count` tiles that counter c of C serves.
constexpr int64_t pool_counter_tiles(int64_t count, int c, int counters) {
    return count > c ? (count - c + counters - 1) / counters : 0;
}

// Workgroups of a grid of `grid` that take from counter c of C.
constexpr int64_t pool_counter_groups(int64_t grid, int c, int counters) {
    return grid > c ? (grid - c + counters - 1) / counters : 0;
}

// Scalars of one launch.  For Adam, c1 = 1 - b1, c2 = 1 - b2 and the
// step's bias corrections k1 = lr / (1 - b1^t), k2 = 1 / (1 - b2^t) are
// computed on the host in double and rounded to fp32 once.
struct OptArgs {
    float nlr;  // -lr
    float mu;
    float wd;
    float b1, b2, c1, c2, k1, k2, eps;
    // burst write-back (see kWritePeriodNsPerStreamTile): the write phases'
    // period and window in ticks of the device's wall clock
    uint32_t wb_period;
    uint32_t wb_window;
};

// The schedule of one launch has two bins per wave.  With
// bins = grid * kBlockThreads / 64 waves, the bin tables hold 2 * bins + 1
// offsets: wave w's cache-resident bin is [begin[w], begin[w+1]) (its state
// stays in the memory-side cache between steps: cache-allocating loads and
// stores), its streamed bin [begin[bins+w], begin[bins+w+1]) (state read
// and written non-temporally).  The fused kernels walk the streamed bin
// first.
struct StepParams {
    const DevTile* tiles;         // grouped by bin
    const int32_t* tile_begin;    // 2 * bins + 1 offsets into tiles
    const DevRem* rems;           // grouped by bin
    const int32_t* rem_begin;     // 2 * bins + 1 offsets into rems
    const WaveHead* heads;        // one per wave (the fixed-N kernels read these, not the offsets)
    const float* const* grads;    // [row * num_workers + worker], 16-byte aligned
    float* const* outs;           // same layout: model buffers that receive w' (pushpull), or null
    float* merge;                 // unfused ablation: sum buffer laid out like W, or null (fused)
    float* weights;               // W arena
    float* moments;               // M arena (momentum, Adam's first moment), or null
    float* second;                // V arena (Adam's second moment), or null
    OptArgs opt;
    int num_workers;
    // dynamic schedule: the launch's streamed full tiles as one pool (the
    // streamed bins then hold only remainders), taken by the waves through
    // pool counters (see PoolCounters).  pool_count 0: none.
    const DevTile* pool;
    int32_t pool_count;
    unsigned long long* pool_counters;  // the group's counters, kPoolCounterStride apart
    uint64_t pool_launch;               // the group's launches before this one
};

// Whether the fused kernel for num_workers and optimizer (an OptKind) can
// walk a tile pool (the fixed-N kernels; not the any-N kernel).
bool takes_tile_pool(int num_workers, int optimizer);

// A part of a key scheduled on its own (a job's cache-resident or
// streamed part of the key): the key's row in the gradient pointer table,
// the part's first element within the key (a multiple of 4) and its
// element count.
struct VirtualKey {
    int row;
    int64_t base;
    int64_t elems;
};

// Device form of schedules: full tiles and remainders grouped by bin, and
// offsets into them (each bin ends where the next begins).
struct DeviceTables {
    std::vector<DevTile> tiles;
    std::vector<DevRem> rems;
    std::vector<int32_t> tile_begin;
    std::vector<int32_t> rem_begin;
};

// Appends the device form of `plan` (built over `vkeys`) to `out`: for each
// of its first `bins` bins, the bin's segments in order, each cut into its
// full tiles and at most one remainder, then the end offsets of the bin.
// row_arena_offset[row] is the arena element offset of the key on that
// row.  Returns the number of elements scheduled, or -1 (nothing usable
// appended) when a table outgrows 32-bit offsets.
int64_t append_device_tables(const Plan& plan, const std::vector<VirtualKey>& vkeys,
                             const std::vector<int64_t>& row_arena_offset, int bins,
                             DeviceTables* out);

// Sets the calling thread's error message (phub_last_error) and returns code.
int report_error(int code, const std::string& message);

// Appends the WaveHead of each of `bins` waves of one launch whose block of
// 2 * bins + 1 bin offsets starts at `block` in dt.tile_begin and
// dt.rem_begin (the resident bins, then the streamed ones).
void append_wave_heads(const DeviceTables& dt, size_t block, int bins,
                       std::vector<WaveHead>* out);

// Enqueues one fused aggregate + optimize pass over the whole schedule
// (and, when p.outs is set, writes the updated weights into every worker's
// model buffer in the same pass; when p.merge is set, runs the unfused
// two-pass ablation instead): `grid` workgroups of kBlockThreads threads,
// two bins per wave as described above.  `optimizer` is an OptKind.
hipError_t launch_fused_step(const StepParams& p, int optimizer, int grid, hipStream_t stream);

}  // namespace phub
