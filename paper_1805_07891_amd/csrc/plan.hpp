// Host-only chunk schedule of the exchange step (no HIP dependency).
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace phub {

// Bytes-equivalent cost charged per segment on top of the bytes it moves:
// a segment costs a descriptor read and N pointer reads before its first
// element streams.
constexpr int64_t kSegmentCostBytes = 4096;

// Smallest piece the LPT schedule cuts a chunk into when the chunks alone
// are too few for the bins.
constexpr int64_t kMinSplitElems = 1024;

constexpr int kMaxWorkers = 4096;
constexpr int64_t kMaxKeyElems = int64_t(1) << 40;
constexpr int64_t kMaxChunkBytes = int64_t(1) << 30;

enum Schedule { kScheduleSplit = 0, kScheduleLpt = 1 };

struct PlanSegment {
    int32_t key;
    int32_t count;
    int64_t offset;
};

struct Plan {
    int64_t item_elems = 0;               // chunk size the items were cut at
    int64_t num_items = 0;
    std::vector<PlanSegment> segments;    // grouped by bin
    std::vector<int64_t> bin_begin;       // bins_used + 1 entries
    std::vector<int64_t> bin_cost;        // bins_used entries
    int bins_used() const { return int(bin_begin.size()) - 1; }
};

// Checks the job shape arguments shared by phub_init and the plan entry
// points.  Returns "" when valid, else a message.
std::string validate_shape(int num_workers, int num_keys, const int64_t* key_elems,
                           int64_t chunk_bytes);

// Computes the schedule.  Returns "" on success, else a message (and leaves
// *out unspecified).
//   kScheduleSplit: the keys, in order, are dealt to num_bins bins as
//     contiguous runs of equal size (to 16 bytes), each run cut into
//     segments at chunk boundaries; every bin is kept, empty or not.
//   kScheduleLpt: chunks (small keys bundled, refined while fewer than
//     min_items) assigned to at most num_bins bins largest first, each to the
//     least loaded bin; bins without work are dropped.
std::string build_plan(int num_workers, int num_keys, const int64_t* key_elems,
                       int64_t chunk_bytes, int schedule, int num_bins, int min_items,
                       Plan* out);

}  // namespace phub
