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

// Smallest piece a chunk is cut into when the chunks alone are too few to
// give every workgroup work.
constexpr int64_t kMinSplitElems = 1024;

constexpr int kMaxWorkers = 4096;
constexpr int64_t kMaxKeyElems = int64_t(1) << 40;
constexpr int64_t kMaxChunkBytes = int64_t(1) << 30;

struct PlanSegment {
    int32_t key;
    int32_t count;
    int64_t offset;
};

struct Plan {
    int64_t item_elems = 0;               // chunk size the items were cut at
    int64_t num_items = 0;
    std::vector<PlanSegment> segments;    // grouped by workgroup
    std::vector<int64_t> group_begin;     // groups_used + 1 entries
    std::vector<int64_t> group_cost;      // groups_used entries
    int groups_used() const { return int(group_begin.size()) - 1; }
};

// Checks the job shape arguments shared by phub_init and the plan entry
// points.  Returns "" when valid, else a message.
std::string validate_shape(int num_workers, int num_keys, const int64_t* key_elems,
                           int64_t chunk_bytes);

// Computes the schedule.  Returns "" on success, else a message (and leaves
// *out unspecified).
std::string build_plan(int num_workers, int num_keys, const int64_t* key_elems,
                       int64_t chunk_bytes, int num_groups, int min_items, Plan* out);

}  // namespace phub
