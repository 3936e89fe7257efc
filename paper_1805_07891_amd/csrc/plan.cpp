// Chunk schedule of the exchange step, computed once at job creation.
//
// Section 3.2.3 of the paper cuts every key into fixed-size chunks ("virtual
// keys", 32 KB by default) that are the unit of load balance; section 3.2.4
// fixes at initialisation which core handles which chunk, so that cores
// never synchronise, and balances the cores with a 4/3-approximate set
// partition.  Here the unit that plays a core is one wave of the fused
// kernel (it has its own scalar unit and walks its own list), and a bin is
// one wave's list of segments.  Two schedules:
//
//   split: a chunk on a GPU can be cut anywhere on a 16-byte boundary, so
//     the keys, in key order, are dealt to the bins as contiguous runs of
//     equal length (within one float4), each run cut at chunk boundaries.
//     The load is balanced exactly (the 4/3 bound is only needed for
//     indivisible chunks) and every bin streams long contiguous ranges.
//   lpt: the paper's mapping of indivisible chunks.  Keys smaller than a
//     chunk (biases, batch-norm vectors) are bundled in key order into
//     items of at most one chunk; while there are fewer items than
//     min_items the chunk is halved (down to kMinSplitElems, keeping 16-byte
//     alignment); items go largest first to the least loaded bin
//     (longest-processing-time-first, within 4/3 - 1/(3G) of the optimal
//     makespan on G bins).
//
// Neither schedule changes the result: every element is updated exactly
// once, by one lane, from the same inputs.
#include "plan.hpp"

#include <algorithm>
#include <cmath>
#include <queue>
#include <utility>

namespace phub {

std::string validate_shape(int num_workers, int num_keys, const int64_t* key_elems,
                           int64_t chunk_bytes) {
    if (num_workers < 1 || num_workers > kMaxWorkers)
        return "num_workers must be in [1, " + std::to_string(kMaxWorkers) + "], got " +
               std::to_string(num_workers);
    if (num_keys < 1) return "num_keys must be >= 1, got " + std::to_string(num_keys);
    if (!key_elems) return "key_elems is NULL";
    for (int k = 0; k < num_keys; ++k) {
        if (key_elems[k] < 0 || key_elems[k] >= kMaxKeyElems)
            return "key_elems[" + std::to_string(k) + "] = " + std::to_string(key_elems[k]) +
                   " is outside [0, 2^40)";
    }
    if (chunk_bytes < 16 || chunk_bytes % 16 != 0 || chunk_bytes > kMaxChunkBytes)
        return "chunk_bytes must be a positive multiple of 16 no larger than 2^30, got " +
               std::to_string(chunk_bytes);
    return "";
}

namespace {

struct Item {
    int64_t cost;
    int64_t first;  // index of its first segment in the creation-order list
    int32_t nseg;
};

// Cuts keys into items of at most `elems` elements: large keys into chunks,
// small keys bundled in key order.
void make_items(int num_workers, int num_keys, const int64_t* key_elems, int64_t elems,
                std::vector<PlanSegment>* segs, std::vector<Item>* items) {
    segs->clear();
    items->clear();
    const int64_t per_elem = int64_t(num_workers + 4) * 4;
    int64_t open_bundle = -1;  // item index of the bundle being filled
    int64_t bundle_elems = 0;
    for (int k = 0; k < num_keys; ++k) {
        const int64_t n = key_elems[k];
        if (n == 0) continue;
        if (n >= elems) {
            for (int64_t off = 0; off < n; off += elems) {
                const int64_t cnt = std::min(elems, n - off);
                items->push_back({cnt * per_elem + kSegmentCostBytes, int64_t(segs->size()), 1});
                segs->push_back({k, int32_t(cnt), off});
            }
        } else {
            if (open_bundle < 0 || bundle_elems + n > elems) {
                open_bundle = int64_t(items->size());
                bundle_elems = 0;
                items->push_back({0, int64_t(segs->size()), 0});
            }
            // segments of one bundle must be adjacent in `segs`; a large key
            // cut in between would break that, so restart the bundle then
            Item& it = (*items)[open_bundle];
            if (it.first + it.nseg != int64_t(segs->size())) {
                open_bundle = int64_t(items->size());
                bundle_elems = 0;
                items->push_back({0, int64_t(segs->size()), 0});
            }
            Item& cur = (*items)[open_bundle];
            cur.cost += n * per_elem + kSegmentCostBytes;
            cur.nseg += 1;
            bundle_elems += n;
            segs->push_back({k, int32_t(n), 0});
        }
    }
}

}  // namespace

namespace {

std::string build_lpt(int num_workers, int num_keys, const int64_t* key_elems,
                      int64_t chunk_bytes, int num_bins, int min_items, Plan* out) {
    std::vector<PlanSegment> segs;
    std::vector<Item> items;
    int64_t elems = chunk_bytes / 4;
    make_items(num_workers, num_keys, key_elems, elems, &segs, &items);
    while (int64_t(items.size()) < int64_t(min_items) && elems / 2 >= kMinSplitElems &&
           (elems / 2) % 4 == 0) {
        elems /= 2;
        make_items(num_workers, num_keys, key_elems, elems, &segs, &items);
    }

    out->item_elems = elems;
    out->num_items = int64_t(items.size());
    if (items.empty()) return "";  // every key is empty: nothing to launch

    // Longest processing time first: largest item first, each to the least
    // loaded bin (lowest index on ties).
    std::vector<int64_t> order(items.size());
    for (size_t i = 0; i < order.size(); ++i) order[i] = int64_t(i);
    std::stable_sort(order.begin(), order.end(),
                     [&](int64_t a, int64_t b) { return items[a].cost > items[b].cost; });
    const int bins = int(std::min<int64_t>(num_bins, int64_t(items.size())));
    using Load = std::pair<int64_t, int>;  // (cost so far, bin)
    std::priority_queue<Load, std::vector<Load>, std::greater<Load>> heap;
    for (int g = 0; g < bins; ++g) heap.push({0, g});
    std::vector<int> owner(items.size());
    std::vector<int64_t> cost(bins, 0);
    for (int64_t i : order) {
        Load l = heap.top();
        heap.pop();
        owner[i] = l.second;
        l.first += items[i].cost;
        cost[l.second] = l.first;
        heap.push(l);
    }

    // Emit each bin's segments in key, then offset, order.
    std::vector<std::vector<PlanSegment>> per(bins);
    for (size_t i = 0; i < items.size(); ++i)
        for (int32_t s = 0; s < items[i].nseg; ++s)
            per[owner[i]].push_back(segs[items[i].first + s]);
    out->segments.reserve(segs.size());
    for (int g = 0; g < bins; ++g) {
        std::sort(per[g].begin(), per[g].end(), [](const PlanSegment& a, const PlanSegment& b) {
            return a.key != b.key ? a.key < b.key : a.offset < b.offset;
        });
        out->segments.insert(out->segments.end(), per[g].begin(), per[g].end());
        out->bin_begin.push_back(int64_t(out->segments.size()));
        out->bin_cost.push_back(cost[g]);
    }
    return "";
}

std::string build_split(int num_workers, int num_keys, const int64_t* key_elems,
                        int64_t chunk_bytes, int num_bins, Plan* out) {
    // Work in float4 slots: key k has ceil(n_k / 4) of them, the last one
    // possibly partial (the key's ragged end).
    const int64_t chunk_vecs = chunk_bytes / 16;
    const int64_t per_elem = int64_t(num_workers + 4) * 4;
    int64_t total = 0;
    for (int k = 0; k < num_keys; ++k) total += (key_elems[k] + 3) / 4;
    out->item_elems = chunk_bytes / 4;
    int k = 0;
    int64_t key_start = 0;  // first slot of key k
    int64_t items = 0;
    for (int b = 0; b < num_bins; ++b) {
        const int64_t lo = int64_t((__int128)total * b / num_bins);
        const int64_t hi = int64_t((__int128)total * (b + 1) / num_bins);
        int64_t cost = 0;
        int64_t pos = lo;
        while (pos < hi) {
            int64_t kv = (key_elems[k] + 3) / 4;
            while (key_start + kv <= pos) {  // skip keys that end before pos
                key_start += kv;
                ++k;
                kv = (key_elems[k] + 3) / 4;
            }
            const int64_t a = pos - key_start;                       // slot within key
            const int64_t b_end = std::min(hi, key_start + kv) - key_start;
            const int64_t next_chunk = (a / chunk_vecs + 1) * chunk_vecs;
            const int64_t e = std::min(b_end, next_chunk);
            const int64_t off = 4 * a;
            const int64_t cnt = std::min(4 * e, key_elems[k]) - off;
            out->segments.push_back({k, int32_t(cnt), off});
            cost += cnt * per_elem + kSegmentCostBytes;
            ++items;
            pos = key_start + e;
        }
        out->bin_begin.push_back(int64_t(out->segments.size()));
        out->bin_cost.push_back(cost);
    }
    out->num_items = items;
    return "";
}

}  // namespace

std::string build_plan(int num_workers, int num_keys, const int64_t* key_elems,
                       int64_t chunk_bytes, int schedule, int num_bins, int min_items,
                       Plan* out) {
    std::string err = validate_shape(num_workers, num_keys, key_elems, chunk_bytes);
    if (!err.empty()) return err;
    if (num_bins < 1) return "num_bins must be >= 1, got " + std::to_string(num_bins);
    if (min_items < 0) return "min_items must be >= 0, got " + std::to_string(min_items);
    if (schedule != kScheduleSplit && schedule != kScheduleLpt)
        return "unknown schedule " + std::to_string(schedule);
    if (!out) return "plan output is NULL";
    out->segments.clear();
    out->bin_begin.assign(1, 0);
    out->bin_cost.clear();
    out->item_elems = 0;
    out->num_items = 0;
    if (schedule == kScheduleLpt)
        return build_lpt(num_workers, num_keys, key_elems, chunk_bytes, num_bins, min_items, out);
    return build_split(num_workers, num_keys, key_elems, chunk_bytes, num_bins, out);
}

}  // namespace phub
