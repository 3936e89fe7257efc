// Native checks of the chunk schedule (paper section 3.2.3: keys cut into
// chunks; section 3.2.4: chunks mapped to cores by a balanced partition
// fixed at initialisation), built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_sanitizers.py.
//
// argv[1] names a file of key lists, one per line: "N n_0 n_1 ...".  For
// each list, both schedules, several bin counts, chunk sizes and item
// minimums: every key's elements are covered by the segments exactly once,
// segments are non-empty and start on a 16-byte boundary of their key, bin
// offsets are monotone and end at the segment count, bin costs add up, and
// the LPT makespan stays within the list-scheduling bound (average load plus
// the largest item).  Then argument errors.  Exit status 0 when all hold.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <fstream>
#include <sstream>
#include <string>
#include <vector>

#include "plan.hpp"

static int failures = 0;

static void check(bool ok, const std::string& what) {
    if (!ok) {
        std::fprintf(stderr, "FAILED: %s\n", what.c_str());
        ++failures;
    }
}

static void check_plan(int n, const std::vector<int64_t>& keys, int64_t chunk, int schedule,
                       int bins, int min_items, const std::string& tag) {
    phub::Plan plan;
    const std::string err = phub::build_plan(n, int(keys.size()), keys.data(), chunk, schedule,
                                             bins, min_items, &plan);
    check(err.empty(), tag + ": " + err);
    if (!err.empty()) return;
    const int used = plan.bins_used();
    check(used >= 0 && used <= bins, tag + ": bins used");
    check(plan.bin_begin.front() == 0 && plan.bin_begin.back() == int64_t(plan.segments.size()),
          tag + ": bin offsets span the segments");
    for (int b = 0; b < used; ++b) check(plan.bin_begin[b] <= plan.bin_begin[b + 1], tag + ": monotone");
    // coverage: per key, sorted segments tile [0, n_k) exactly
    std::vector<std::vector<std::pair<int64_t, int64_t>>> per_key(keys.size());
    for (const phub::PlanSegment& s : plan.segments) {
        const bool in_range = s.key >= 0 && size_t(s.key) < keys.size();
        check(in_range, tag + ": segment key in range");
        if (!in_range) continue;
        check(s.count >= 1, tag + ": non-empty segment");
        check(s.offset % 4 == 0, tag + ": 16-byte aligned segment start");
        per_key[s.key].push_back({s.offset, s.count});
    }
    for (size_t k = 0; k < keys.size(); ++k) {
        auto& v = per_key[k];
        std::sort(v.begin(), v.end());
        int64_t at = 0;
        for (auto& [off, cnt] : v) {
            check(off == at, tag + ": key " + std::to_string(k) + " covered once, in order");
            at = off + cnt;
        }
        check(at == keys[k], tag + ": key " + std::to_string(k) + " covered to its end");
    }
    if (!plan.bin_cost.empty()) {
        int64_t total = 0, most = 0;
        for (int64_t c : plan.bin_cost) {
            total += c;
            most = std::max(most, c);
        }
        int64_t want = 0;
        for (const phub::PlanSegment& s : plan.segments)
            want += int64_t(n + 4) * 4 * s.count + phub::kSegmentCostBytes;
        check(total == want, tag + ": bin costs add up");
        if (schedule == phub::kScheduleLpt && used > 0) {
            // list scheduling: makespan <= average + largest item (an item is at most one chunk
            // plus the bundling overhead of its segments)
            const int64_t item = int64_t(n + 4) * 4 * std::max<int64_t>(plan.item_elems, 1) +
                                 phub::kSegmentCostBytes * 64;
            check(most <= total / bins + item, tag + ": LPT within the list-scheduling bound");
        }
    }
}

int main(int argc, char** argv) {
    if (argc < 2) {
        std::fprintf(stderr, "usage: plan_check key_lists.txt\n");
        return 2;
    }
    std::ifstream in(argv[1]);
    std::string line;
    int lists = 0;
    while (std::getline(in, line)) {
        std::istringstream ss(line);
        int n = 0;
        if (!(ss >> n)) continue;
        std::vector<int64_t> keys;
        for (int64_t x; ss >> x;) keys.push_back(x);
        ++lists;
        int64_t total = 0;
        for (int64_t x : keys) total += x;
        // 16-byte chunks only on small lists: on 100 M elements they make tens of
        // millions of items
        const int64_t smallest = total <= (int64_t(1) << 20) ? 16 : 32768;
        for (int schedule : {phub::kScheduleSplit, phub::kScheduleLpt})
            for (int bins : {1, 7, 1024})
                for (int64_t chunk : {smallest, int64_t(32768), int64_t(4) << 20}) {
                    const int min_items = schedule == phub::kScheduleLpt ? 128 * bins : 0;
                    check_plan(n, keys, chunk, schedule, bins, min_items,
                               "list " + std::to_string(lists) + " schedule " +
                                   std::to_string(schedule) + " bins " + std::to_string(bins) +
                                   " chunk " + std::to_string(chunk));
                }
    }
    check(lists > 0, "read some key lists");
    // argument errors
    phub::Plan plan;
    const std::vector<int64_t> ok = {4, 4};
    const std::vector<int64_t> neg = {4, -1};
    check(!phub::build_plan(0, 2, ok.data(), 32768, phub::kScheduleLpt, 4, 0, &plan).empty(), "N = 0");
    check(!phub::build_plan(2, 2, ok.data(), 20, phub::kScheduleLpt, 4, 0, &plan).empty(), "chunk 20");
    check(!phub::build_plan(2, 2, neg.data(), 32768, phub::kScheduleLpt, 4, 0, &plan).empty(),
          "negative key");
    check(!phub::build_plan(2, 2, ok.data(), 32768, 7, 4, 0, &plan).empty(), "unknown schedule");
    check(!phub::build_plan(2, 2, ok.data(), 32768, phub::kScheduleLpt, 0, 0, &plan).empty(), "0 bins");
    if (failures) std::fprintf(stderr, "%d checks failed\n", failures);
    else std::printf("plan checks passed over %d key lists\n", lists);
    return failures ? 1 : 0;
}
