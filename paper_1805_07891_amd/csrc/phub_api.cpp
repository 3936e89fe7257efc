// C interface of the exchange step: job state, push/step/pull, schedule.
//
// The paper's service (section 3.1) creates a job with its own namespace and
// buffers, then serves Push and Pull.  A job here owns its master weights W
// and momentum M in HBM, the schedule computed at creation (section 3.2.4),
// a device copy of the (worker, key) -> gradient pointer table, and the
// stream its work is ordered on.  A push only records a pointer (the
// zero-copy registration of section 3.2.1); a step uploads the pointer table
// if it changed and launches one fused kernel for all keys.
//
// Readiness groups (sections 3.2.2-3.2.3: PHub aggregates a chunk as soon
// as all of its pieces have arrived, overlapping reception with
// aggregation): a job may partition its keys into groups at creation.  Each
// group has its own schedule, and the fused kernel for a group is enqueued
// as soon as every worker has pushed every key of the group, after waiting
// on the device for the ready events given with the pushes.  The pointer
// table is laid out by group (keys of a group on consecutive rows), so a
// group uploads only its own rows.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "kernels.hpp"
#include "phub.h"
#include "plan.hpp"

// Workgroups per compute unit of the persistent launch.
#ifndef PHUB_GROUPS_PER_CU
#define PHUB_GROUPS_PER_CU 1
#endif
// Default cache budget per device, shared by the jobs created with the
// default option: the size of MI355X's memory-side cache (256 MiB).  A job
// takes as much of what is left as its optimizer state needs: that part of
// the state (a prefix of the arena) is read and written with the
// cache-allocating policy, so that it can stay in that cache between steps
// (the paper's cached model, section 4.5); the rest streams non-temporally
// like the gradients.
#ifndef PHUB_DEVICE_CACHE_BYTES
#define PHUB_DEVICE_CACHE_BYTES (int64_t(256) << 20)
#endif
// The LPT schedule refines chunks until there are this many items per bin
// (never below 1024 elements).  With ~1000 waves this yields one-tile items
// for every workload up to ~130 M parameters: the waves then work on
// neighbouring tiles at any moment, which keeps the window of addresses in
// flight per array compact (measured: +2.6 points on a 102 M-parameter,
// 16-worker job over two-tile items).
#ifndef PHUB_LPT_ITEMS_PER_BIN
#define PHUB_LPT_ITEMS_PER_BIN 128
#endif
constexpr int kLptItemsPerBin = PHUB_LPT_ITEMS_PER_BIN;

namespace {

constexpr int kStageSlots = 4;       // pinned staging buffers for pointer-table uploads
constexpr int kMaxWorkgroups = 1 << 16;  // largest persistent grid a job may ask for
constexpr int64_t kArenaAlign = 64;  // elements: 256-byte aligned key slices
constexpr size_t kCountersPerGroup = size_t(phub::kMaxPoolCounters) * phub::kPoolCounterStride;

thread_local std::string g_error;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_error = buf;
    return code;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(PHUB_EHIP, "%s failed: %s (%d)", what, hipGetErrorString(e), int(e));
}

std::mutex g_live_mu;
std::unordered_set<const void*> g_live;
// Bytes of the default cache budget held by live jobs, per device (under g_live_mu).
std::unordered_map<int, int64_t> g_cache_claimed;

}  // namespace

struct phub_job {
    int num_workers = 0;
    int num_keys = 0;
    std::vector<int64_t> key_elems;
    std::vector<int64_t> arena_offset;  // per key, elements
    int64_t arena_elems = 0;
    int64_t chunk_bytes = 0;
    float lr = 0, mu = 0, wd = 0;
    bool nesterov = false;
    int opt = phub::kOptNesterov;  // an OptKind
    float b1 = 0, b2 = 0, eps = 0;  // Adam
    int64_t steps_done = 0;         // completed steps (Adam's bias correction)

    int device = 0;
    int64_t wall_clock_khz = 0;  // rate of the device's constant wall clock
    hipStream_t stream = nullptr;
    bool own_stream = false;

    int schedule = phub::kScheduleLpt;
    bool dynamic = false;  // the streamed full tiles are taken from a pool (PHUB_SCHEDULE_DYNAMIC)
    int groups = 0;  // workgroups of one launch (0: no key has elements)
    int bins = 0;    // waves with a segment list (groups * waves per workgroup)
    int64_t num_segments = 0;
    int64_t num_tiles = 0;
    int64_t num_rems = 0;
    int num_states = 2;         // optimizer state arrays (W, then M and V)
    int64_t resident_elems = 0; // arena elements [0, resident_elems) keep their state
                                // in the memory-side cache between steps
    int64_t resident_bytes = 0; // state bytes of the tiles actually scheduled as resident
    int64_t cache_claim = 0;    // bytes of the device's default cache budget this job holds

    // Readiness groups.  Without groups the job has one group holding every
    // key, launched by phub_step.
    bool streaming = false;              // groups launch as soon as they are complete
    int num_rgroups = 1;
    std::vector<int> key_rgroup;         // per key
    std::vector<int> row_of_key;         // pointer-table row of each key
    std::vector<int> key_of_row;
    std::vector<int> rgroup_row_begin;   // rows of group g: [begin[g], begin[g + 1])
    std::vector<uint8_t> rgroup_work;    // the group's schedule has segments
    std::vector<int64_t> rgroup_pushed;  // (worker, key) pairs pushed this step
    std::vector<uint8_t> rgroup_launched;
    std::vector<uint8_t> rgroup_dirty;   // its rows changed since they were last uploaded
    std::vector<int64_t> rgroup_outs;    // pushpull: model buffers registered this step
    std::vector<uint8_t> rgroup_out_dirty;

    float* weights = nullptr;
    float* moments = nullptr;  // null for plain SGD
    float* second = nullptr;   // Adam's second moment, else null
    float* merge = nullptr;  // unfused ablation only: the sum, laid out like W
    phub::DevTile* d_tiles = nullptr;
    int32_t* d_tile_begin = nullptr;  // num_rgroups blocks of 2 * bins + 1 entries
    phub::DevRem* d_rems = nullptr;
    int32_t* d_rem_begin = nullptr;   // same layout
    phub::WaveHead* d_heads = nullptr;  // num_rgroups blocks of bins heads
    std::vector<int32_t> pool_begin;  // per readiness group: its tile pool in d_tiles
    std::vector<int32_t> pool_count;  // (0: the group's schedule is static)
    unsigned long long* d_counters = nullptr;  // takes from the pools: per group, never reset
    std::vector<uint64_t> pool_launches;        // per group: launches so far
    const float** d_grads = nullptr;  // [row * N + worker]
    float** d_outs = nullptr;         // same layout: pushpull model buffers

    std::vector<const float*> grads;  // host table, [row * N + worker]
    std::vector<hipEvent_t> ready;    // same layout: event to wait for (none if null)
    bool ordered_events = false;      // each worker's events are ordered on one stream
    std::vector<hipEvent_t> group_last_event;  // [group * N + worker]: last event pushed this step
    std::vector<int64_t> rgroup_events;  // pushes with a ready event this step, per group
    int64_t step_events = 0;             // the same over all groups
    int64_t step_outs = 0;               // model buffers registered this step
    std::vector<hipEvent_t> wait_events; // reused by each launch: the events it waits for
    std::vector<uint8_t> pushed;      // same layout: pushed since the last step
    int64_t num_pushed = 0;
    std::vector<float*> outs;         // same layout: pushpull model buffers of this step
    std::vector<uint8_t> has_out;

    // Pinned staging of the pointer table: one slot per step, reused after
    // kStageSlots steps once the copies that read it have run.
    const float** stage[kStageSlots] = {};
    float** stage_out[kStageSlots] = {};
    hipEvent_t stage_done[kStageSlots] = {};
    bool stage_used[kStageSlots] = {};
    int stage_slot = 0;
    bool stage_claimed = false;  // this step has waited for its slot
};

namespace {

// Makes the job's device current for the duration of a call.
class DeviceScope {
  public:
    explicit DeviceScope(int device) {
        if (hipGetDevice(&prev_) != hipSuccess) prev_ = -1;
        if (prev_ != device) ok_ = hipSetDevice(device) == hipSuccess;
    }
    ~DeviceScope() {
        int cur = -1;
        if (prev_ >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev_) (void)hipSetDevice(prev_);
    }
    bool ok() const { return ok_; }

  private:
    int prev_ = -1;
    bool ok_ = true;
};

bool is_live(const phub_job* j) {
    std::lock_guard<std::mutex> lk(g_live_mu);
    return j && g_live.count(j) != 0;
}

void release(phub_job* j) {
    if (j->d_grads) (void)hipFree(j->d_grads);
    if (j->d_outs) (void)hipFree(j->d_outs);
    if (j->d_tile_begin) (void)hipFree(j->d_tile_begin);
    if (j->d_tiles) (void)hipFree(j->d_tiles);
    if (j->d_rem_begin) (void)hipFree(j->d_rem_begin);
    if (j->d_heads) (void)hipFree(j->d_heads);
    if (j->d_rems) (void)hipFree(j->d_rems);
    if (j->d_counters) (void)hipFree(j->d_counters);
    if (j->moments) (void)hipFree(j->moments);
    if (j->second) (void)hipFree(j->second);
    if (j->merge) (void)hipFree(j->merge);
    if (j->weights) (void)hipFree(j->weights);
    for (int i = 0; i < kStageSlots; ++i) {
        if (j->stage_done[i]) (void)hipEventDestroy(j->stage_done[i]);
        if (j->stage[i]) (void)hipHostFree(j->stage[i]);
        if (j->stage_out[i]) (void)hipHostFree(j->stage_out[i]);
    }
    if (j->own_stream && j->stream) (void)hipStreamDestroy(j->stream);
    delete j;
}

int check_key(const phub_job* j, int key) {
    if (key < 0 || key >= j->num_keys)
        return fail(PHUB_EINVAL, "key %d out of range [0, %d)", key, j->num_keys);
    return PHUB_OK;
}

int check_grad(const phub_job* j, int worker, int key, const float* grad) {
    if (worker < 0 || worker >= j->num_workers)
        return fail(PHUB_EINVAL, "worker %d out of range [0, %d)", worker, j->num_workers);
    if (int rc = check_key(j, key)) return rc;
    if (!grad && j->key_elems[key] != 0)
        return fail(PHUB_EINVAL, "gradient of worker %d for key %d is NULL", worker, key);
    if (reinterpret_cast<uintptr_t>(grad) % 16 != 0)
        return fail(PHUB_EINVAL, "gradient of worker %d for key %d is not 16-byte aligned", worker,
                    key);
    if (j->streaming && j->rgroup_launched[j->key_rgroup[key]])
        return fail(PHUB_ESTATE,
                    "key %d belongs to readiness group %d, which was already launched this step",
                    key, j->key_rgroup[key]);
    return PHUB_OK;
}

// Claims the current step's pinned staging slot: waits until the copies
// that last read it (kStageSlots steps ago) have run.
int claim_stage(phub_job* j) {
    const int slot = j->stage_slot;
    if (!j->stage_claimed) {
        if (j->stage_used[slot]) {
            hipError_t e = hipEventSynchronize(j->stage_done[slot]);
            if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize (pointer staging)");
        }
        j->stage_claimed = true;
    }
    return PHUB_OK;
}

// Copies rows [r0, r1) of a host pointer table to the device, through the
// current step's staging slot, on the job's stream.
template <typename T>
int upload_range(phub_job* j, T* const* host, T** stage, T** dev, size_t r0, size_t r1) {
    if (int rc = claim_stage(j)) return rc;
    if (r1 > r0) {
        const int slot = j->stage_slot;
        std::memcpy(stage + r0, host + r0, (r1 - r0) * sizeof(T*));
        hipError_t e = hipMemcpyAsync(dev + r0, stage + r0, (r1 - r0) * sizeof(T*),
                                      hipMemcpyHostToDevice, j->stream);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (pointer table)");
        e = hipEventRecord(j->stage_done[slot], j->stream);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord (pointer staging)");
        j->stage_used[slot] = true;
    }
    return PHUB_OK;
}

// The gradient rows of group g.
int upload_rows(phub_job* j, int g) {
    const size_t n = size_t(j->num_workers);
    if (int rc = upload_range<const float>(j, j->grads.data(), j->stage[j->stage_slot], j->d_grads,
                                           size_t(j->rgroup_row_begin[g]) * n,
                                           size_t(j->rgroup_row_begin[g + 1]) * n))
        return rc;
    j->rgroup_dirty[g] = 0;
    return PHUB_OK;
}

// The model-buffer rows of group g (pushpull).
int upload_out_rows(phub_job* j, int g) {
    const size_t n = size_t(j->num_workers);
    if (int rc = upload_range<float>(j, j->outs.data(), j->stage_out[j->stage_slot], j->d_outs,
                                     size_t(j->rgroup_row_begin[g]) * n,
                                     size_t(j->rgroup_row_begin[g + 1]) * n))
        return rc;
    j->rgroup_out_dirty[g] = 0;
    return PHUB_OK;
}

// Scalars of this step's launches.  Adam's are derived from the fp32
// hyperparameters in double and rounded to fp32 once; the step number
// counts from 1 for each job.
phub::OptArgs optimizer_args(const phub_job* j) {
    phub::OptArgs o{};
    o.nlr = -j->lr;
    o.mu = j->mu;
    o.wd = j->wd;
    phub::write_phase_ticks(j->num_workers, j->num_states, j->wall_clock_khz, &o.wb_period,
                            &o.wb_window);
    if (j->opt == phub::kOptAdam) {
        const double t = double(j->steps_done + 1);
        o.b1 = j->b1;
        o.b2 = j->b2;
        o.c1 = float(1.0 - double(j->b1));
        o.c2 = float(1.0 - double(j->b2));
        o.k1 = float(double(j->lr) / (1.0 - std::pow(double(j->b1), t)));
        o.k2 = float(1.0 / (1.0 - std::pow(double(j->b2), t)));
        o.eps = j->eps;
    }
    return o;
}

// Enqueues group g: its pointer rows if they changed, a wait for every
// distinct ready event of its pushes, then the fused kernel over its
// schedule.
int launch_group(phub_job* j, int g) {
    const size_t n = size_t(j->num_workers);
    const int64_t pairs = int64_t(j->rgroup_row_begin[g + 1] - j->rgroup_row_begin[g]) * j->num_workers;
    const bool pull = j->rgroup_outs[g] > 0;
    if (pull && j->merge)
        return fail(PHUB_EINVAL, "the unfused variant does not take pushpull");
    if (pull && j->rgroup_outs[g] != pairs) {
        for (size_t i = size_t(j->rgroup_row_begin[g]) * n; i < size_t(j->rgroup_row_begin[g + 1]) * n; ++i)
            if (!j->has_out[i])
                return fail(PHUB_EINVAL,
                            "pushpull: worker %d gave no model buffer for key %d while other "
                            "pushes of its readiness group did",
                            int(i % n), j->key_of_row[i / n]);
    }
    DeviceScope ds(j->device);
    if (!ds.ok()) return fail(PHUB_EHIP, "cannot make device %d current", j->device);
    if (j->rgroup_dirty[g])
        if (int rc = upload_rows(j, g)) return rc;
    if (pull && j->rgroup_out_dirty[g])
        if (int rc = upload_out_rows(j, g)) return rc;
    // The events to wait for: every distinct one of the group's pushes, or
    // with ordered events each worker's last one; events already complete
    // need no wait.
    std::vector<hipEvent_t>& evs = j->wait_events;
    evs.clear();
    if (j->rgroup_events[g] == 0) {
        // no push of this group came with an event
    } else if (j->ordered_events) {
        for (size_t w = 0; w < n; ++w)
            if (hipEvent_t ev = j->group_last_event[size_t(g) * n + w]) evs.push_back(ev);
    } else {
        for (size_t i = size_t(j->rgroup_row_begin[g]) * n;
             i < size_t(j->rgroup_row_begin[g + 1]) * n; ++i)
            if (j->ready[i]) evs.push_back(j->ready[i]);
    }
    std::sort(evs.begin(), evs.end());
    evs.erase(std::unique(evs.begin(), evs.end()), evs.end());
    for (hipEvent_t ev : evs) {
        hipError_t e = hipEventQuery(ev);
        if (e == hipSuccess) continue;
        if (e != hipErrorNotReady) return hip_fail(e, "hipEventQuery (ready event)");
        e = hipStreamWaitEvent(j->stream, ev, 0);
        if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent (ready event)");
    }
    if (j->rgroup_work[g]) {
        phub::StepParams p{};
        p.tiles = j->d_tiles;
        p.tile_begin = j->d_tile_begin + size_t(g) * (2 * size_t(j->bins) + 1);
        p.rems = j->d_rems;
        p.rem_begin = j->d_rem_begin + size_t(g) * (2 * size_t(j->bins) + 1);
        p.heads = j->d_heads + size_t(g) * size_t(j->bins);
        p.grads = j->d_grads;
        p.outs = pull ? j->d_outs : nullptr;
        p.merge = j->merge;
        p.weights = j->weights;
        p.moments = j->moments;
        p.second = j->second;
        p.opt = optimizer_args(j);
        p.num_workers = j->num_workers;
        const int32_t pool = j->pool_count.empty() ? 0 : j->pool_count[g];
        if (pool > 0) {
            p.pool = j->d_tiles + j->pool_begin[g];
            p.pool_count = pool;
            p.pool_counters = j->d_counters + size_t(g) * kCountersPerGroup;
            p.pool_launch = j->pool_launches[g];
        }
        hipError_t e = phub::launch_fused_step(p, j->opt, j->groups, j->stream);
        if (e != hipSuccess) return hip_fail(e, "launch of the fused step kernel");
        if (pool > 0) ++j->pool_launches[g];
    }
    j->rgroup_launched[g] = 1;
    return PHUB_OK;
}

// Registers worker `worker`'s model buffer for key `key` in this step.
void record_out(phub_job* j, int worker, int key, float* out) {
    const int g = j->key_rgroup[key];
    const size_t i = size_t(j->row_of_key[key]) * j->num_workers + worker;
    if (j->outs[i] != out) {
        j->outs[i] = out;
        j->rgroup_out_dirty[g] = 1;
    }
    if (!j->has_out[i]) {
        j->has_out[i] = 1;
        ++j->rgroup_outs[g];
        ++j->step_outs;
    }
}

int check_out(const phub_job* j, int worker, int key, const float* out) {
    if (!out && j->key_elems[key] != 0)
        return fail(PHUB_EINVAL, "model buffer of worker %d for key %d is NULL", worker, key);
    if (reinterpret_cast<uintptr_t>(out) % 16 != 0)
        return fail(PHUB_EINVAL, "model buffer of worker %d for key %d is not 16-byte aligned",
                    worker, key);
    return PHUB_OK;
}

int record_push(phub_job* j, int worker, int key, const float* grad, hipEvent_t ev) {
    const int g = j->key_rgroup[key];
    if (j->streaming && j->rgroup_launched[g])  // e.g. a key repeated in one batch
        return fail(PHUB_ESTATE,
                    "key %d belongs to readiness group %d, which was already launched this step",
                    key, g);
    const size_t i = size_t(j->row_of_key[key]) * j->num_workers + worker;
    if (j->grads[i] != grad) {
        j->grads[i] = grad;
        j->rgroup_dirty[g] = 1;
    }
    j->ready[i] = ev;
    if (ev) {
        ++j->rgroup_events[g];
        ++j->step_events;
        if (j->ordered_events) j->group_last_event[size_t(g) * j->num_workers + worker] = ev;
    }
    if (!j->pushed[i]) {
        j->pushed[i] = 1;
        ++j->num_pushed;
        ++j->rgroup_pushed[g];
        const int64_t need =
            int64_t(j->rgroup_row_begin[g + 1] - j->rgroup_row_begin[g]) * j->num_workers;
        if (j->streaming && j->rgroup_pushed[g] == need) return launch_group(j, g);
    }
    return PHUB_OK;
}

}  // namespace

namespace phub {

int report_error(int code, const std::string& message) {
    g_error = message;
    return code;
}

int64_t append_device_tables(const Plan& plan, const std::vector<VirtualKey>& vkeys,
                             const std::vector<int64_t>& row_arena_offset, int bins,
                             DeviceTables* out) {
    int64_t elems = 0;
    for (int b = 0; b < bins; ++b) {
        for (int64_t i = plan.bin_begin[b]; i < plan.bin_begin[b + 1]; ++i) {
            const PlanSegment& sg = plan.segments[i];
            const VirtualKey& v = vkeys[sg.key];
            const int64_t koff = v.base + sg.offset;  // first element within the key
            const int64_t ao = row_arena_offset[v.row] + koff;
            elems += sg.count;
            const int64_t nfull = sg.count / kTileElems;
            for (int64_t t = 0; t < nfull; ++t)
                out->tiles.push_back(
                    {ao + t * kTileElems, v.row, uint32_t((koff + t * kTileElems) / 4)});
            const int64_t done = nfull * kTileElems;
            if (done < sg.count)
                out->rems.push_back({ao + done, koff + done, v.row, int32_t(sg.count - done), 0});
        }
        if (out->tiles.size() > size_t(INT32_MAX) || out->rems.size() > size_t(INT32_MAX))
            return -1;
        out->tile_begin.push_back(int32_t(out->tiles.size()));
        out->rem_begin.push_back(int32_t(out->rems.size()));
    }
    return elems;
}

void append_wave_heads(const DeviceTables& dt, size_t block, int bins,
                       std::vector<WaveHead>* out) {
    const int32_t* tb = dt.tile_begin.data() + block;
    const int32_t* rb = dt.rem_begin.data() + block;
    for (int w = 0; w < bins; ++w) {
        WaveHead h{};
        h.tiles_resident[0] = tb[w];
        h.tiles_resident[1] = tb[w + 1];
        h.tiles_streamed[0] = tb[bins + w];
        h.tiles_streamed[1] = tb[bins + w + 1];
        h.rems_resident[0] = rb[w];
        h.rems_resident[1] = rb[w + 1];
        h.rems_streamed[0] = rb[bins + w];
        h.rems_streamed[1] = rb[bins + w + 1];
        if (tb[w] < tb[w + 1]) h.first_resident = dt.tiles[size_t(tb[w])];
        if (tb[bins + w] < tb[bins + w + 1]) h.first_streamed = dt.tiles[size_t(tb[bins + w])];
        if (rb[w] < rb[w + 1]) h.first_rem_resident = dt.rems[size_t(rb[w])];
        if (rb[bins + w] < rb[bins + w + 1]) h.first_rem_streamed = dt.rems[size_t(rb[bins + w])];
        out->push_back(h);
    }
}

}  // namespace phub

extern "C" {

const char* phub_last_error(void) { return g_error.c_str(); }

int phub_plan_count(int num_workers, int num_keys, const int64_t* key_elems, int64_t chunk_bytes,
                    int schedule, int num_bins, int min_items, int64_t* num_segments,
                    int* bins_used, int64_t* item_elems) {
    phub::Plan plan;
    std::string err;
    try {
        err = phub::build_plan(num_workers, num_keys, key_elems, chunk_bytes, schedule, num_bins,
                               min_items, &plan);
    } catch (const std::bad_alloc&) {
        return fail(PHUB_ENOMEM, "host allocation failed while building the schedule");
    }
    if (!err.empty()) return fail(PHUB_EINVAL, "%s", err.c_str());
    if (num_segments) *num_segments = int64_t(plan.segments.size());
    if (bins_used) *bins_used = plan.bins_used();
    if (item_elems) *item_elems = plan.item_elems;
    return PHUB_OK;
}

int phub_plan_build(int num_workers, int num_keys, const int64_t* key_elems, int64_t chunk_bytes,
                    int schedule, int num_bins, int min_items, phub_segment* segments,
                    int64_t* bin_begin, int64_t* bin_cost) {
    phub::Plan plan;
    std::string err;
    try {
        err = phub::build_plan(num_workers, num_keys, key_elems, chunk_bytes, schedule, num_bins,
                               min_items, &plan);
    } catch (const std::bad_alloc&) {
        return fail(PHUB_ENOMEM, "host allocation failed while building the schedule");
    }
    if (!err.empty()) return fail(PHUB_EINVAL, "%s", err.c_str());
    if ((!segments && !plan.segments.empty()) || !bin_begin)
        return fail(PHUB_EINVAL, "output arrays are NULL");
    for (size_t i = 0; i < plan.segments.size(); ++i)
        segments[i] = {plan.segments[i].key, plan.segments[i].count, plan.segments[i].offset};
    std::copy(plan.bin_begin.begin(), plan.bin_begin.end(), bin_begin);
    if (bin_cost) std::copy(plan.bin_cost.begin(), plan.bin_cost.end(), bin_cost);
    return PHUB_OK;
}

int phub_init(phub_job** out, int num_workers, int num_keys, const int64_t* key_elems,
              int64_t chunk_bytes, float lr, float momentum, float weight_decay, int nesterov,
              void* hip_stream) {
    return phub_init_ex(out, num_workers, num_keys, key_elems, chunk_bytes, lr, momentum,
                        weight_decay, nesterov, hip_stream, nullptr);
}

int phub_init_ex(phub_job** out, int num_workers, int num_keys, const int64_t* key_elems,
                 int64_t chunk_bytes, float lr, float momentum, float weight_decay, int nesterov,
                 void* hip_stream, const phub_options* options) {
    if (!out) return fail(PHUB_EINVAL, "out is NULL");
    *out = nullptr;
    {
        std::string err = phub::validate_shape(num_workers, num_keys, key_elems, chunk_bytes);
        if (!err.empty()) return fail(PHUB_EINVAL, "%s", err.c_str());
    }
    for (int k = 0; k < num_keys; ++k)
        if (key_elems[k] >= phub::kMaxDeviceKeyElems)
            return fail(PHUB_EINVAL, "key_elems[%d] = %lld exceeds the %lld elements a key may hold",
                        k, (long long)key_elems[k], (long long)(phub::kMaxDeviceKeyElems - 1));
    if (!std::isfinite(lr) || !std::isfinite(momentum) || !std::isfinite(weight_decay))
        return fail(PHUB_EINVAL, "lr, momentum and weight_decay must be finite");
    int schedule = phub::kScheduleLpt;
    int64_t resident_bytes = -1;  // -1: the shared per-device budget
    int num_rgroups = 0;          // 0: no readiness groups
    bool unfused = false;
    int optimizer = PHUB_OPT_MOMENTUM;
    float beta1 = 0, beta2 = 0, eps = 0;
    int workgroups = 0;  // 0: one per compute unit
    bool ordered_events = false;
    bool whole_chunks = false;
    if (options) {
        if (options->workgroups < 0 || options->workgroups > kMaxWorkgroups)
            return fail(PHUB_EINVAL, "workgroups must be in [0, %d], got %d", kMaxWorkgroups,
                        options->workgroups);
        workgroups = options->workgroups;
        if (options->schedule != PHUB_SCHEDULE_SPLIT && options->schedule != PHUB_SCHEDULE_LPT &&
            options->schedule != PHUB_SCHEDULE_DYNAMIC)
            return fail(PHUB_EINVAL, "unknown schedule %d", options->schedule);
        if (options->resident_bytes < -1)
            return fail(PHUB_EINVAL, "resident_bytes must be >= -1, got %lld",
                        (long long)options->resident_bytes);
        if (options->num_groups < 0)
            return fail(PHUB_EINVAL, "num_groups must be >= 0, got %d", options->num_groups);
        if (options->num_groups > 0) {
            if (!options->key_group) return fail(PHUB_EINVAL, "key_group is NULL");
            for (int k = 0; k < num_keys; ++k)
                if (options->key_group[k] < 0 || options->key_group[k] >= options->num_groups)
                    return fail(PHUB_EINVAL, "key_group[%d] = %d is outside [0, %d)", k,
                                options->key_group[k], options->num_groups);
        }
        if (options->unfused != 0 && options->num_groups > 0)
            return fail(PHUB_EINVAL, "the unfused variant does not take readiness groups");
        if (options->optimizer != PHUB_OPT_MOMENTUM && options->optimizer != PHUB_OPT_SGD &&
            options->optimizer != PHUB_OPT_ADAM)
            return fail(PHUB_EINVAL, "unknown optimizer %d", options->optimizer);
        if (options->optimizer == PHUB_OPT_ADAM) {
            if (!(options->beta1 >= 0.0f && options->beta1 < 1.0f) ||
                !(options->beta2 >= 0.0f && options->beta2 < 1.0f))
                return fail(PHUB_EINVAL, "Adam needs 0 <= beta1, beta2 < 1");
            if (!(options->eps >= 0.0f) || !std::isfinite(options->eps))
                return fail(PHUB_EINVAL, "Adam needs a finite eps >= 0");
        }
        optimizer = options->optimizer;
        beta1 = options->beta1;
        beta2 = options->beta2;
        eps = options->eps;
        schedule = options->schedule;
        if (options->resident_bytes >= 0) resident_bytes = options->resident_bytes;
        num_rgroups = options->num_groups;
        unfused = options->unfused != 0;
        if (options->ordered_events != 0 && options->ordered_events != 1)
            return fail(PHUB_EINVAL, "ordered_events must be 0 or 1, got %d", options->ordered_events);
        ordered_events = options->ordered_events == 1;
        if (options->whole_chunks != 0 && options->whole_chunks != 1)
            return fail(PHUB_EINVAL, "whole_chunks must be 0 or 1, got %d", options->whole_chunks);
        whole_chunks = options->whole_chunks == 1;
    }

    phub_job* j = new (std::nothrow) phub_job;
    if (!j) return fail(PHUB_ENOMEM, "host allocation of the job failed");
    int rc = PHUB_OK;
    try {
        j->num_workers = num_workers;
        j->num_keys = num_keys;
        j->key_elems.assign(key_elems, key_elems + num_keys);
        j->arena_offset.resize(num_keys);
        for (int k = 0; k < num_keys; ++k) {
            j->arena_offset[k] = j->arena_elems;
            j->arena_elems += (key_elems[k] + kArenaAlign - 1) / kArenaAlign * kArenaAlign;
        }
        j->chunk_bytes = chunk_bytes;
        j->lr = lr;
        j->mu = momentum;
        j->wd = weight_decay;
        j->nesterov = nesterov != 0;
        j->opt = optimizer == PHUB_OPT_SGD    ? phub::kOptSgd
                 : optimizer == PHUB_OPT_ADAM ? phub::kOptAdam
                 : j->nesterov                ? phub::kOptNesterov
                                              : phub::kOptMomentum;
        j->b1 = beta1;
        j->b2 = beta2;
        j->eps = eps;
        j->grads.assign(size_t(num_workers) * num_keys, nullptr);
        j->ready.assign(size_t(num_workers) * num_keys, nullptr);
        j->ordered_events = ordered_events;
        j->pushed.assign(size_t(num_workers) * num_keys, 0);
        j->outs.assign(size_t(num_workers) * num_keys, nullptr);
        j->has_out.assign(size_t(num_workers) * num_keys, 0);
        // readiness groups; rows of the pointer table ordered by group, then key
        j->streaming = num_rgroups > 0;
        j->num_rgroups = j->streaming ? num_rgroups : 1;
        j->key_rgroup.assign(num_keys, 0);
        if (j->streaming) j->key_rgroup.assign(options->key_group, options->key_group + num_keys);
        j->rgroup_row_begin.assign(j->num_rgroups + 1, 0);
        for (int k = 0; k < num_keys; ++k) ++j->rgroup_row_begin[j->key_rgroup[k] + 1];
        for (int g = 0; g < j->num_rgroups; ++g) j->rgroup_row_begin[g + 1] += j->rgroup_row_begin[g];
        j->row_of_key.assign(num_keys, 0);
        j->key_of_row.assign(num_keys, 0);
        std::vector<int> next(j->rgroup_row_begin.begin(), j->rgroup_row_begin.end() - 1);
        for (int k = 0; k < num_keys; ++k) {
            const int row = next[j->key_rgroup[k]]++;
            j->row_of_key[k] = row;
            j->key_of_row[row] = k;
        }
        j->rgroup_work.assign(j->num_rgroups, 0);
        j->group_last_event.assign(size_t(j->num_rgroups) * num_workers, nullptr);
        j->rgroup_events.assign(j->num_rgroups, 0);
        j->rgroup_pushed.assign(j->num_rgroups, 0);
        j->rgroup_launched.assign(j->num_rgroups, 0);
        j->rgroup_dirty.assign(j->num_rgroups, 1);
        j->rgroup_outs.assign(j->num_rgroups, 0);
        j->rgroup_out_dirty.assign(j->num_rgroups, 1);
    } catch (const std::bad_alloc&) {
        delete j;
        return fail(PHUB_ENOMEM, "host allocation of the job tables failed");
    }

    hipError_t e = hipGetDevice(&j->device);
    if (e != hipSuccess) {
        delete j;
        return hip_fail(e, "hipGetDevice");
    }
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, j->device);
    if (e != hipSuccess || cus < 1) {
        delete j;
        return e != hipSuccess ? hip_fail(e, "hipDeviceGetAttribute(CU count)")
                               : fail(PHUB_EHIP, "device reports no compute units");
    }
    int clock_khz = 0;
    e = hipDeviceGetAttribute(&clock_khz, hipDeviceAttributeWallClockRate, j->device);
    if (e != hipSuccess || clock_khz < 1) {
        delete j;
        return e != hipSuccess ? hip_fail(e, "hipDeviceGetAttribute(wall clock rate)")
                               : fail(PHUB_EHIP, "device reports no wall clock");
    }
    j->wall_clock_khz = clock_khz;

    // Cache residency: the state of arena elements [0, resident_elems) is
    // kept in the memory-side cache.  An explicit budget is the job's own;
    // the default takes what is left of the device's shared budget, first
    // come first served.  Jobs whose streamed state is written back in
    // bursts (burst_write_back) step faster with all of their state
    // streamed than with part of it cached, and as fast as with all of it
    // cached once the cache no longer holds it from the previous step, so by
    // default they take none of the shared budget (measured on MI355X,
    // fraction of peak, nothing cached against the default: 102 M
    // parameters with 16 workers 0.82 against 0.79; four concurrent
    // 8-worker jobs 0.77 against 0.76; 25.6 M parameters with 8 workers
    // 0.79 streamed, 0.83 cached while the cache keeps the state from the
    // previous step and 0.75 after the cache was flushed).  Jobs without
    // bursts (few workers, the any-N kernel, the unfused variant) still gain
    // from the cache.
    j->num_states = j->opt == phub::kOptSgd ? 1 : j->opt == phub::kOptAdam ? 3 : 2;
    const int64_t elem_state_bytes = j->num_states * int64_t(sizeof(float));
    {
        std::lock_guard<std::mutex> lk(g_live_mu);
        int64_t budget = resident_bytes;
        const bool stream_all = !unfused && phub::burst_write_back(num_workers, j->num_states);
        if (budget < 0)
            budget = stream_all ? 0 : std::max<int64_t>(0, PHUB_DEVICE_CACHE_BYTES - g_cache_claimed[j->device]);
        j->resident_elems = std::min(j->arena_elems, budget / elem_state_bytes);
        if (resident_bytes < 0) {
            j->cache_claim = j->resident_elems * elem_state_bytes;
            g_cache_claimed[j->device] += j->cache_claim;
        }
    }

    // Two schedules per readiness group over the group's keys in row order:
    // phase 0 holds the cache-resident part of the keys, phase 1 the rest.
    // A key that straddles resident_elems is cut at a tile boundary of the
    // key (the part below the cut is resident), so both parts keep the
    // 16-byte alignment of the key's start.  A part is a "virtual key": a
    // row and a first element within the key.
    using VKey = phub::VirtualKey;
    std::vector<phub::Plan> plans;  // [group * 2 + phase]
    std::vector<std::vector<VKey>> vkeys;
    {
        const int groups = workgroups > 0 ? workgroups : cus * PHUB_GROUPS_PER_CU;
        const int bins = groups * (phub::kBlockThreads / 64);
        std::string err;
        try {
            plans.resize(size_t(j->num_rgroups) * 2);
            vkeys.resize(size_t(j->num_rgroups) * 2);
            for (int g = 0; g < j->num_rgroups && err.empty(); ++g) {
                for (int r = j->rgroup_row_begin[g]; r < j->rgroup_row_begin[g + 1]; ++r) {
                    const int k = j->key_of_row[r];
                    const int64_t n = key_elems[k], o = j->arena_offset[k];
                    int64_t cut = 0;  // elements of the key that are resident
                    if (o + n <= j->resident_elems)
                        cut = n;
                    else if (o < j->resident_elems)
                        cut = (j->resident_elems - o) / phub::kTileElems * phub::kTileElems;
                    if (cut > 0) vkeys[g * 2].push_back({r, 0, cut});
                    if (cut < n || n == 0) vkeys[g * 2 + 1].push_back({r, cut, n - cut});
                }
                for (int ph = 0; ph < 2 && err.empty(); ++ph) {
                    const std::vector<VKey>& vk = vkeys[g * 2 + ph];
                    phub::Plan& plan = plans[g * 2 + ph];
                    if (!vk.empty()) {
                        std::vector<int64_t> elems(vk.size());
                        for (size_t i = 0; i < vk.size(); ++i) elems[i] = vk[i].elems;
                        err = phub::build_plan(num_workers, int(vk.size()), elems.data(),
                                               chunk_bytes,
                                               schedule == PHUB_SCHEDULE_DYNAMIC ? phub::kScheduleLpt
                                                                                : schedule,
                                               bins, whole_chunks ? 0 : kLptItemsPerBin * bins,
                                               &plan);
                    } else {
                        plan.bin_begin.assign(1, 0);
                    }
                    // every wave of the grid reads its bins: pad dropped bins as empty
                    while (plan.bin_begin.size() < size_t(bins) + 1)
                        plan.bin_begin.push_back(plan.bin_begin.back());
                    if (!plan.segments.empty()) j->rgroup_work[g] = 1;
                    j->num_segments += int64_t(plan.segments.size());
                }
            }
        } catch (const std::bad_alloc&) {
            err = "host allocation failed while building the schedule";
        }
        if (!err.empty()) {
            if (j->cache_claim) {
                std::lock_guard<std::mutex> lk(g_live_mu);
                g_cache_claimed[j->device] -= j->cache_claim;
            }
            delete j;
            return fail(PHUB_EINVAL, "%s", err.c_str());
        }
        j->groups = j->num_segments == 0 ? 0 : groups;
        j->bins = bins;
    }
    j->schedule = schedule;
    // the pool walk exists in the fixed-N fused kernels only
    j->dynamic = schedule == PHUB_SCHEDULE_DYNAMIC && !unfused && j->groups > 0 &&
                 phub::takes_tile_pool(num_workers, j->opt);
    const int num_states = j->num_states;

#define PHUB_TRY(call, what)                 \
    do {                                     \
        hipError_t e_ = (call);              \
        if (e_ != hipSuccess) {              \
            rc = hip_fail(e_, what);         \
            goto fail_cleanup;               \
        }                                    \
    } while (0)

    {
        if (hip_stream) {
            j->stream = static_cast<hipStream_t>(hip_stream);
        } else {
            PHUB_TRY(hipStreamCreateWithFlags(&j->stream, hipStreamNonBlocking), "hipStreamCreate");
            j->own_stream = true;
        }
        const size_t arena_bytes = size_t(std::max<int64_t>(j->arena_elems, 1)) * sizeof(float);
        if (hipMalloc(&j->weights, arena_bytes) != hipSuccess ||
            (num_states >= 2 && hipMalloc(&j->moments, arena_bytes) != hipSuccess) ||
            (num_states >= 3 && hipMalloc(&j->second, arena_bytes) != hipSuccess)) {
            (void)hipGetLastError();
            rc = fail(PHUB_ENOMEM, "device allocation of the optimizer state (%zu bytes per array) failed",
                      arena_bytes);
            goto fail_cleanup;
        }
        if (unfused && hipMalloc(&j->merge, arena_bytes) != hipSuccess) {
            (void)hipGetLastError();
            rc = fail(PHUB_ENOMEM, "device allocation of the merge buffer (%zu bytes) failed",
                      arena_bytes);
            goto fail_cleanup;
        }
        PHUB_TRY(hipMemsetAsync(j->weights, 0, arena_bytes, j->stream), "hipMemsetAsync(W)");
        if (j->moments)
            PHUB_TRY(hipMemsetAsync(j->moments, 0, arena_bytes, j->stream), "hipMemsetAsync(M)");
        if (j->second)
            PHUB_TRY(hipMemsetAsync(j->second, 0, arena_bytes, j->stream), "hipMemsetAsync(V)");

        // Device form of the schedules: each bin's segments become full tiles
        // (the kernel's straight-line hot loop) and at most one remainder
        // each (partial tile and ragged end), in segment order; one block of
        // 2 * bins + 1 offsets per readiness group (the resident bins, then
        // the streamed ones).  A descriptor's key is the key's row in the
        // pointer table.
        phub::DeviceTables dt;
        {
            std::vector<int64_t> row_arena_offset(num_keys);
            for (int r = 0; r < num_keys; ++r) row_arena_offset[r] = j->arena_offset[j->key_of_row[r]];
            for (int g = 0; g < j->num_rgroups; ++g) {
                dt.tile_begin.push_back(int32_t(dt.tiles.size()));
                dt.rem_begin.push_back(int32_t(dt.rems.size()));
                for (int ph = 0; ph < 2; ++ph) {
                    const size_t t0 = dt.tiles.size();
                    const int64_t elems = phub::append_device_tables(
                        plans[g * 2 + ph], vkeys[g * 2 + ph], row_arena_offset, j->bins, &dt);
                    if (elems < 0) {
                        rc = fail(PHUB_EINVAL, "schedule too large");
                        goto fail_cleanup;
                    }
                    if (ph == 0) j->resident_bytes += elems * elem_state_bytes;
                    if (ph == 1 && j->dynamic) {
                        // the streamed full tiles become the group's pool, in
                        // address order; its bins keep their remainders only
                        std::sort(dt.tiles.begin() + t0, dt.tiles.end(),
                                  [](const phub::DevTile& x, const phub::DevTile& y) {
                                      return x.arena_offset < y.arena_offset;
                                  });
                        j->pool_begin.push_back(int32_t(t0));
                        j->pool_count.push_back(int32_t(dt.tiles.size() - t0));
                        std::fill(dt.tile_begin.end() - j->bins, dt.tile_begin.end(), int32_t(t0));
                    }
                }
            }
        }
        const std::vector<phub::DevTile>& dtiles = dt.tiles;
        const std::vector<phub::DevRem>& drems = dt.rems;
        const std::vector<int32_t>& tile_begin = dt.tile_begin;
        const std::vector<int32_t>& rem_begin = dt.rem_begin;
        std::vector<phub::WaveHead> heads;
        for (int g = 0; g < j->num_rgroups; ++g)
            phub::append_wave_heads(dt, size_t(g) * (2 * size_t(j->bins) + 1), j->bins, &heads);
        j->num_tiles = int64_t(dtiles.size());
        j->num_rems = int64_t(drems.size());
        const size_t tile_bytes = std::max<size_t>(dtiles.size(), 1) * sizeof(phub::DevTile);
        const size_t rem_bytes = std::max<size_t>(drems.size(), 1) * sizeof(phub::DevRem);
        const size_t tb_bytes = tile_begin.size() * sizeof(int32_t);
        const size_t rb_bytes = rem_begin.size() * sizeof(int32_t);
        const size_t head_bytes = heads.size() * sizeof(phub::WaveHead);
        const size_t tab_bytes = j->grads.size() * sizeof(const float*);
        const size_t counter_bytes =
            size_t(j->num_rgroups) * kCountersPerGroup * sizeof(unsigned long long);
        j->pool_launches.assign(j->num_rgroups, 0);
        if (hipMalloc(&j->d_tiles, tile_bytes) != hipSuccess ||
            hipMalloc(&j->d_tile_begin, tb_bytes) != hipSuccess ||
            hipMalloc(&j->d_rems, rem_bytes) != hipSuccess ||
            hipMalloc(&j->d_rem_begin, rb_bytes) != hipSuccess ||
            hipMalloc(&j->d_heads, head_bytes) != hipSuccess ||
            hipMalloc(&j->d_grads, tab_bytes) != hipSuccess ||
            hipMalloc(&j->d_outs, tab_bytes) != hipSuccess ||
            (j->dynamic && hipMalloc(&j->d_counters, counter_bytes) != hipSuccess)) {
            (void)hipGetLastError();
            rc = fail(PHUB_ENOMEM, "device allocation of the schedule failed");
            goto fail_cleanup;
        }
        if (!dtiles.empty())
            PHUB_TRY(hipMemcpy(j->d_tiles, dtiles.data(), dtiles.size() * sizeof(phub::DevTile),
                               hipMemcpyHostToDevice),
                     "hipMemcpy(tiles)");
        if (!drems.empty())
            PHUB_TRY(hipMemcpy(j->d_rems, drems.data(), drems.size() * sizeof(phub::DevRem),
                               hipMemcpyHostToDevice),
                     "hipMemcpy(remainders)");
        PHUB_TRY(hipMemcpy(j->d_tile_begin, tile_begin.data(), tb_bytes, hipMemcpyHostToDevice),
                 "hipMemcpy(tile bins)");
        if (j->d_counters)
            PHUB_TRY(hipMemsetAsync(j->d_counters, 0, counter_bytes, j->stream),
                     "hipMemsetAsync(pool counters)");
        PHUB_TRY(hipMemcpy(j->d_rem_begin, rem_begin.data(), rb_bytes, hipMemcpyHostToDevice),
                 "hipMemcpy(remainder bins)");
        PHUB_TRY(hipMemcpy(j->d_heads, heads.data(), head_bytes, hipMemcpyHostToDevice),
                 "hipMemcpy(wave heads)");
        for (int i = 0; i < kStageSlots; ++i) {
            if (hipHostMalloc(reinterpret_cast<void**>(&j->stage[i]), tab_bytes,
                              hipHostMallocDefault) != hipSuccess ||
                hipHostMalloc(reinterpret_cast<void**>(&j->stage_out[i]), tab_bytes,
                              hipHostMallocDefault) != hipSuccess) {
                (void)hipGetLastError();
                rc = fail(PHUB_ENOMEM, "pinned host allocation of the pointer staging failed");
                goto fail_cleanup;
            }
            PHUB_TRY(hipEventCreateWithFlags(&j->stage_done[i], hipEventDisableTiming),
                     "hipEventCreate");
        }
        PHUB_TRY(hipStreamSynchronize(j->stream), "hipStreamSynchronize (init)");
    }
#undef PHUB_TRY

    {
        std::lock_guard<std::mutex> lk(g_live_mu);
        g_live.insert(j);
    }
    *out = j;
    return PHUB_OK;

fail_cleanup:
    if (j->cache_claim) {
        std::lock_guard<std::mutex> lk(g_live_mu);
        g_cache_claimed[j->device] -= j->cache_claim;
    }
    release(j);
    return rc;
}

int phub_set_weights(phub_job* j, int key, const float* src) {
    if (!is_live(j)) return fail(PHUB_ESTATE, "not a live job handle");
    if (int rc = check_key(j, key)) return rc;
    const int64_t n = j->key_elems[key];
    if (n == 0) return PHUB_OK;
    if (!src) return fail(PHUB_EINVAL, "src is NULL");
    DeviceScope ds(j->device);
    if (!ds.ok()) return fail(PHUB_EHIP, "cannot make device %d current", j->device);
    const size_t bytes = size_t(n) * sizeof(float);
    hipError_t e = hipMemcpyAsync(j->weights + j->arena_offset[key], src, bytes, hipMemcpyDefault,
                                  j->stream);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(set_weights)");
    for (float* st : {j->moments, j->second}) {
        if (!st) continue;
        e = hipMemsetAsync(st + j->arena_offset[key], 0, bytes, j->stream);
        if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync(optimizer state)");
    }
    return PHUB_OK;
}

int phub_push(phub_job* j, int worker, int key, const float* grad) {
    return phub_push_event(j, worker, key, grad, nullptr);
}

int phub_push_event(phub_job* j, int worker, int key, const float* grad, void* hip_event) {
    if (!is_live(j)) return fail(PHUB_ESTATE, "not a live job handle");
    if (int rc = check_grad(j, worker, key, grad)) return rc;
    return record_push(j, worker, key, grad, static_cast<hipEvent_t>(hip_event));
}

int phub_pushpull(phub_job* j, int worker, int key, const float* grad, float* model_out) {
    return phub_pushpull_keys(j, worker, 1, &key, &grad, &model_out, nullptr);
}

int phub_pushpull_keys(phub_job* j, int worker, int count, const int* keys,
                       const float* const* grads, float* const* model_outs, void* hip_event) {
    if (!is_live(j)) return fail(PHUB_ESTATE, "not a live job handle");
    if (count < 0) return fail(PHUB_EINVAL, "count %d is negative", count);
    if (count > 0 && (!grads || !model_outs)) return fail(PHUB_EINVAL, "grads or model_outs is NULL");
    if (!keys && count > j->num_keys)
        return fail(PHUB_EINVAL, "count %d exceeds the %d keys", count, j->num_keys);
    for (int i = 0; i < count; ++i) {
        const int key = keys ? keys[i] : i;
        if (int rc = check_grad(j, worker, key, grads[i])) return rc;
        if (int rc = check_out(j, worker, key, model_outs[i])) return rc;
    }
    const hipEvent_t ev = static_cast<hipEvent_t>(hip_event);
    for (int i = 0; i < count; ++i) {
        const int key = keys ? keys[i] : i;
        if (j->streaming && j->rgroup_launched[j->key_rgroup[key]])
            return fail(PHUB_ESTATE,
                        "key %d belongs to readiness group %d, which was already launched this "
                        "step", key, j->key_rgroup[key]);
        record_out(j, worker, key, model_outs[i]);  // before the push that may launch the group
        if (int rc = record_push(j, worker, key, grads[i], ev)) return rc;
    }
    return PHUB_OK;
}

int phub_push_keys(phub_job* j, int worker, int count, const int* keys,
                   const float* const* grads) {
    return phub_push_keys_event(j, worker, count, keys, grads, nullptr);
}

int phub_push_keys_event(phub_job* j, int worker, int count, const int* keys,
                         const float* const* grads, void* hip_event) {
    if (!is_live(j)) return fail(PHUB_ESTATE, "not a live job handle");
    if (count < 0) return fail(PHUB_EINVAL, "count %d is negative", count);
    if (count > 0 && !grads) return fail(PHUB_EINVAL, "grads is NULL");
    if (!keys && count > j->num_keys)
        return fail(PHUB_EINVAL, "count %d exceeds the %d keys", count, j->num_keys);
    for (int i = 0; i < count; ++i)
        if (int rc = check_grad(j, worker, keys ? keys[i] : i, grads[i])) return rc;
    const hipEvent_t ev = static_cast<hipEvent_t>(hip_event);
    for (int i = 0; i < count; ++i)
        if (int rc = record_push(j, worker, keys ? keys[i] : i, grads[i], ev)) return rc;
    return PHUB_OK;
}

int phub_push_all(phub_job* j, const float* const* grads) {
    if (!is_live(j)) return fail(PHUB_ESTATE, "not a live job handle");
    if (!grads) return fail(PHUB_EINVAL, "grads is NULL");
    const int nk = j->num_keys;
    for (int w = 0; w < j->num_workers; ++w)
        for (int k = 0; k < nk; ++k)
            if (int rc = check_grad(j, w, k, grads[size_t(w) * nk + k])) return rc;
    if (j->streaming)
        for (int g = 0; g < j->num_rgroups; ++g)
            if (j->rgroup_launched[g])
                return fail(PHUB_ESTATE,
                            "readiness group %d was already launched this step; nothing pushed", g);
    for (int w = 0; w < j->num_workers; ++w)
        for (int k = 0; k < nk; ++k)
            if (int rc = record_push(j, w, k, grads[size_t(w) * nk + k], nullptr)) return rc;
    return PHUB_OK;
}

int phub_step(phub_job* j) {
    if (!is_live(j)) return fail(PHUB_ESTATE, "not a live job handle");
    const int64_t need = int64_t(j->num_workers) * j->num_keys;
    if (j->num_pushed != need) {
        for (int k = 0; k < j->num_keys; ++k)
            for (int w = 0; w < j->num_workers; ++w)
                if (!j->pushed[size_t(j->row_of_key[k]) * j->num_workers + w])
                    return fail(PHUB_ENOTREADY,
                                "%lld of %lld (worker, key) pairs pushed; worker %d has not "
                                "pushed key %d",
                                (long long)j->num_pushed, (long long)need, w, k);
    }
    for (int g = 0; g < j->num_rgroups; ++g)
        if (!j->rgroup_launched[g])
            if (int rc = launch_group(j, g)) return rc;
    std::fill(j->pushed.begin(), j->pushed.end(), 0);
    if (j->step_events) {
        std::fill(j->ready.begin(), j->ready.end(), nullptr);
        std::fill(j->group_last_event.begin(), j->group_last_event.end(), nullptr);
        std::fill(j->rgroup_events.begin(), j->rgroup_events.end(), 0);
        j->step_events = 0;
    }
    std::fill(j->rgroup_pushed.begin(), j->rgroup_pushed.end(), 0);
    std::fill(j->rgroup_launched.begin(), j->rgroup_launched.end(), 0);
    if (j->step_outs) {
        std::fill(j->has_out.begin(), j->has_out.end(), 0);
        std::fill(j->rgroup_outs.begin(), j->rgroup_outs.end(), 0);
        j->step_outs = 0;
    }
    j->num_pushed = 0;
    ++j->steps_done;
    if (j->stage_claimed) {
        j->stage_slot = (j->stage_slot + 1) % kStageSlots;
        j->stage_claimed = false;
    }
    return PHUB_OK;
}

int phub_pull(phub_job* j, int key, const float** weights) {
    if (!is_live(j)) return fail(PHUB_ESTATE, "not a live job handle");
    if (int rc = check_key(j, key)) return rc;
    if (!weights) return fail(PHUB_EINVAL, "weights is NULL");
    *weights = j->weights + j->arena_offset[key];
    return PHUB_OK;
}

int phub_get_state(phub_job* j, int key, const float** weights, const float** momentum) {
    if (!is_live(j)) return fail(PHUB_ESTATE, "not a live job handle");
    if (int rc = check_key(j, key)) return rc;
    if (weights) *weights = j->weights + j->arena_offset[key];
    if (momentum) *momentum = j->moments ? j->moments + j->arena_offset[key] : nullptr;
    return PHUB_OK;
}

int phub_get_second_moment(phub_job* j, int key, const float** second) {
    if (!is_live(j)) return fail(PHUB_ESTATE, "not a live job handle");
    if (int rc = check_key(j, key)) return rc;
    if (!second) return fail(PHUB_EINVAL, "second is NULL");
    *second = j->second ? j->second + j->arena_offset[key] : nullptr;
    return PHUB_OK;
}

int phub_sync(phub_job* j) {
    if (!is_live(j)) return fail(PHUB_ESTATE, "not a live job handle");
    DeviceScope ds(j->device);
    if (!ds.ok()) return fail(PHUB_EHIP, "cannot make device %d current", j->device);
    hipError_t e = hipStreamSynchronize(j->stream);
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    return PHUB_OK;
}

int phub_get_stream(phub_job* j, void** hip_stream) {
    if (!is_live(j)) return fail(PHUB_ESTATE, "not a live job handle");
    if (!hip_stream) return fail(PHUB_EINVAL, "hip_stream is NULL");
    *hip_stream = j->stream;
    return PHUB_OK;
}

int phub_job_info(phub_job* j, int* workgroups, int* threads_per_group, int64_t* segments,
                  int64_t* state_bytes, int64_t* resident_bytes) {
    if (!is_live(j)) return fail(PHUB_ESTATE, "not a live job handle");
    if (workgroups) *workgroups = j->groups;
    if (threads_per_group) *threads_per_group = phub::kBlockThreads;
    if (segments) *segments = j->num_segments;
    if (state_bytes) *state_bytes = j->num_states * j->arena_elems * int64_t(sizeof(float));
    if (resident_bytes) *resident_bytes = j->resident_bytes;
    return PHUB_OK;
}

int phub_destroy(phub_job* j) {
    {
        std::lock_guard<std::mutex> lk(g_live_mu);
        if (!j || g_live.erase(j) == 0) return fail(PHUB_ESTATE, "not a live job handle");
        if (j->cache_claim) g_cache_claimed[j->device] -= j->cache_claim;
    }
    DeviceScope ds(j->device);
    hipError_t e = hipStreamSynchronize(j->stream);
    release(j);
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize (destroy)");
    return PHUB_OK;
}

}  // extern "C"
