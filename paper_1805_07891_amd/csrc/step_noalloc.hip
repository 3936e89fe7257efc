// One exchange step that allocates nothing: phub_step_noalloc.
//
// For callers that cannot allocate device memory (serving loops that must
// not call hipMalloc, harnesses that forbid allocation).  The caller passes
// the gradients and the master weights and momentum; everything else the
// fused kernel reads (the chunk schedule of section 3.2.4 in its device form
// and the gradient pointer table) goes into `scratch` below, a file-scope
// device array that each GPU holds for the life of the process.  The kernel
// is the job path's fused kernel, with the same schedule rules, so the
// results are those of phub_init + phub_push_all + phub_step on the same
// inputs (and do not depend on the schedule anyway).
//
// The array's name in host code is a host-side stand-in, not a device
// address: its device address is taken once per device with
// hipGetSymbolAddress, with that device current, and only that address is
// used from host code.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "kernels.hpp"
#include "phub.h"
#include "plan.hpp"

// Largest schedule plus pointer table one call can hold: 4 MiB, enough for
// about 240 M parameters in 1024-element tiles (16 bytes each, beside the
// 128 KB of wave heads) with the
// pointer table of thousands of (worker, key) pairs.
#define PHUB_NOALLOC_SCRATCH_BYTES (size_t(4) << 20)

static __device__ __align__(256) unsigned char scratch[PHUB_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr size_t kScratchBytes = PHUB_NOALLOC_SCRATCH_BYTES;
constexpr int64_t kArenaAlign = 64;  // elements: key slices of the arena start 256-byte aligned
constexpr size_t kRegionAlign = 256;

// What one device needs for a call, found once per device.
struct DeviceSetup {
    unsigned char* scratch = nullptr;  // device address of `scratch` on this device
    int compute_units = 0;
    int64_t wall_clock_khz = 0;
};

std::mutex g_setup_mu;
std::unordered_map<int, DeviceSetup> g_setup;

// The device's setup, found on the first call made on it (the device is
// current during the call).
int device_setup(int device, DeviceSetup* out) {
    std::lock_guard<std::mutex> lk(g_setup_mu);
    auto it = g_setup.find(device);
    if (it != g_setup.end()) {
        *out = it->second;
        return PHUB_OK;
    }
    DeviceSetup s;
    void* ptr = nullptr;
    hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
        return phub::report_error(PHUB_EHIP, std::string("hipGetSymbolAddress(scratch) failed: ") +
                                                 hipGetErrorString(e));
    s.scratch = static_cast<unsigned char*>(ptr);
    e = hipDeviceGetAttribute(&s.compute_units, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess || s.compute_units < 1)
        return phub::report_error(PHUB_EHIP, "hipDeviceGetAttribute(CU count) failed");
    int khz = 0;
    e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, device);
    if (e != hipSuccess || khz < 1)
        return phub::report_error(PHUB_EHIP, "hipDeviceGetAttribute(wall clock rate) failed");
    s.wall_clock_khz = khz;
    g_setup[device] = s;
    *out = s;
    return PHUB_OK;
}

size_t align_up(size_t x) { return (x + kRegionAlign - 1) / kRegionAlign * kRegionAlign; }

std::string fmt(const char* f, long long a, long long b = 0, long long c = 0) {
    char buf[256];
    std::snprintf(buf, sizeof buf, f, a, b, c);
    return buf;
}

}  // namespace

extern "C" int phub_step_noalloc(int num_workers, int num_keys, const int64_t* key_elems,
                                 int64_t chunk_bytes, float lr, float momentum,
                                 float weight_decay, int nesterov, const float* const* grads,
                                 float* weights, float* moments, void* hip_stream) {
    using phub::report_error;
    {
        const std::string err = phub::validate_shape(num_workers, num_keys, key_elems, chunk_bytes);
        if (!err.empty()) return report_error(PHUB_EINVAL, err);
    }
    if (!std::isfinite(lr) || !std::isfinite(momentum) || !std::isfinite(weight_decay))
        return report_error(PHUB_EINVAL, "lr, momentum and weight_decay must be finite");
    if (!grads) return report_error(PHUB_EINVAL, "grads is NULL");
    // the arena layout of a job's state: key slices padded to 64 elements
    std::vector<int64_t> arena_offset(num_keys);
    int64_t arena_elems = 0;
    for (int k = 0; k < num_keys; ++k) {
        if (key_elems[k] >= phub::kMaxDeviceKeyElems)
            return report_error(PHUB_EINVAL, fmt("key_elems[%lld] = %lld exceeds the %lld elements a key may hold",
                                                 k, key_elems[k], phub::kMaxDeviceKeyElems - 1));
        arena_offset[k] = arena_elems;
        arena_elems += (key_elems[k] + kArenaAlign - 1) / kArenaAlign * kArenaAlign;
    }
    if (arena_elems > 0) {
        if (!weights || !moments) return report_error(PHUB_EINVAL, "weights or moments is NULL");
        if (reinterpret_cast<uintptr_t>(weights) % 16 || reinterpret_cast<uintptr_t>(moments) % 16)
            return report_error(PHUB_EINVAL, "weights and moments must be 16-byte aligned");
    }
    for (int w = 0; w < num_workers; ++w)
        for (int k = 0; k < num_keys; ++k) {
            const float* g = grads[size_t(w) * num_keys + k];
            if (!g && key_elems[k] != 0)
                return report_error(PHUB_EINVAL, fmt("gradient of worker %lld for key %lld is NULL", w, k));
            if (reinterpret_cast<uintptr_t>(g) % 16)
                return report_error(PHUB_EINVAL,
                                    fmt("gradient of worker %lld for key %lld is not 16-byte aligned", w, k));
        }
    // Bound the scratch need before any HIP call: the schedule holds at most
    // one tile per 1024 elements plus a remainder per segment, and a bin
    // table; the pointer table one pointer per (worker, key).  The exact
    // size is checked again once the schedule is built.
    const size_t table_bytes = size_t(num_workers) * size_t(num_keys) * sizeof(const float*);
    if (table_bytes > kScratchBytes || arena_elems / phub::kTileElems * int64_t(sizeof(phub::DevTile)) >
                                           int64_t(kScratchBytes))
        return report_error(PHUB_EINVAL,
                            fmt("the step needs more than the %lld bytes of scratch this entry point "
                                "has (%lld parameters, %lld gradient pointers)",
                                (long long)kScratchBytes, arena_elems,
                                (long long)num_workers * num_keys));

    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return report_error(PHUB_EHIP, "hipGetDevice failed");
    DeviceSetup setup;
    if (int rc = device_setup(device, &setup)) return rc;

    // The schedule, as phub_init builds it for one readiness group with
    // nothing cache-resident: every key is a streamed virtual key.
    const int grid = setup.compute_units;
    const int bins = grid * (phub::kBlockThreads / 64);
    phub::DeviceTables dt;
    try {
        std::vector<phub::VirtualKey> vkeys;
        for (int k = 0; k < num_keys; ++k) vkeys.push_back({k, 0, key_elems[k]});
        std::vector<int64_t> elems(num_keys);
        for (int k = 0; k < num_keys; ++k) elems[k] = key_elems[k];
        phub::Plan plan;
        const std::string err = phub::build_plan(num_workers, num_keys, elems.data(), chunk_bytes,
                                                 phub::kScheduleLpt, bins, 128 * bins, &plan);
        if (!err.empty()) return report_error(PHUB_EINVAL, err);
        while (plan.bin_begin.size() < size_t(bins) + 1) plan.bin_begin.push_back(plan.bin_begin.back());
        // resident bins (empty), then streamed bins
        dt.tile_begin.assign(bins + 1, 0);
        dt.rem_begin.assign(bins + 1, 0);
        if (phub::append_device_tables(plan, vkeys, arena_offset, bins, &dt) < 0)
            return report_error(PHUB_EINVAL, "schedule too large");
    } catch (const std::bad_alloc&) {
        return report_error(PHUB_ENOMEM, "host allocation failed while building the schedule");
    }
    if (dt.tiles.empty() && dt.rems.empty()) return PHUB_OK;  // every key is empty
    std::vector<phub::WaveHead> heads;
    try {
        phub::append_wave_heads(dt, 0, bins, &heads);
    } catch (const std::bad_alloc&) {
        return report_error(PHUB_ENOMEM, "host allocation failed while building the schedule");
    }

    // Scratch layout, each region 256-byte aligned: bin offsets of tiles and
    // remainders, the waves' heads, tiles, remainders, gradient pointer
    // table (row = key).
    const size_t off_tb = 0;
    const size_t off_rb = align_up(off_tb + dt.tile_begin.size() * sizeof(int32_t));
    const size_t off_heads = align_up(off_rb + dt.rem_begin.size() * sizeof(int32_t));
    const size_t off_tiles = align_up(off_heads + heads.size() * sizeof(phub::WaveHead));
    const size_t off_rems = align_up(off_tiles + dt.tiles.size() * sizeof(phub::DevTile));
    const size_t off_grads = align_up(off_rems + dt.rems.size() * sizeof(phub::DevRem));
    const size_t total = off_grads + table_bytes;
    if (total > kScratchBytes)
        return report_error(PHUB_EINVAL,
                            fmt("the step needs %lld bytes of scratch; this entry point has %lld",
                                (long long)total, (long long)kScratchBytes));
    std::vector<unsigned char> host;
    try {
        host.assign(total, 0);
    } catch (const std::bad_alloc&) {
        return report_error(PHUB_ENOMEM, "host allocation of the scratch image failed");
    }
    std::memcpy(host.data() + off_tb, dt.tile_begin.data(), dt.tile_begin.size() * sizeof(int32_t));
    std::memcpy(host.data() + off_rb, dt.rem_begin.data(), dt.rem_begin.size() * sizeof(int32_t));
    std::memcpy(host.data() + off_heads, heads.data(), heads.size() * sizeof(phub::WaveHead));
    if (!dt.tiles.empty())
        std::memcpy(host.data() + off_tiles, dt.tiles.data(), dt.tiles.size() * sizeof(phub::DevTile));
    if (!dt.rems.empty())
        std::memcpy(host.data() + off_rems, dt.rems.data(), dt.rems.size() * sizeof(phub::DevRem));
    // pointer table [key * num_workers + worker]
    const float** table = reinterpret_cast<const float**>(host.data() + off_grads);
    for (int k = 0; k < num_keys; ++k)
        for (int w = 0; w < num_workers; ++w)
            table[size_t(k) * num_workers + w] = grads[size_t(w) * num_keys + k];

    // Upload after the stream's earlier work (an earlier call's kernel may
    // still read the scratch), then wait, so that the host image may go.
    hipStream_t stream = static_cast<hipStream_t>(hip_stream);
    e = hipMemcpyAsync(setup.scratch, host.data(), total, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess)
        return report_error(PHUB_EHIP, std::string("hipMemcpyAsync (scratch) failed: ") +
                                           hipGetErrorString(e));
    e = hipStreamSynchronize(stream);
    if (e != hipSuccess)
        return report_error(PHUB_EHIP, std::string("hipStreamSynchronize failed: ") +
                                           hipGetErrorString(e));

    phub::StepParams p{};
    p.tile_begin = reinterpret_cast<const int32_t*>(setup.scratch + off_tb);
    p.rem_begin = reinterpret_cast<const int32_t*>(setup.scratch + off_rb);
    p.heads = reinterpret_cast<const phub::WaveHead*>(setup.scratch + off_heads);
    p.tiles = reinterpret_cast<const phub::DevTile*>(setup.scratch + off_tiles);
    p.rems = reinterpret_cast<const phub::DevRem*>(setup.scratch + off_rems);
    p.grads = reinterpret_cast<const float* const*>(setup.scratch + off_grads);
    p.outs = nullptr;
    p.merge = nullptr;
    p.weights = weights;
    p.moments = moments;
    p.second = nullptr;
    p.opt.nlr = -lr;
    p.opt.mu = momentum;
    p.opt.wd = weight_decay;
    phub::write_phase_ticks(num_workers, 2, setup.wall_clock_khz, &p.opt.wb_period, &p.opt.wb_window);
    p.num_workers = num_workers;
    e = phub::launch_fused_step(p, nesterov ? phub::kOptNesterov : phub::kOptMomentum, grid, stream);
    if (e != hipSuccess)
        return report_error(PHUB_EHIP, std::string("launch of the fused step kernel failed: ") +
                                           hipGetErrorString(e));
    return PHUB_OK;
}
