#!/usr/bin/env python3
"""Benchmark of the fused PHub exchange step on one MI355X.

One step = every worker pushes all its keys (pointer registration) and the
job runs one fused aggregate + optimize launch over all keys, for every job
of the workload (the tenants of a multi-job workload each on their own
stream, concurrently).  Gradients, weights and momentum are resident in HBM
before the timed region starts.  Prints one JSON line:

  metric   worker-gradient GB/s aggregated+optimized per step
  value    N * P * 4 bytes per step / wall time per step, summed over jobs
  roofline the fused kernel's algorithmic HBM bytes ((N + 4) * P * 4 per
           launch, summed over the step's launches) / its duration, measured
           with HIP events on the jobs' streams, against the 8 TB/s HBM3E
           peak, beside ceilings measured in the same run (read-only,
           write-only and mixed read/write streams)
  cpu_baseline the CPU oracle timed on the host over a bounded sample
  configs  (without --workload) the same figures, compact, for each of the
           five workloads; the top-level line is the multi-tenant workload

Usage: python bench.py [--steps K] [--warmup W] [--workload NAME]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# Sources that decide what the measured kernel reads and writes: the kernel
# itself and the host code that builds its schedule and tables.
KERNEL_SOURCES = ["paper_1805_07891_amd/csrc/fused_step.hip", "paper_1805_07891_amd/csrc/kernels.hpp",
                  "paper_1805_07891_amd/csrc/plan.cpp", "paper_1805_07891_amd/csrc/plan.hpp",
                  "paper_1805_07891_amd/csrc/phub_api.cpp"]
HEADLINE_WORKLOAD = "multitenant"
# The memory-side cache of MI355X, given to --pushpull jobs by default.
PUSHPULL_CACHE_BYTES = 256 << 20


def _code_only(text: str) -> str:
    """C++ source without comments and blank space, so that the hash follows
    the code and not its commentary."""
    out, i, n = [], 0, len(text)
    while i < n:
        if text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
        elif text[i] == '"':
            j = i + 1
            while j < n and text[j] != '"':
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        else:
            out.append(text[i])
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel)) as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per step (all of the step's launches) from the committed
    counter summary, if it was taken on the kernel as it is now (same source
    hash); else None."""
    path = os.path.join(ROOT, "profiles", f"fused_step_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None
    return rec.get("bytes_per_step")


NOTES = {
    "tiny": "cache-resident and launch-bound: 26.5 MB per step (3.3 us at peak) fits in the "
            "256 MiB memory-side cache, and back-to-back kernels on one stream start about "
            "0.95 us apart on MI355X; host_us_per_step is the time in the push and step "
            "calls, which over many steps includes waiting for a full launch queue",
}


def _probe_lib():
    import ctypes
    from paper_1805_07891_amd import build as hip_build
    if not os.path.exists(hip_build.PROBE_LIB):
        raise RuntimeError(f"{hip_build.PROBE_LIB} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(hip_build.PROBE_LIB)
    vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float
    pp = ctypes.POINTER(ctypes.c_void_p)
    lib.phub_probe_read.argtypes = [pp, i32, i64, i32, f32, vp, vp]
    lib.phub_probe_write.argtypes = [pp, i32, i64, i32, f32, vp]
    lib.phub_probe_mixed.argtypes = [pp, i32, pp, i32, i64, i32, f32, vp, vp]
    for f in (lib.phub_probe_read, lib.phub_probe_write, lib.phub_probe_mixed):
        f.restype = i32
    lib.phub_probe_tile_elems.restype = i32
    return lib


def ceilings(torch, dev, grads, num_states: int, stream, reps: int = 5):
    """HBM ceilings measured in the same run over the dominant job's buffers
    (best of `reps` passes each, GB/s): the bandwidth probes reading its N
    gradient arenas (read-only), writing S scratch arenas of the same size
    (write-only), and reading the N arenas while reading and writing back
    the S scratch arenas in place, tile by tile (the step's (N + S) : S mix of
    reads and writes without its arithmetic or the timing of its writes).
    Also the phase-separated bound: the step's bytes if its reads ran at the
    read ceiling and its writes at the write ceiling, one after the other."""
    import ctypes
    lib = _probe_lib()
    tile = lib.phub_probe_tile_elems()
    n = min(a.numel() for a in grads) // tile * tile
    scratch = [torch.zeros(n, dtype=torch.float32, device=dev) for _ in range(num_states)]
    grid = torch.cuda.get_device_properties(dev).multi_processor_count
    sink = torch.empty(grid * 256, dtype=torch.float32, device=dev)
    gp = (ctypes.c_void_p * len(grads))(*[a.data_ptr() for a in grads])
    sp = (ctypes.c_void_p * num_states)(*[a.data_ptr() for a in scratch])
    sv = ctypes.c_void_p(stream.cuda_stream)
    sk = ctypes.c_void_p(sink.data_ptr())
    runs = {
        "read": (lambda: lib.phub_probe_read(gp, len(grads), n, grid, -1.2345678e30, sk, sv),
                 len(grads) * n * 4),
        "write": (lambda: lib.phub_probe_write(sp, num_states, n, grid, 0.0, sv),
                  num_states * n * 4),
        "mixed": (lambda: lib.phub_probe_mixed(gp, len(grads), sp, num_states, n, grid,
                                               -1.2345678e30, sk, sv),
                  (len(grads) + 2 * num_states) * n * 4),
    }
    torch.cuda.synchronize()
    best = {}
    for name, (run, nbytes) in runs.items():
        b = 0.0
        for _ in range(reps + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            rc = run()
            e1.record(stream)
            if rc != 0:
                raise RuntimeError(f"phub_probe_{name} failed: {rc}")
            torch.cuda.synchronize()
            b = max(b, nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e9)
        best[name] = b
    del scratch
    nr, nw = len(grads) + num_states, num_states
    phase = (nr + nw) / (nr / best["read"] + nw / best["write"])
    out = {k: {"GBps": round(v, 1), "frac_of_peak": round(v / HBM_PEAK_GBS, 4)} for k, v in best.items()}
    out["read"]["kind"] = "read-only non-temporal stream over the dominant job's gradient arenas"
    out["write"]["kind"] = f"write-only non-temporal stream over {num_states} arenas of the same size"
    out["mixed"]["kind"] = (f"the {len(grads)} gradient arenas read and {num_states} arenas read and "
                            f"written back in place, tile by tile ({nr}:{nw} reads:writes)")
    out["phase_separated"] = {"GBps": round(phase, 1), "frac_of_peak": round(phase / HBM_PEAK_GBS, 4),
                              "kind": "the step's reads at the read ceiling, then its writes at the "
                                      "write ceiling"}
    return out


def cu_masked_streams(torch, dev, wl):
    """(stream, compute units) per job: HIP streams restricted to disjoint
    sets of compute units, in proportion to each job's bytes per step (at
    least one each), wrapped as torch external streams."""
    import ctypes
    from paper_1805_07891_amd.job import hip_runtime
    hip = hip_runtime()
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    by = [j.hbm_bytes_per_step() for j in wl.jobs]
    share = [max(1, int(cus * b / sum(by))) for b in by]
    share[by.index(max(by))] += cus - sum(share)     # the rest to the largest job
    hip.hipExtStreamCreateWithCUMask.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint32,
                                                 ctypes.POINTER(ctypes.c_uint32)]
    hip.hipExtStreamCreateWithCUMask.restype = ctypes.c_int
    out, first = [], 0
    for n in share:
        words = (ctypes.c_uint32 * ((cus + 31) // 32))()
        for cu in range(first, first + n):
            words[cu // 32] |= 1 << (cu % 32)
        first += n
        handle = ctypes.c_void_p()
        rc = hip.hipExtStreamCreateWithCUMask(ctypes.byref(handle), len(words), words)
        if rc != 0:
            raise RuntimeError(f"hipExtStreamCreateWithCUMask failed: {rc}")
        out.append((torch.cuda.ExternalStream(handle.value, device=dev), n))
    return out


def span_of_steps(torch, dev, jobs, push, steps: int, helper, before=None):
    """Device time of one step of every job (ms; a list).  Without `before`:
    `steps` steps back to back between one pair of HIP events, on the job's
    stream for one job, else on a helper stream that every job stream waits
    on at the start and that waits on every job stream at the end (the
    tenants' launches overlap); one value, the average.  With `before`
    (e.g. a cache flush), called on each job's stream before each step,
    every step is timed on its own after its `before` work has completed;
    one value per step.  `helper` is a stream of its own (unused for one
    job)."""
    one = len(jobs) == 1
    if one:
        helper = jobs[0].stream
    ms = []
    for _ in range(steps if before is not None else 1):
        if before is not None:
            for job in jobs:
                with torch.cuda.stream(job.stream):
                    before()
                if not one:
                    done = torch.cuda.Event()
                    done.record(job.stream)
                    helper.wait_event(done)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(helper)
        if not one:
            for job in jobs:
                job.stream.wait_event(e0)
        for _ in range(1 if before is not None else steps):
            for job in jobs:
                push(job)
                job.step()
        if not one:
            for job in jobs:
                ev = torch.cuda.Event()
                ev.record(job.stream)
                helper.wait_event(ev)
        e1.record(helper)
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1) / (1 if before is not None else steps))
    return ms


def cold_steps(torch, dev, jobs, push, steps: int, step_bytes: int, helper):
    """The step with a cold memory-side cache: before each step, a 1 GiB
    buffer is read with ordinary (cache-allocating) loads on every job's
    stream, which replaces the 256 MiB cache's contents with clean lines, so
    that state cached by the previous step starts from HBM (and no dirty
    data of the flush is written back during the step).  Each step is timed
    on its own (span_of_steps), and so are as many steps after a read of a
    1-element buffer instead (isolated but warm), since an isolated step of
    concurrent tenants also loses the overlap of one step's tail with the
    next step's launches."""
    if steps <= 0:
        return None
    flush = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    tiny = torch.ones(1, dtype=torch.float32, device=dev)
    sink = torch.empty((), dtype=torch.float32, device=dev)
    cold = sorted(span_of_steps(torch, dev, jobs, push, steps, helper,
                                before=lambda: torch.sum(flush, 0, out=sink)))
    warm = sorted(span_of_steps(torch, dev, jobs, push, steps, helper,
                                before=lambda: torch.sum(tiny, 0, out=sink)))
    avg = sum(cold) / len(cold)
    wavg = sum(warm) / len(warm)
    del flush
    return {"kind": "memory-side cache flushed (1 GiB read) before each step, each step timed "
                    "on its own",
            "steps": steps, "avg_step_us": round(avg * 1e3, 2),
            "median_step_us": round(cold[len(cold) // 2] * 1e3, 2),
            "frac": round(step_bytes / (avg * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "isolated_warm_avg_step_us": round(wavg * 1e3, 2),
            "isolated_warm_frac": round(step_bytes / (wavg * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}


def cpu_baseline(wl, grads_dev, w0_dev, budget_s: float):
    """The oracle on the host, single-threaded, over the workload's first job
    (all keys) or a prefix of its keys, until `budget_s` seconds of work."""
    import numpy as np
    import oracle
    spec = wl.jobs[0]
    # bound host memory: take a prefix of keys with at most ~2 GB of inputs
    limit = 2e9 / ((spec.num_workers + 2) * 4)
    nkeys, acc = 0, 0
    for n in spec.key_elems:
        if acc + n > limit and nkeys > 0:
            break
        acc += n
        nkeys += 1
    from paper_1805_07891_amd.workloads import key_offsets
    offs, _ = key_offsets(spec.key_elems)
    g_host = [grads_dev[w].cpu().numpy() for w in range(spec.num_workers)]
    w_host = w0_dev.cpu().numpy()
    grads = [[g[o:o + n] for o, n in zip(offs[:nkeys], spec.key_elems[:nkeys])] for g in g_host]
    W = [w_host[o:o + n].copy() for o, n in zip(offs[:nkeys], spec.key_elems[:nkeys])]
    M = [np.zeros(n, np.float32) for n in spec.key_elems[:nkeys]]
    try:
        cores = os.sched_getaffinity(0)
        os.sched_setaffinity(0, {min(cores)})
    except (AttributeError, OSError):
        cores = None
    steps, t0 = 0, time.perf_counter()
    try:
        while True:
            oracle.step(grads, W, M, spec.lr, spec.momentum, spec.weight_decay, spec.nesterov)
            steps += 1
            if time.perf_counter() - t0 >= budget_s:
                break
    finally:
        if cores is not None:
            os.sched_setaffinity(0, cores)
    dt = time.perf_counter() - t0
    params = sum(spec.key_elems[:nkeys])
    return {
        "value": round(spec.num_workers * params * 4 * steps / dt / 1e9, 3),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"{spec.name}: {nkeys} of {spec.num_keys} keys ({params:,} of "
                   f"{spec.num_params:,} params), N={spec.num_workers}, {steps} steps in "
                   f"{dt:.1f} s, one thread pinned to one core"),
        "host_cpus": os.cpu_count(),
        "host_cpu_model": cpu_model(),
    }


def readiness_groups(spec, bucket_bytes: float):
    """Keys grouped in backward order (last key first) into runs of at
    least `bucket_bytes` of fp32 gradient per worker; group 0 holds the last
    keys, which the backward pass produces first."""
    group = [0] * spec.num_keys
    g, acc = 0, 0
    for k in reversed(range(spec.num_keys)):
        group[k] = g
        acc += spec.key_elems[k] * 4
        if acc >= bucket_bytes:
            g, acc = g + 1, 0
    return group, g + (1 if acc > 0 else 0)


def streaming_bench(torch, dev, lib, wl, args) -> int:
    """The step overlapped with a simulated backward pass that produces the
    gradients (sections 3.2.2-3.2.3: a chunk is aggregated as soon as all of
    its pieces have arrived).  Every worker has its own stream and delivers its keys in
    backward order (last key first), in buckets of --producer-mb, one event
    per bucket; the host pushes each bucket's keys with that event at once.
    Each bucket is first computed on the same GPU (bf16 GEMMs proportional
    to the bucket's parameters: the layers' backward work), then written.
    With --arrival link, the buckets instead arrive through one ingress
    stream at N times --link-gbps (a sleep kernel paces them, then they are
    copied into place as a network card's DMA would).  For one launch at
    phub_step and for readiness groups of --bucket-mb launched as they
    complete, the exposed time is measured within each run on the device:
    the end of the step minus the end of the last producer's work.""" 
    import statistics
    from paper_1805_07891_amd import workloads
    from paper_1805_07891_amd.job import TorchJob
    spec = wl.jobs[0]
    N, K = spec.num_workers, spec.num_keys
    key_group, ngroups = readiness_groups(spec, args.bucket_mb * 1e6)
    prod_group, nprod = readiness_groups(spec, args.producer_mb * 1e6)
    buckets = [[k for k in range(K) if prod_group[k] == b] for b in range(nprod)]
    dim, mrows = 4096, 1024                       # one fixed GEMM shape for every bucket
    flop_per_mm = 2.0 * mrows * dim * dim
    n_mm = [max(1, int(round(args.backward_tflop * 1e12 * sum(spec.key_elems[k] for k in b)
                             / spec.num_params / flop_per_mm))) for b in buckets]
    weight = torch.randn(dim, dim, device=dev, dtype=torch.bfloat16)
    acts = [torch.randn(mrows, dim, device=dev, dtype=torch.bfloat16) for _ in range(N)]
    link = args.arrival == "link"
    # link arrival: one ingress stream.  Streams share the process's few
    # hardware queues in creation order, so the run creates no stream it does
    # not use (a job's stream sharing a queue with the ingress would run its
    # launches in line with the arrivals).
    producers = [torch.cuda.Stream(device=dev) for _ in range(1 if link else N)]
    sleep_cycles = []
    if link:
        # calibrate the sleep kernel: cycles per microsecond of device time
        cal = producers[0]
        rates = []
        for _ in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            with torch.cuda.stream(cal):
                e0.record(cal)
                torch.cuda._sleep(1 << 22)
                e1.record(cal)
            torch.cuda.synchronize()
            rates.append((1 << 22) / (e0.elapsed_time(e1) * 1e3))
        per_us = statistics.median(rates)
        # one ingress for all workers (the server's network), N links' worth of rate:
        # a bucket of every worker arrives in its bytes / (N * link rate)
        link_bytes_per_us = args.link_gbps * 1e9 / 8 / 1e6
        sleep_cycles = [max(1, int(4 * sum(spec.key_elems[k] for k in b) / link_bytes_per_us * per_us))
                        for b in buckets]
    src = [workloads.device_grad_arena(torch, dev, spec, wl.seed_index, 0, 0, w) for w in range(N)]
    w0 = workloads.device_weight_arena(torch, dev, spec, wl.seed_index, 0)

    jobs = {}
    for mode, kg in (("one_launch", None), ("groups", key_group)):
        # each worker's bucket events are recorded on its own producer stream,
        # in push order
        job = TorchJob(spec, dev, lib=lib, key_group=kg, ordered_events=not args.unordered_events)
        job.set_weights(w0)
        arenas = [torch.zeros_like(src[w]) for w in range(N)]
        for w in range(N):
            job.attach_grads(w, arenas[w])
        pushes = [[job.bucket(w, b) for b in buckets] for w in range(N)]
        jobs[mode] = (job, arenas, pushes)
    offs, arena_elems = workloads.key_offsets(spec.key_elems)
    bounds = []
    for b in buckets:
        lo = offs[min(b)]
        hi = offs[max(b) + 1] if max(b) + 1 < K else arena_elems
        bounds.append((lo, hi))
    torch.cuda.synchronize()

    def backward(job, arenas, pushes):
        start = torch.cuda.Event(enable_timing=True)
        start.record(producers[0])
        for p in producers[1:]:
            p.wait_event(start)
        events = []
        arrived = []   # per producer stream: timed marker after its last bucket
        last = len(buckets) - 1
        for bi in range(len(buckets)):
            lo, hi = bounds[bi]
            if link:
                # the ingress stream delivers bucket bi of every worker, then one event
                with torch.cuda.stream(producers[0]):
                    torch.cuda._sleep(sleep_cycles[bi])
                    for w in range(N):
                        arenas[w][lo:hi].copy_(src[w][lo:hi])
                    ev = torch.cuda.Event(enable_timing=bi == last)
                    ev.record(producers[0])
                events.append(ev)
                if bi == last:
                    arrived.append(ev)
                if pushes is not None:
                    for w in range(N):
                        job.push_bucket(w, pushes[w][bi], ev)
                continue
            for w in range(N):
                with torch.cuda.stream(producers[w]):
                    for _ in range(n_mm[bi]):
                        torch.mm(acts[w], weight)
                    arenas[w][lo:hi].copy_(src[w][lo:hi])
                    ev = torch.cuda.Event(enable_timing=bi == last)
                    ev.record(producers[w])
                events.append(ev)
                if bi == last:
                    arrived.append(ev)
                if pushes is not None:
                    job.push_bucket(w, pushes[w][bi], ev)
        return start, arrived

    def run(mode, reps):
        """(start to end, last arrival to end) in us for each repetition."""
        out = []
        for _ in range(reps):
            job, arenas, pushes = jobs["one_launch"] if mode == "backward_only" else jobs[mode]
            # arrived: the end of every producer stream's work, recorded before
            # the push that may enqueue the last group
            start, arrived = backward(job, arenas, None if mode == "backward_only" else pushes)
            end = torch.cuda.Event(enable_timing=True)
            if mode == "backward_only":
                for p in producers[1:]:
                    producers[0].wait_stream(p)
                end.record(producers[0])
            else:
                job.step()
                end.record(job.stream)
            torch.cuda.synchronize()
            out.append((start.elapsed_time(end) * 1e3,
                        min(e.elapsed_time(end) for e in arrived) * 1e3))
        return out

    print(f"streaming: {wl.name}, {N} workers, {len(buckets)} buckets per worker, "
          + (f"arriving at {args.link_gbps} Gb/s per worker" if link else
             f"{sum(n_mm)} GEMMs of {mrows}x{dim}x{dim}")
          + f", {ngroups} readiness groups", file=sys.stderr, flush=True)
    for mode in ("backward_only", "one_launch", "groups"):
        print(f"streaming: warm-up {mode}", file=sys.stderr, flush=True)
        run(mode, 3)
    reps = max(5, args.steps // 25)
    t = {m: [] for m in ("backward_only", "one_launch", "groups")}
    after = {m: [] for m in ("one_launch", "groups")}
    for r in range(reps):                       # interleaved, so drift hits every mode
        for m in t:
            total, tail = run(m, 1)[0]
            t[m].append(total)
            if m in after:
                after[m].append(tail)
        print(f"streaming: rep {r + 1}/{reps}: " + ", ".join(f"{m} {v[-1]:.0f} us" for m, v in t.items())
              + "; after the last arrival: " + ", ".join(f"{m} {v[-1]:.0f} us" for m, v in after.items()),
              file=sys.stderr, flush=True)
    med = {m: statistics.median(v) for m, v in t.items()}
    med_after = {m: statistics.median(v) for m, v in after.items()}
    out = {
        "metric": ("exchange time exposed after the last gradient arrives (step end - arrival end)"
                   if link else
                   "exchange time exposed after the backward pass (step end - backward end)"),
        "value": round(med_after["groups"], 1),
        "unit": "us",
        "higher_is_better": False,
        "n_gpus": 1,
        "reps": reps,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "job": spec.name, "workers": N, "keys": K,
                   "params": spec.num_params, "readiness_groups": ngroups,
                   "bucket_mb": args.bucket_mb, "producer_buckets": nprod,
                   "producer_mb": args.producer_mb,
                   "ordered_events": not args.unordered_events,
                   **({"arrival": "link", "link_gbps_per_worker": args.link_gbps}
                      if link else
                      {"arrival": "gemm", "gemm": [mrows, dim, dim],
                       "bf16_tflop_per_worker": args.backward_tflop})},
        "median_us": {m: round(v, 1)
                      for m, v in med.items()},
        "min_us": {m: round(min(v), 1)
                   for m, v in t.items()},
        # measured within each run: step end - end of the last producer's work
        "exposed_us": {m: round(v, 1) for m, v in med_after.items()},
        # difference of medians over separate runs (noisier: producer time varies)
        "total_minus_producers_only_us": {m: round(med[m] - med["backward_only"], 1)
                                          for m in ("one_launch", "groups")},
    }
    print(json.dumps(out), flush=True)
    for job, _, _ in jobs.values():
        job.destroy()
    return 0


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default=None,
                    help="one workload (tiny, resnet50, alexnet, resnet269, multitenant); "
                         "default: all five, the multi-tenant one as the headline")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="budget of the CPU oracle baseline of the headline workload (0 skips it)")
    ap.add_argument("--config-cpu-seconds", type=float, default=2.0,
                    help="budget of the CPU oracle baseline of each other workload (0 skips it)")
    ap.add_argument("--min-timed-ms", type=float, default=0.0,
                    help="time at least this long: more than --steps steps where a step is "
                         "short (the five-workload run passes 50 to every workload but the "
                         "headline, which always times exactly --steps)")
    ap.add_argument("--chunk-bytes", type=int, default=None,
                    help="chunk size of the schedule (default: the workload's, 32 KB)")
    ap.add_argument("--schedule", choices=("lpt", "split", "dynamic"), default="lpt",
                    help="chunk-to-wave schedule: the paper's balanced partition (lpt), "
                         "contiguous, exactly balanced runs (split), or lpt with the streamed "
                         "tiles taken by the waves from a shared counter (dynamic)")
    ap.add_argument("--whole-chunks", action="store_true",
                    help="ablation: chunks of --chunk-bytes are indivisible items of the "
                         "schedule, as in the paper (by default they are split while there are "
                         "fewer than 128 items per wave)")
    ap.add_argument("--library", default=None,
                    help="ablation: run the step from another build of the library, e.g. "
                         "paper_1805_07891_amd/libphub_gradients_cached.so (gradients loaded "
                         "cache-allocating; python -m paper_1805_07891_amd.build "
                         "--gradients-cached builds it)")
    ap.add_argument("--resident-bytes", type=int, default=None,
                    help="per-job budget for keeping W and M in the memory-side cache "
                         "(library default if omitted)")
    ap.add_argument("--optimizer", choices=("momentum", "sgd", "adam"), default="momentum",
                    help="the pluggable optimizer (default: the workload's Nesterov momentum)")
    ap.add_argument("--pushpull", action="store_true",
                    help="every worker also receives the updated weights in its own model "
                         "buffer, written by the same fused pass (PushPull)")
    ap.add_argument("--unfused", action="store_true",
                    help="ablation: the step as two launches (sum into a merge buffer, then "
                         "the optimizer); roofline bytes stay the fused method's")
    ap.add_argument("--streaming", action="store_true",
                    help="instead of the throughput line: time the step overlapped with a "
                         "simulated backward pass, one launch vs readiness groups")
    ap.add_argument("--bucket-mb", type=float, default=25.0,
                    help="readiness group size for --streaming (MB of fp32 gradient per worker)")
    ap.add_argument("--arrival", choices=("gemm", "link"), default="gemm",
                    help="--streaming: how gradients become ready: computed by a simulated "
                         "backward on the same GPU (gemm), or arriving at a fixed link rate per "
                         "worker, paced by a sleep kernel then copied into place as a network "
                         "card's DMA would (link)")
    ap.add_argument("--link-gbps", type=float, default=56.0,
                    help="--streaming --arrival link: per-worker link rate in Gb/s (the paper's "
                         "InfiniBand interfaces run at 56); all workers' buckets arrive through "
                         "one ingress stream at N times that rate")
    ap.add_argument("--unordered-events", action="store_true",
                    help="--streaming: do not tell the library that each worker's events are "
                         "ordered on its stream (every distinct event is then waited for)")
    ap.add_argument("--backward-tflop", type=float, default=1.0,
                    help="--streaming: simulated backward work per worker (bf16 TFLOP)")
    ap.add_argument("--producer-mb", type=float, default=8.0,
                    help="--streaming: the simulated backward writes its gradients in buckets "
                         "of this many MB per worker, one event each")
    ap.add_argument("--workgroups", type=int, default=None,
                    help="ablation: workgroups of each launch (default one per compute unit, "
                         "persistent); a value of at least a quarter of the job's tiles gives "
                         "every wave at most one item, the non-persistent form")
    ap.add_argument("--cold-steps", type=int, default=20,
                    help="after the timed steps, this many more with the memory-side cache "
                         "flushed before each job's step (a 1 GiB read); reported as "
                         "roofline.cold (0 skips)")
    ap.add_argument("--cu-masks", action="store_true",
                    help="ablation for multi-job workloads: each job on its own stream restricted "
                         "to a disjoint set of compute units in proportion to its bytes, with a "
                         "persistent grid of that many workgroups")
    ap.add_argument("--shared-stream", action="store_true",
                    help="multi-job workloads: the jobs share one stream and take turns, each "
                         "launch with the whole GPU (default: each job on its own stream, its "
                         "launches concurrent with the other jobs')")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 512 MiB device copy three times (a known-size "
                         "reference for hardware byte counters)")
    args = ap.parse_args(argv)

    if args.streaming and "GPU_MAX_HW_QUEUES" not in os.environ:
        # one hardware queue per stream (set before the HIP runtime starts):
        # producer streams that shared a queue with the job's stream would run
        # its launches in line with their own work
        os.environ["GPU_MAX_HW_QUEUES"] = "16"

    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the exchange step here runs on a single "
              f"MI355X with all workers simulated in its HBM; --gpus {args.gpus} is not "
              f"supported.", file=sys.stderr)
        return 2

    if not args.workload and not args.streaming:
        return run_all(args, argv if argv is not None else sys.argv[1:])

    import torch
    from paper_1805_07891_amd import workloads
    from paper_1805_07891_amd.job import load_library

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    lib = load_library(os.path.abspath(args.library) if args.library else None)

    if args.streaming:
        return streaming_bench(torch, dev, lib, workloads.workload(args.workload or "resnet50"),
                               args)

    if args.copy_calibration:
        src = torch.ones(128 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    wl = workloads.workload(args.workload)
    # The streams, created first: one per job, then a helper for timing
    # events and probes.
    streams = [torch.cuda.Stream(device=dev) for _ in wl.jobs]
    helper = torch.cuda.Stream(device=dev)
    line = measure(torch, dev, lib, wl, args, args.cpu_seconds, streams, helper)
    print(json.dumps(line), flush=True)
    return 0


# Flags main() handles itself and does not pass on to a workload's process.
_OWN_FLAGS = {"--workload": 1, "--cpu-seconds": 1, "--config-cpu-seconds": 1, "--min-timed-ms": 1}

# Shortest timed region of the workloads other than the headline: with the
# driver's 20 steps the tiny workload's 5 us steps make 0.1 ms of work, and
# the two synchronisations around it (about 3 us each, plus the queue's
# start) would count as a third of it.
CONFIG_MIN_TIMED_MS = 50.0


def child_args(argv) -> list:
    """The command-line arguments a workload's process gets from the parent:
    all but the flags the parent handles itself (with their values, given
    as `--flag value` or `--flag=value`)."""
    passed = []
    i = 0
    while i < len(argv):
        a = argv[i]
        flag = a.split("=", 1)[0]
        if flag in _OWN_FLAGS:
            i += 1 if "=" in a else 1 + _OWN_FLAGS[flag]
            continue
        passed.append(a)
        i += 1
    return passed


def run_all(args, argv) -> int:
    """The five workloads, each measured by this script in a process of its
    own (this process never touches the GPU).  Measured in one process one
    after another, every workload after the first lost 1.5-3 points (the
    multi-tenant step 77.4% -> 75.9% -> 75.2% on three runs in a row,
    ResNet-269 81.5% -> 79.0% after the multi-tenant run), whatever the
    order: memory freed by one workload and allocated by the next is laid
    out differently.  A job of a training run starts in a fresh process, so
    each workload is measured in one.  The line printed is the headline
    (multi-tenant) workload's, with every workload's compact figures under
    "configs"."""
    import subprocess
    from paper_1805_07891_amd import workloads
    passed = child_args(argv)
    lines = {}
    for name in workloads.WORKLOAD_NAMES:
        budget = args.cpu_seconds if name == HEADLINE_WORKLOAD else args.config_cpu_seconds
        cmd = [sys.executable, "-u", os.path.abspath(__file__), "--workload", name,
               "--cpu-seconds", str(budget), *passed]
        if name != HEADLINE_WORKLOAD:
            cmd += ["--min-timed-ms", str(CONFIG_MIN_TIMED_MS)]
        print(f"bench: {name}", file=sys.stderr, flush=True)
        r = subprocess.run(cmd, stdout=subprocess.PIPE, text=True)
        if r.returncode != 0:
            print(f"bench: {name} failed with status {r.returncode}", file=sys.stderr, flush=True)
            return r.returncode
        lines[name] = json.loads(r.stdout.strip().splitlines()[-1])
    out = lines[HEADLINE_WORKLOAD]
    out["configs"] = {n: compact(lines[n]) for n in workloads.WORKLOAD_NAMES}
    out["configs_kind"] = "each workload measured by bench.py --workload NAME in a process of its own"
    print(json.dumps(out), flush=True)
    return 0


def compact(line: dict) -> dict:
    """The figures of one workload's line that the five-workload summary
    keeps."""
    r, c = line["roofline"], line["config"]
    cold, ceil, base = r.get("cold"), r["ceilings"], line.get("cpu_baseline")
    step_bytes = r["algorithmic_bytes_per_launch"]
    return {
        "ms_per_step": line["ms_per_step"],
        "value_GBps": line["value"],
        "whole_step_pct": c["hbm_pct_of_peak_whole_step"],
        "kernel_frac": r["frac"],
        "kernel_frac_cold": cold["frac"] if cold else None,
        "kernel_frac_isolated_warm": cold["isolated_warm_frac"] if cold else None,
        "state_cached_fraction": [j["state_cached_fraction"] for j in c["jobs"]],
        "read_ceiling_frac": ceil["read"]["frac_of_peak"],
        "mixed_ceiling_frac": ceil["mixed"]["frac_of_peak"],
        "phase_separated_frac": ceil["phase_separated"]["frac_of_peak"],
        "frac_of_mixed_ceiling": r["frac_of_mixed_ceiling"],
        "traffic_over_algorithmic": (round(r["traffic"] / step_bytes, 4) if r["traffic"] else None),
        "host_us_per_step": c["host_us_per_step"],
        "cpu_baseline_GBps": base["value"] if base else None,
        "cpu_sample": base["sample"] if base else None,
        **({"note": c["note"]} if c.get("note") else {}),
    }


def measure(torch, dev, lib, wl, args, cpu_seconds: float, streams, helper) -> dict:
    """One workload: set-up, warm-up, the timed steps, kernel timing,
    ceilings, cold-cache steps and the CPU baseline.  Job j runs on
    streams[j] (all on streams[0] with --shared-stream); `helper` carries
    the timing events of several jobs and the probes.  Returns the JSON
    line."""
    from paper_1805_07891_amd import workloads
    from paper_1805_07891_amd.job import TorchJob
    from paper_1805_07891_amd.phub import PHUB_SCHEDULE_DYNAMIC, PHUB_SCHEDULE_SPLIT

    # Co-running jobs each have their own stream (their launches run
    # concurrently); with --shared-stream they take turns on one stream,
    # each launch with the whole GPU.
    shared_stream = len(wl.jobs) > 1 and args.shared_stream
    masked = cu_masked_streams(torch, dev, wl) if args.cu_masks and len(wl.jobs) > 1 else None
    jobs, grads, w0s = [], [], []
    for ji, spec in enumerate(wl.jobs):
        stream = streams[0] if shared_stream else streams[ji]
        if masked is not None:
            stream = masked[ji][0]
        # pushpull's kernels have no burst write-back: its jobs cache their
        # state (256 MiB shared among the jobs) unless told otherwise
        resident = args.resident_bytes
        if resident is None and args.pushpull:
            resident = PUSHPULL_CACHE_BYTES // len(wl.jobs)
        job = TorchJob(spec, dev, stream=stream, lib=lib, resident_bytes=resident,
                       chunk_bytes=args.chunk_bytes, unfused=args.unfused,
                       optimizer=None if args.optimizer == "momentum" else args.optimizer,
                       schedule={"lpt": None, "split": PHUB_SCHEDULE_SPLIT,
                                 "dynamic": PHUB_SCHEDULE_DYNAMIC}[args.schedule],
                       workgroups=masked[ji][1] if masked is not None else args.workgroups,
                       whole_chunks=args.whole_chunks)
        w0 = workloads.device_weight_arena(torch, dev, spec, wl.seed_index, ji)
        g = [workloads.device_grad_arena(torch, dev, spec, wl.seed_index, ji, 0, w)
             for w in range(spec.num_workers)]
        torch.cuda.synchronize()
        job.set_weights(w0)
        for w, a in enumerate(g):
            job.attach_grads(w, a)
        if args.pushpull:
            for w in range(spec.num_workers):
                job.attach_models(w, torch.empty_like(w0))
        jobs.append(job)
        grads.append(g)
        w0s.append(w0)
    torch.cuda.synchronize()

    def push(job):
        if args.pushpull:
            job.pushpull_all()
        else:
            job.push_all()

    for _ in range(args.warmup):
        for job in jobs:
            push(job)
            job.step()
    torch.cuda.synchronize()

    K = args.steps
    if args.min_timed_ms > 0:
        # the step's time, from 50 more untimed steps
        tw = time.perf_counter()
        for _ in range(50):
            for job in jobs:
                push(job)
                job.step()
        torch.cuda.synchronize()
        est_ms = (time.perf_counter() - tw) * 1e3 / 50
        K = max(K, int(args.min_timed_ms / max(est_ms, 1e-4)) + 1)
    # Timed region: K steps of every job, wall clock between two device
    # synchronizations, with nothing else on the streams.
    torch.cuda.synchronize()
    host_s = 0.0
    t0 = time.perf_counter()
    for s in range(K):
        h0 = time.perf_counter()
        for job in jobs:
            push(job)
            job.step()
        host_s += time.perf_counter() - h0
    torch.cuda.synchronize()
    t1 = time.perf_counter()

    # Each job's launches: K more steps with HIP events recorded on each
    # job's stream around its phub_step (kept out of the wall-clock loop
    # above, where the event records would add their own time to small
    # steps).
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(K)] for _ in jobs]
    for s in range(K):
        for j, job in enumerate(jobs):
            push(job)
            ev[j][s][0].record(job.stream)
            job.step()
            ev[j][s][1].record(job.stream)
    torch.cuda.synchronize()

    states = {"momentum": 2, "sgd": 1, "adam": 3}[args.optimizer]

    def job_bytes(spec):
        # N gradient reads, each state array read and written, and with
        # pushpull w' written once more per worker
        return (spec.num_workers + 2 * states) * spec.num_params * 4 + \
            (spec.worker_grad_bytes_per_step() if args.pushpull else 0)

    ms_per_step = (t1 - t0) * 1e3 / K
    worker_bytes = wl.worker_grad_bytes_per_step()
    value = worker_bytes / (ms_per_step * 1e-3) / 1e9
    step_bytes = sum(job_bytes(j) for j in wl.jobs)
    whole_hbm = step_bytes / (ms_per_step * 1e-3) / 1e9

    # The kernel: the step's launches of the fused kernel (one per job),
    # K steps back to back between one pair of HIP events; with several
    # jobs on their own streams the launches overlap, and the span covers
    # all of them (span_of_steps).  An event pair around every launch adds
    # 2-5 us to each, so the per-launch events above serve only for the
    # spread and for each job's share.
    # at least 50 ms of launches, so that tiny's microsecond launches are not
    # dominated by the two events' own cost
    span_steps = max(K, int(50.0 / max(ms_per_step, 1e-3)))
    avg_ms = sum(span_of_steps(torch, dev, jobs, push, span_steps, helper))
    per_job = []
    for j, spec in enumerate(wl.jobs):
        d = sorted(ev[j][s][0].elapsed_time(ev[j][s][1]) for s in range(K))
        jm = sum(d) / K
        per_job.append({"job": spec.name, "avg_launch_us": round(jm * 1e3, 2),
                        "median_launch_us": round(d[K // 2] * 1e3, 2),
                        "min_launch_us": round(d[0] * 1e3, 2),
                        "frac": round(job_bytes(spec) / (jm * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)})
    achieved = step_bytes / (avg_ms * 1e-3) / 1e9
    dom = max(range(len(jobs)), key=lambda j: job_bytes(wl.jobs[j]))
    traffic = (None if (args.pushpull or args.unfused or args.optimizer != "momentum" or
                        args.resident_bytes is not None or args.shared_stream or args.cu_masks or
                        args.whole_chunks or args.schedule != "lpt" or args.chunk_bytes or
                        args.library)
               else measured_traffic(wl.name))
    groups, threads, segs, _, _ = jobs[dom].info()
    cached = [job.cached_fraction() for job in jobs]
    n_any = any(not (s.num_workers <= 16 or s.num_workers in (20, 24, 32)) for s in wl.jobs)
    kernel = ("aggregate_only + optimize_only" if args.unfused else
              "fused_step_any" if n_any else "fused_step_fixed")
    if len(jobs) > 1:
        kernel += (f" x{len(jobs)} (one launch per job, " +
                   ("taking turns on one stream)" if shared_stream else "concurrent on their own streams)"))

    ceil = ceilings(torch, dev, grads[dom], states, helper)
    cold = cold_steps(torch, dev, jobs, push, args.cold_steps, step_bytes, helper)

    baseline = None
    if cpu_seconds > 0:
        baseline = cpu_baseline(wl, grads[0], w0s[0], cpu_seconds)

    frac = achieved / HBM_PEAK_GBS
    line = {
        "metric": "worker-gradient GB/s aggregated+optimized per step; % of HBM peak",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": wl.name,
            "jobs": [{"name": j.name, "workers": j.num_workers, "keys": j.num_keys,
                      "params": j.num_params, "state_cached_fraction": round(r, 4)}
                     for j, r in zip(wl.jobs, cached)],
            "chunk_bytes": args.chunk_bytes or wl.jobs[0].chunk_bytes,
            "schedule": args.schedule,
            "whole_chunks": args.whole_chunks,
            "workgroups_option": args.workgroups,
            "optimizer": ({"lr": wl.jobs[0].lr, "momentum": wl.jobs[0].momentum,
                           "weight_decay": wl.jobs[0].weight_decay, "nesterov": wl.jobs[0].nesterov}
                          if args.optimizer == "momentum" else
                          {"kind": args.optimizer, "lr": wl.jobs[0].lr,
                           "weight_decay": wl.jobs[0].weight_decay,
                           **({"betas": [0.9, 0.999], "eps": 1e-8} if args.optimizer == "adam" else {})}),
            "hbm_bytes_per_step": step_bytes,
            "pushpull": args.pushpull,
            "optimizer_kind": args.optimizer,
            "unfused": args.unfused,
            "library": args.library or "paper_1805_07891_amd/libphub.so",
            "streams": ("one shared by the jobs" if shared_stream else
                        "one per job, CU-masked" if masked is not None else
                        "one per job" if len(wl.jobs) > 1 else "one"),
            **({"cu_per_job": [m[1] for m in masked]} if masked is not None else {}),
            "hbm_pct_of_peak_whole_step": round(100 * whole_hbm / HBM_PEAK_GBS, 2),
            "launch": {"workgroups": groups, "threads": threads, "segments": segs},
            "host_us_per_step": round(host_s * 1e6 / K, 2),
            "note": NOTES.get(wl.name, ""),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": kernel,
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(frac, 4),
            "traffic": traffic,
            "avg_launch_us": round(avg_ms * 1e3, 2),
            "avg_launch_us_kind": (f"{span_steps} launches back to back on the job's stream "
                                   "between one pair of HIP events" if len(jobs) == 1 else
                                   f"{span_steps} steps of every job back to back between one "
                                   "pair of HIP events that the job streams wait on and for; "
                                   "per step"),
            "per_job_events": per_job,
            "ceilings": ceil,
            "frac_of_read_ceiling": round(achieved / ceil["read"]["GBps"], 4),
            "frac_of_mixed_ceiling": round(achieved / ceil["mixed"]["GBps"], 4),
            "frac_of_phase_separated": round(achieved / ceil["phase_separated"]["GBps"], 4),
            "cold": cold,
            "algorithmic_bytes_per_launch": step_bytes,
            "kernel_source_hash": kernel_source_hash(),
        },
        "cpu_baseline": baseline,
    }
    for job in jobs:
        job.destroy()
    del grads, w0s
    return line


if __name__ == "__main__":
    sys.exit(main())
