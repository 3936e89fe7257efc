"""GPU parity of the fused exchange step against the CPU oracle.

Every test drives the HIP library through its C interface (ctypes binding)
on seeded synthetic inputs and compares the job's master weights W and
momentum M with the oracle's, element by element.  The accumulation order
is pinned on both sides (ascending worker index) and both evaluate the same
fused multiply-adds, so the bar is bit-exact equality; the 1e-6 relative
tolerance is reported alongside as a diagnostic.
"""

import os
import sys

import numpy as np
import pytest

import oracle
from paper_1805_07891_amd import phub, workloads
from paper_1805_07891_amd.job import TorchJob, load_library
from paper_1805_07891_amd.workloads import Job, key_offsets

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    return torch, torch.device("cuda:0")


@pytest.fixture(scope="module")
def lib(torch_dev):
    return load_library()


def _bits_equal(a, b):
    return np.array_equal(np.asarray(a, np.float32).view(np.uint32),
                          np.asarray(b, np.float32).view(np.uint32))


def _rel_err(x, ref):
    ref = ref.astype(np.float64)
    if ref.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(ref ** 2)) or 1.0
    return float(np.max(np.abs(x.astype(np.float64) - ref) / np.maximum(np.abs(ref), rms)))


def run_small_case(torch, dev, lib, n_workers, key_elems, steps=2, chunk_bytes=32768,
                   lr=0.1, mu=0.9, wd=1e-4, nesterov=True, seed=0, push="keys",
                   reuse_buffers=False, stream=None, schedule=None, resident_bytes=None,
                   unfused=False, workgroups=None, whole_chunks=False):
    """Runs `steps` steps on the GPU and in the oracle; returns the job and
    per-step (gpu W, gpu M, oracle W, oracle M) lists per key."""
    spec = Job("case", n_workers, tuple(int(n) for n in key_elems), chunk_elems=chunk_bytes // 4,
               lr=lr, momentum=mu, weight_decay=wd, nesterov=nesterov, sigma_g=1e-2)
    job = TorchJob(spec, dev, stream=stream, chunk_bytes=chunk_bytes, lib=lib, schedule=schedule,
                   resident_bytes=resident_bytes, unfused=unfused, workgroups=workgroups,
                   whole_chunks=whole_chunks)
    offs, total = key_offsets(spec.key_elems)
    rng = np.random.default_rng(seed)
    w0 = np.zeros(total, np.float32)
    for o, n in zip(offs, spec.key_elems):
        w0[o:o + n] = rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
    job.set_weights(torch.from_numpy(w0).to(dev))
    W = [w0[o:o + n].copy() for o, n in zip(offs, spec.key_elems)]
    M = [np.zeros(n, np.float32) for n in spec.key_elems]
    dev_arenas = None
    results = []
    for t in range(steps):
        host = []
        for w in range(n_workers):
            a = np.zeros(total, np.float32)
            for o, n in zip(offs, spec.key_elems):
                a[o:o + n] = rng.standard_normal(n, dtype=np.float32) * np.float32(1e-2)
            host.append(a)
        if reuse_buffers and dev_arenas is not None:
            for w in range(n_workers):
                dev_arenas[w].copy_(torch.from_numpy(host[w]))
        else:
            dev_arenas = [torch.from_numpy(a).to(dev) for a in host]
            for w in range(n_workers):
                job.attach_grads(w, dev_arenas[w])
        torch.cuda.synchronize()
        if push == "keys":
            job.push_all()
        elif push == "per_worker":
            for w in reversed(range(n_workers)):
                lib.phub_push_keys(job.handle, w, job.key_pointers(dev_arenas[w]))
        elif push == "single_reversed":
            for k in reversed(range(spec.num_keys)):
                for w in reversed(range(n_workers)):
                    lib.phub_push(job.handle, w, k, job.key_pointers(dev_arenas[w])[k])
        else:
            raise ValueError(push)
        job.step()
        oracle.step([[h[o:o + n] for o, n in zip(offs, spec.key_elems)] for h in host],
                    W, M, lr, mu, wd, nesterov)
        Wg, Mg = job.state_arenas()
        results.append((job.split(Wg), job.split(Mg), [x.copy() for x in W], [x.copy() for x in M]))
    return job, results


def assert_parity(results, label=""):
    for t, (wg, mg, wo, mo) in enumerate(results):
        for k in range(len(wo)):
            if not _bits_equal(wg[k], wo[k]) or not _bits_equal(mg[k], mo[k]):
                raise AssertionError(
                    f"{label} step {t} key {k} (n={wo[k].size}): W rel err {_rel_err(wg[k], wo[k]):.3g}, "
                    f"M rel err {_rel_err(mg[k], mo[k]):.3g}; first W mismatch at "
                    f"{int(np.argmax(wg[k].view(np.uint32) != wo[k].view(np.uint32)))}")


def test_library_is_in_tree_and_shares_torchs_hip_runtime(lib, torch_dev):
    torch, dev = torch_dev
    torch.zeros(1, device=dev)
    with open("/proc/self/maps") as f:
        maps = f.read()
    hip = {line.split()[-1] for line in maps.splitlines() if "libamdhip64" in line}
    assert len(hip) == 1, f"more than one HIP runtime mapped: {hip}"
    phubs = {line.split()[-1] for line in maps.splitlines() if line.endswith("libphub.so")}
    assert phubs == {os.path.realpath(phub.DEFAULT_LIB)}, phubs


def test_tiny_workload_full_parity(lib, torch_dev):
    torch, dev = torch_dev
    wl = workloads.workload("tiny")
    spec = wl.jobs[0]
    _say("tiny: N", spec.num_workers, "K", spec.num_keys, "P", spec.num_params)
    job, res = run_small_case(torch, dev, lib, spec.num_workers, spec.key_elems, steps=wl.steps,
                              chunk_bytes=spec.chunk_bytes, lr=spec.lr, mu=spec.momentum,
                              wd=spec.weight_decay, nesterov=spec.nesterov, seed=1805)
    assert_parity(res, "tiny")
    job.destroy()


EDGE = [1, 2, 3, 4, 5, 7, 8, 15, 16, 17, 63, 64, 65, 1023, 1024, 1025, 8191, 8192, 8193,
        2 * 8192 + 3, 0, 3 * 8192]


@pytest.mark.parametrize("n_workers", [1, 2, 3, 5, 8, 11, 16, 17, 33])
@pytest.mark.parametrize("nesterov", [True, False])
def test_edge_shapes(lib, torch_dev, n_workers, nesterov):
    torch, dev = torch_dev
    _say("edge shapes N", n_workers, "nesterov", nesterov)
    job, res = run_small_case(torch, dev, lib, n_workers, EDGE, steps=2, nesterov=nesterov,
                              seed=100 + n_workers)
    assert_parity(res, f"N={n_workers}")
    job.destroy()


@pytest.mark.parametrize("hp", [dict(mu=0.0), dict(lr=0.0), dict(wd=0.0, mu=0.0),
                                dict(lr=0.5, mu=0.5, wd=0.25), dict(lr=-1.0, mu=0.99, wd=0.3)])
def test_hyperparameter_corners(lib, torch_dev, hp):
    torch, dev = torch_dev
    for nest in (True, False):
        job, res = run_small_case(torch, dev, lib, 4, [5, 8192, 10007], steps=2, nesterov=nest,
                                  seed=7, **hp)
        assert_parity(res, f"{hp} nesterov={nest}")
        job.destroy()


@pytest.mark.parametrize("whole_chunks", [False, True])
def test_chunk_size_does_not_change_results(lib, torch_dev, whole_chunks):
    torch, dev = torch_dev
    keys = [3, 100, 8192 * 3 + 5, 70000, 1]
    outs = []
    for cb in (16, 48, 4096, 32768, 1 << 22):
        _say("chunk bytes", cb, "whole chunks", whole_chunks)
        job, res = run_small_case(torch, dev, lib, 6, keys, steps=2, chunk_bytes=cb, seed=99,
                                  whole_chunks=whole_chunks)
        assert_parity(res, f"chunk={cb}")
        outs.append(res[-1][:2])
        job.destroy()
    for wg, mg in outs[1:]:
        for k in range(len(keys)):
            assert _bits_equal(wg[k], outs[0][0][k]) and _bits_equal(mg[k], outs[0][1][k])


@pytest.mark.parametrize("schedule", [phub.PHUB_SCHEDULE_SPLIT, phub.PHUB_SCHEDULE_LPT,
                                      phub.PHUB_SCHEDULE_DYNAMIC])
@pytest.mark.parametrize("resident", [0, 4096, 1 << 20, 8 * 150001, 1 << 40])
def test_schedule_and_cache_residency_do_not_change_results(lib, torch_dev, schedule, resident):
    torch, dev = torch_dev
    keys = [3, 100, 8192 * 3 + 5, 70000, 1, 4096, 333333]
    for n in (4, 8, 16, 19):
        _say("schedule", schedule, "resident", resident, "N", n)
        job, res = run_small_case(torch, dev, lib, n, keys, steps=2, seed=1000 + n,
                                  schedule=schedule, resident_bytes=resident)
        assert_parity(res, f"schedule={schedule} resident={resident} N={n}")
        job.destroy()


def test_push_order_and_single_pushes(lib, torch_dev):
    torch, dev = torch_dev
    keys = [17, 9000, 4]
    job, res = run_small_case(torch, dev, lib, 5, keys, steps=2, seed=5, push="single_reversed")
    assert_parity(res, "reversed single pushes")
    job.destroy()
    job, res = run_small_case(torch, dev, lib, 5, keys, steps=2, seed=5, push="per_worker")
    assert_parity(res, "one batched push per worker")
    job.destroy()


def test_push_all_checks_every_pointer_before_recording(lib, torch_dev):
    """phub_push_all validates all N * K entries first: a bad entry anywhere
    leaves nothing recorded, so the step is refused; a good table then
    steps."""
    torch, dev = torch_dev
    keys = (300, 1024, 5)
    spec = Job("pushall", 3, keys)
    job = TorchJob(spec, dev, lib=lib)
    arenas = [torch.zeros(job.arena_elems, device=dev) for _ in range(3)]
    table = [p for a in arenas for p in job.key_pointers(a)]
    bad = list(table)
    bad[-1] = table[-1] + 4                      # last entry misaligned
    assert lib.phub_push_all(job.handle, bad, check=False) == phub.PHUB_EINVAL
    assert "aligned" in lib.last_error()
    assert lib.phub_step(job.handle, check=False) == phub.PHUB_ENOTREADY
    assert lib.phub_push_all(job.handle, None, check=False) == phub.PHUB_EINVAL
    lib.phub_push_all(job.handle, table)
    lib.phub_step(job.handle)
    job.sync()
    job.destroy()


def test_reused_buffers_skip_pointer_upload(lib, torch_dev):
    torch, dev = torch_dev
    job, res = run_small_case(torch, dev, lib, 4, [1000, 20000], steps=3, seed=6,
                              reuse_buffers=True)
    assert_parity(res, "reused buffers")
    job.destroy()


def test_step_before_all_pushes_is_refused(lib, torch_dev):
    torch, dev = torch_dev
    spec = Job("nr", 3, (100, 200))
    job = TorchJob(spec, dev, lib=lib)
    arenas = [torch.randn(job.arena_elems, device=dev) for _ in range(3)]
    for w in range(3):
        job.attach_grads(w, arenas[w])
    W0, M0 = job.state_arenas()
    for w in range(2):
        lib.phub_push_keys(job.handle, w, job._ptr_arrays[w])
    lib.phub_push(job.handle, 2, 0, job.key_pointers(arenas[2])[0])
    assert lib.phub_step(job.handle, check=False) == phub.PHUB_ENOTREADY
    assert "worker 2" in lib.last_error() and "key 1" in lib.last_error()
    W1, M1 = job.state_arenas()
    assert _bits_equal(W0, W1) and _bits_equal(M0, M1)
    # completing the pushes makes the step go
    lib.phub_push(job.handle, 2, 1, job.key_pointers(arenas[2])[1])
    lib.phub_step(job.handle)
    job.sync()
    # after a step every pair counts as not pushed again
    assert lib.phub_step(job.handle, check=False) == phub.PHUB_ENOTREADY
    job.destroy()


def test_argument_errors_on_a_live_job(lib, torch_dev):
    torch, dev = torch_dev
    spec = Job("err", 2, (100, 0))
    job = TorchJob(spec, dev, lib=lib)
    buf = torch.zeros(1024, device=dev)
    p = buf.data_ptr()
    assert lib.phub_push(job.handle, 0, 0, p + 4, check=False) == phub.PHUB_EINVAL  # misaligned
    assert lib.phub_push(job.handle, 2, 0, p, check=False) == phub.PHUB_EINVAL      # worker
    assert lib.phub_push(job.handle, 0, 2, p, check=False) == phub.PHUB_EINVAL      # key
    assert lib.phub_push(job.handle, 0, 0, 0, check=False) == phub.PHUB_EINVAL      # null
    assert lib.phub_push(job.handle, 0, 1, 0, check=False) == phub.PHUB_OK          # empty key
    assert lib.phub_push_keys(job.handle, 1, [p, p + 4], check=False) == phub.PHUB_EINVAL
    assert lib.phub_push_keys(job.handle, 1, [p, p, p], check=False) == phub.PHUB_EINVAL
    h = job.handle
    job.destroy()
    assert lib.phub_step(h, check=False) == phub.PHUB_ESTATE
    assert lib.phub_destroy(h, check=False) == phub.PHUB_ESTATE


def test_all_keys_empty(lib, torch_dev):
    torch, dev = torch_dev
    spec = Job("empty", 2, (0, 0, 0))
    job = TorchJob(spec, dev, lib=lib)
    for w in range(2):
        for k in range(3):
            lib.phub_push(job.handle, w, k, 0)
    lib.phub_step(job.handle)
    job.sync()
    assert job.info()[0] == 0
    job.destroy()


def test_default_cache_budget_is_shared(lib, torch_dev):
    """Jobs created with the default option share a 256 MiB per-device
    budget for cache-resident optimizer state, first come first served: each
    takes what its state needs of what is left (a prefix of its arena,
    possibly partial); destroying a job gives its share back; an explicit
    budget is the job's own."""
    torch, dev = torch_dev
    MiB = 1 << 20
    elems = 75 << 18                     # W + M = 150 MiB, no arena padding
    spec = Job("budget", 1, (elems,))
    a = TorchJob(spec, dev, lib=lib)
    b = TorchJob(spec, dev, lib=lib)
    c = TorchJob(spec, dev, lib=lib, resident_bytes=1 << 40)
    d = TorchJob(spec, dev, lib=lib, resident_bytes=0)
    e = None
    try:
        assert a.info()[3] == 150 * MiB and a.info()[4] == 150 * MiB
        assert b.info()[4] == 106 * MiB  # what is left: 106 MiB = 13568 whole tiles
        assert c.info()[4] == 150 * MiB
        assert d.info()[4] == 0
        a.destroy()
        a = None
        e = TorchJob(spec, dev, lib=lib)
        assert e.info()[4] == 150 * MiB  # a's share came back
        e.destroy()
        e = None
        tiny = TorchJob(Job("budget.tiny", 1, (1000,)), dev, lib=lib)
        assert tiny.cached_fraction() == 1.0
        tiny.destroy()
        # jobs with burst write-back (momentum and plain SGD with 6-16, 20, 24
        # or 32 workers, Adam with 14-16, 20, 24 or 32) take none of the
        # default budget; the others, the any-N kernel (17 workers) and the
        # unfused variant cache
        for n, opt, want in ((6, "sgd", 0.0), (16, "sgd", 0.0), (5, "sgd", 1.0), (17, "sgd", 1.0),
                             (5, None, 1.0), (6, None, 0.0), (8, None, 0.0), (16, None, 0.0),
                             (17, None, 1.0), (32, None, 0.0), (13, "adam", 1.0), (14, "adam", 0.0),
                             (20, "adam", 0.0), (24, "sgd", 0.0)):
            jb = TorchJob(Job("budget.n", n, (1000,)), dev, lib=lib, optimizer=opt)
            assert jb.cached_fraction() == want, (n, opt)
            jb.destroy()
        for opt in ("sgd", None):
            jb = TorchJob(Job("budget.unfused", 8, (1000,)), dev, lib=lib, optimizer=opt,
                          unfused=True)
            assert jb.cached_fraction() == 1.0, opt
            jb.destroy()
        # an explicit budget that ends inside the key: cut at a tile boundary
        f = TorchJob(spec, dev, lib=lib, resident_bytes=8 * 5000)
        assert f.info()[4] == 8 * 4096
        f.destroy()
    finally:
        for j in (a, b, c, d, e):
            if j is not None:
                j.destroy()


def test_bandwidth_probe_reads_and_leaves_sink(torch_dev):
    """The probe runs on a small set of buffers, rejects bad arguments, and
    writes the sink only where a sum hits the sentinel."""
    import ctypes
    torch, dev = torch_dev
    from paper_1805_07891_amd import build
    probe = ctypes.CDLL(build.PROBE_LIB)
    probe.phub_probe_read.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_int, ctypes.c_int64,
                                      ctypes.c_int, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p]
    tile = probe.phub_probe_tile_elems()
    bufs = [torch.ones(tile * 3, device=dev) for _ in range(3)]
    ptrs = (ctypes.c_void_p * 3)(*[b.data_ptr() for b in bufs])
    sink = torch.zeros(8 * 256, device=dev)
    _say("probe: 3 buffers of", tile * 3, "floats, grid 8")
    assert probe.phub_probe_read(ptrs, 3, tile * 3, 8, -7.0, ctypes.c_void_p(sink.data_ptr()), None) == 0
    torch.cuda.synchronize()
    assert torch.count_nonzero(sink).item() == 0
    assert probe.phub_probe_read(ptrs, 3, tile * 3 + 1, 8, -7.0, ctypes.c_void_p(sink.data_ptr()), None) == -1
    assert probe.phub_probe_read(ptrs, 0, tile, 8, -7.0, ctypes.c_void_p(sink.data_ptr()), None) == -1
    # a sentinel the data does hit: every lane of a wave that read one tile of
    # ones sums 4 * 8 = 32 per tile it read
    one = (ctypes.c_void_p * 1)(bufs[0].data_ptr())
    assert probe.phub_probe_read(one, 1, tile, 1, 32.0, ctypes.c_void_p(sink.data_ptr()), None) == 0
    torch.cuda.synchronize()
    assert torch.count_nonzero(sink[:64]).item() == 64      # wave 0 read the single tile
    assert torch.count_nonzero(sink[64:]).item() == 0


def test_write_and_mixed_probes(torch_dev):
    """The write probe fills its buffers with the value; the mixed probe
    reads its read buffers and writes its read-write buffers back unchanged,
    leaving the sink alone unless a sum hits the sentinel; both reject bad
    arguments."""
    import ctypes
    torch, dev = torch_dev
    from paper_1805_07891_amd import build
    probe = ctypes.CDLL(build.PROBE_LIB)
    pp = ctypes.POINTER(ctypes.c_void_p)
    probe.phub_probe_write.argtypes = [pp, ctypes.c_int, ctypes.c_int64, ctypes.c_int,
                                       ctypes.c_float, ctypes.c_void_p]
    probe.phub_probe_mixed.argtypes = [pp, ctypes.c_int, pp, ctypes.c_int, ctypes.c_int64,
                                       ctypes.c_int, ctypes.c_float, ctypes.c_void_p,
                                       ctypes.c_void_p]
    tile = probe.phub_probe_tile_elems()
    n = tile * 5
    out = [torch.zeros(n + 16, device=dev) for _ in range(2)]
    optr = (ctypes.c_void_p * 2)(*[b.data_ptr() for b in out])
    _say("write probe: 2 buffers of", n, "floats, grid 3")
    assert probe.phub_probe_write(optr, 2, n, 3, 2.5, None) == 0
    torch.cuda.synchronize()
    for b in out:
        assert torch.all(b[:n] == 2.5).item() and not b[n:].any().item()
    assert probe.phub_probe_write(optr, 2, n + 1, 3, 2.5, None) == -1
    assert probe.phub_probe_write(optr, 0, n, 3, 2.5, None) == -1
    reads = [torch.randn(n, device=dev) for _ in range(3)]
    rw = [torch.randn(n, device=dev) for _ in range(2)]
    before = [b.clone() for b in rw]
    rptr = (ctypes.c_void_p * 3)(*[b.data_ptr() for b in reads])
    wptr = (ctypes.c_void_p * 2)(*[b.data_ptr() for b in rw])
    sink = torch.zeros(4 * 256, device=dev)
    _say("mixed probe: 3 read and 2 read-write buffers of", n, "floats, grid 4")
    assert probe.phub_probe_mixed(rptr, 3, wptr, 2, n, 4, -1.0e30,
                                  ctypes.c_void_p(sink.data_ptr()), None) == 0
    torch.cuda.synchronize()
    for a, b in zip(rw, before):
        assert torch.equal(a, b)
    assert torch.count_nonzero(sink).item() == 0
    assert probe.phub_probe_mixed(rptr, 3, wptr, 2, n + 4, 4, -1.0e30,
                                  ctypes.c_void_p(sink.data_ptr()), None) == -1
    assert probe.phub_probe_mixed(rptr, 0, wptr, 0, n, 4, -1.0e30,
                                  ctypes.c_void_p(sink.data_ptr()), None) == -1


@pytest.mark.parametrize("n", [1, 4, 8, 16, 17])
@pytest.mark.parametrize("nesterov", [True, False])
def test_unfused_variant_gives_the_same_bits(lib, torch_dev, n, nesterov):
    """The two-pass ablation (sum into a merge buffer, then the optimizer)
    performs the same operations in the same order."""
    torch, dev = torch_dev
    keys = (5, 1024, 8193, 40000, 3, 70001, 1)
    _say("unfused N", n, "nesterov", nesterov)
    for resident in (0, 1 << 40):
        job, res = run_small_case(torch, dev, lib, n, keys, steps=2, nesterov=nesterov,
                                  seed=40 + n, resident_bytes=resident, unfused=True)
        assert_parity(res, f"unfused N={n} nesterov={nesterov} resident={resident}")
        job.destroy()


@pytest.mark.parametrize("workgroups", [1, 7, 64, 1000])
def test_launch_size_does_not_change_results(lib, torch_dev, workgroups):
    """Any persistent grid (fewer or more workgroups than compute units)
    covers the whole schedule once."""
    torch, dev = torch_dev
    keys = (5, 1024, 8193, 40000, 3, 70001, 1 << 20)
    _say("workgroups", workgroups)
    for resident in (0, 1 << 40):
        job, res = run_small_case(torch, dev, lib, 8, keys, steps=2, seed=70 + workgroups,
                                  resident_bytes=resident, workgroups=workgroups)
        assert job.info()[0] == workgroups
        assert_parity(res, f"workgroups={workgroups} resident={resident}")
        job.destroy()


def test_set_weights_resets_momentum(lib, torch_dev):
    torch, dev = torch_dev
    job, res = run_small_case(torch, dev, lib, 2, [300], steps=2, seed=8)
    new_w = torch.full((job.arena_elems,), 0.5, device=dev)
    job.set_weights(new_w)
    W, M = job.state_arenas()
    assert np.all(W[:300] == 0.5) and np.all(M[:300] == 0.0)
    job.destroy()


def test_concurrent_jobs_equal_sequential(lib, torch_dev):
    torch, dev = torch_dev
    specs = [(8, [70000, 3, 8193]), (4, [12345, 64]), (16, [30000]), (3, [1, 2, 3, 100000])]
    # concurrent: one stream each, steps interleaved
    seq = [run_small_case(torch, dev, lib, n, k, steps=2, seed=40 + i) for i, (n, k) in enumerate(specs)]
    for job, res in seq:
        assert_parity(res, "sequential")
        job.destroy()
    streams = [torch.cuda.Stream(device=dev) for _ in specs]
    jobs = []
    rng_inputs = []
    for i, (n, keys) in enumerate(specs):
        spec = Job(f"c{i}", n, tuple(keys))
        job = TorchJob(spec, dev, stream=streams[i], lib=lib)
        offs, total = key_offsets(keys)
        rng = np.random.default_rng(40 + i)
        w0 = np.zeros(total, np.float32)
        for o, m in zip(offs, keys):
            w0[o:o + m] = rng.standard_normal(m, dtype=np.float32) * np.float32(0.05)
        job.set_weights(torch.from_numpy(w0).to(dev))
        steps_host = []
        for t in range(2):
            host = []
            for w in range(n):
                a = np.zeros(total, np.float32)
                for o, m in zip(offs, keys):
                    a[o:o + m] = rng.standard_normal(m, dtype=np.float32) * np.float32(1e-2)
                host.append(a)
            steps_host.append([torch.from_numpy(a).to(dev) for a in host])
        jobs.append(job)
        rng_inputs.append(steps_host)
    torch.cuda.synchronize()
    for t in range(2):
        for job, inputs in zip(jobs, rng_inputs):
            for w, a in enumerate(inputs[t]):
                job.attach_grads(w, a)
            job.push_and_step()
    for i, job in enumerate(jobs):
        W, M = job.state_arenas()
        wg, mg = job.split(W), job.split(M)
        sw, sm = seq[i][1][-1][0], seq[i][1][-1][1]
        for k in range(len(wg)):
            assert _bits_equal(wg[k], sw[k]) and _bits_equal(mg[k], sm[k]), (i, k)
        job.destroy()


# --------------------------------------------------------------------------
# Full-size workloads in the benchmark's launch configuration, checked on
# every element (tests/test_gpu_fullsize.py).  The largest key below is
# checked on sampled elements that the oracle recomputes one by one.
# --------------------------------------------------------------------------

def test_key_past_four_gib_sampled(lib, torch_dev):
    """One key of 1.2 G elements (4.8 GB per array, the largest size here):
    element offsets past 2^32 bytes inside a key, the 16 MB folds of the
    kernel's 32-bit lane offsets, and both bins (the cache budget ends
    inside the key).  Two steps; sampled elements (each key's ends, around
    2^30 elements, around the folds and the budget's cut, random) checked
    bit for bit against the oracle."""
    torch, dev = torch_dev
    big = 1_200_000_003
    keys = (5, big, 1027)
    spec = Job("large", 2, keys)
    resident_elems = 3_000_000
    _say("key of", big, "elements, resident", resident_elems)
    job = TorchJob(spec, dev, lib=lib, resident_bytes=8 * resident_elems)
    assert 0.0 < job.cached_fraction() < 0.01
    _, total = key_offsets(keys)
    w0 = workloads.device_normal_arena(torch, dev, 7, total, 0.05)
    job.set_weights(w0)
    grads = [[workloads.device_normal_arena(torch, dev, 100 + 10 * t + w, total, 1e-2)
              for w in range(2)] for t in range(2)]
    for t in range(2):
        for w in range(2):
            job.attach_grads(w, grads[t][w])
        job.push_and_step()
    W, M = job.state_arenas()
    pos = set()
    for k, n in enumerate(keys):
        pos.update((k, i) for i in list(range(min(n, 3))) + list(range(max(0, n - 5), n)))
    near = [1 << 30, resident_elems - job.offsets[1]] + [m << 22 for m in (1, 2, 255, 256, 286)]
    for c in near:
        pos.update((1, i) for i in range(c - 3, c + 4) if 0 <= i < big)
    rng = np.random.default_rng(11)
    pos.update((1, int(i)) for i in rng.integers(0, big, size=20000))
    idx = np.array(sorted(job.offsets[k] + i for k, i in pos), dtype=np.int64)
    tidx = torch.from_numpy(idx).to(dev)
    ws = w0.index_select(0, tidx).cpu().numpy()
    ms = np.zeros_like(ws)
    for t in range(2):
        gs = [grads[t][w].index_select(0, tidx).cpu().numpy() for w in range(2)]
        oracle.step_flat(gs, ws, ms, spec.lr, spec.momentum, spec.weight_decay, spec.nesterov)
    _say(f"  {idx.size} sampled elements; W rel err {_rel_err(W[idx], ws):.3g}")
    assert _bits_equal(W[idx], ws), "W mismatch"
    assert _bits_equal(M[idx], ms), "M mismatch"
    job.destroy()
    del grads, W, M
    torch.cuda.empty_cache()


def test_jobs_driven_from_several_threads(lib, torch_dev):
    """Different jobs may be driven from different threads: each thread
    creates its own job (claiming from the shared cache budget), steps it
    and checks it against the oracle, then destroys it; the threads run at
    the same time, several rounds."""
    import threading
    torch, dev = torch_dev
    errors = []

    def work(i):
        try:
            torch.cuda.set_device(dev)
            for r in range(3):
                keys = [1000 + 37 * i, 70001, 5 + r]
                job, res = run_small_case(torch, dev, lib, 3 + i, keys, steps=2, seed=500 + 10 * i + r,
                                          stream=torch.cuda.Stream(device=dev))
                assert_parity(res, f"thread {i} round {r}")
                job.destroy()
        except Exception as e:  # reported by the main thread
            errors.append(f"thread {i}: {e!r}")

    threads = [threading.Thread(target=work, args=(i,)) for i in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
