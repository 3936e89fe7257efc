"""Every element of the five evaluation workloads, checked against the oracle.

Each workload runs in the benchmark's launch configuration (the jobs of the
multi-tenant workload each on their own stream, and, as the alternative the
library allows, all on one shared stream), for the workload's own number of
steps, with fresh seeded gradients every step.  While the GPU steps, the
host copies the same gradients back and the oracle steps them; at the end
every key's W and M is read through the per-key pointers of the Pull
interface (phub_pull, phub_get_state) and compared bit for bit, and the
arena padding between keys is checked to be untouched.

Host memory stays bounded: one step's gradients at a time (multi-tenant:
about 7 GB).  Each step is synchronised before its gradient buffers are
released, since the library reads them in place.
"""

import sys
import time

import numpy as np
import pytest

import oracle
from paper_1805_07891_amd import workloads
from paper_1805_07891_amd.job import TorchJob, load_library

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


def _mismatches(a, b):
    return int(np.count_nonzero(np.asarray(a, np.float32).view(np.uint32) !=
                                np.asarray(b, np.float32).view(np.uint32)))


@pytest.mark.parametrize("name,own_streams", [("tiny", True), ("resnet50", True), ("alexnet", True),
                                               ("resnet269", True), ("multitenant", True),
                                               ("multitenant", False)])
def test_full_size_workload_every_element(lib, torch_dev, name, own_streams):
    torch, dev = torch_dev
    wl = workloads.workload(name)
    steps = wl.steps
    _say("every element:", name, "own streams" if own_streams else "one shared stream",
         f"{steps} steps;", workloads.describe(wl))
    t_start = time.time()
    shared = torch.cuda.Stream(device=dev)
    jobs, W, M = [], [], []
    for ji, spec in enumerate(wl.jobs):
        stream = torch.cuda.Stream(device=dev) if own_streams else shared
        job = TorchJob(spec, dev, stream=stream, lib=lib)
        w0 = workloads.device_weight_arena(torch, dev, spec, wl.seed_index, ji)
        torch.cuda.synchronize()
        job.set_weights(w0)
        w0h = w0.cpu().numpy()
        W.append([w0h[o:o + n].copy() for o, n in zip(job.offsets, spec.key_elems)])
        M.append([np.zeros(n, np.float32) for n in spec.key_elems])
        jobs.append(job)
        del w0, w0h
    torch.cuda.synchronize()
    for t in range(steps):
        grads = [[workloads.device_grad_arena(torch, dev, spec, wl.seed_index, ji, t, w)
                  for w in range(spec.num_workers)] for ji, spec in enumerate(wl.jobs)]
        torch.cuda.synchronize()
        for job, g in zip(jobs, grads):
            for w, a in enumerate(g):
                job.attach_grads(w, a)
            job.push_and_step()
        # the oracle steps the same gradients on the host meanwhile
        for ji, (job, spec) in enumerate(zip(jobs, wl.jobs)):
            host = [a.cpu().numpy() for a in grads[ji]]
            oracle.step([[h[o:o + n] for o, n in zip(job.offsets, spec.key_elems)] for h in host],
                        W[ji], M[ji], spec.lr, spec.momentum, spec.weight_decay, spec.nesterov)
            del host
        for job in jobs:
            job.sync()
        del grads
        _say(f"  step {t + 1}/{steps} done ({time.time() - t_start:.1f} s)")
    for ji, (job, spec) in enumerate(zip(jobs, wl.jobs)):
        pulled = job.pulled_keys()
        bad = []
        for k, (pw, pm, _) in enumerate(pulled):
            nw, nm = _mismatches(pw, W[ji][k]), _mismatches(pm, M[ji][k])
            if nw or nm:
                bad.append((k, spec.key_elems[k], nw, nm))
        _say(f"  {spec.name}: {spec.num_params:,} elements of W and M compared, "
             f"{len(bad)} keys differ")
        assert not bad, f"{spec.name}: keys (key, elems, W mismatches, M mismatches) {bad[:10]}"
        # the arena padding between keys is never written
        Wa, Ma = job.state_arenas()
        pad = np.ones(Wa.size, bool)
        for o, n in zip(job.offsets, spec.key_elems):
            pad[o:o + n] = False
        assert not Wa[pad].any() and not Ma[pad].any(), f"{spec.name}: padding written"
        job.destroy()
    del W, M
    torch.cuda.empty_cache()
