"""GPU parity of the streamed bin's burst write-back (the LDS stash of the
fixed-N kernels): worker counts and optimizers that have it, with grids
small enough that a wave walks many tiles (several full write-backs and a
partial last one), with nothing cached and with a cache budget that ends
inside a key, in one launch or one per readiness group; bit-exact against
the CPU oracle over two steps.  The stash is written back when the wall
clock is in a write window as well as when it is full, so how many tiles a
write-back covers changes from run to run: the results must not."""

import sys

import numpy as np
import pytest

import oracle
from paper_1805_07891_amd import phub
from paper_1805_07891_amd.job import TorchJob, load_library
from paper_1805_07891_amd.workloads import Job, key_offsets

pytestmark = pytest.mark.gpu

LR, MU, WD, B1, B2, EPS = 0.05, 0.9, 1e-3, 0.9, 0.999, 1e-8

# (workers, optimizer): kernels that stash (momentum, Nesterov and plain SGD
# with 6-16 workers, Adam with 14-16), and, next to them, counts at the
# rule's edge (5 momentum, 5 SGD, 13 Adam) that write piece by piece
STASHED = [(6, "nesterov"), (7, "momentum"), (8, "nesterov"), (8, "momentum"), (9, "nesterov"),
           (10, "momentum"), (11, "momentum"), (12, "nesterov"), (13, "momentum"),
           (14, "nesterov"), (15, "momentum"), (16, "nesterov"), (16, "momentum"), (6, "sgd"),
           (8, "sgd"), (11, "sgd"), (16, "sgd"), (14, "adam"), (15, "adam"), (16, "adam"),
           (5, "momentum"), (5, "sgd"), (13, "adam")]
# 107 full tiles and ragged ends: a wave of a 1-workgroup grid (4 waves)
# walks about 27 tiles
KEYS = (5, 1024 * 37 + 3, 70001, 1024 * 11, 4097, 1, 1024 * 6)


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


def _run(lib, torch_dev, n, opt, workgroups, resident, key_group=None, schedule=None):
    torch, dev = torch_dev
    states = {"sgd": 1, "adam": 3}.get(opt, 2)
    if resident == "partial":
        resident = 4 * states * 50000
    _say("stash", opt, "N", n, "workgroups", workgroups, "resident", resident, "groups", key_group,
         "schedule", schedule)
    spec = Job("stash", n, KEYS, lr=LR, momentum=MU, weight_decay=WD, nesterov=opt == "nesterov")
    job = TorchJob(spec, dev, lib=lib, resident_bytes=resident, workgroups=workgroups,
                   optimizer={"momentum": None, "nesterov": None}.get(opt, opt), betas=(B1, B2),
                   eps=EPS, key_group=key_group, schedule=schedule)
    offs, total = key_offsets(KEYS)
    rng = np.random.default_rng(1000 + n)
    w0 = np.zeros(total, np.float32)
    for o, m in zip(offs, KEYS):
        w0[o:o + m] = rng.standard_normal(m, dtype=np.float32) * np.float32(0.05)
    job.set_weights(torch.from_numpy(w0).to(dev))
    W = [w0[o:o + m].copy() for o, m in zip(offs, KEYS)]
    M = [np.zeros(m, np.float32) for m in KEYS]
    V = [np.zeros(m, np.float32) for m in KEYS]
    for t in range(2):
        host = []
        for _ in range(n):
            a = np.zeros(total, np.float32)
            for o, m in zip(offs, KEYS):
                a[o:o + m] = rng.standard_normal(m, dtype=np.float32) * np.float32(1e-2)
            host.append(a)
        arenas = [torch.from_numpy(a).to(dev) for a in host]
        for w in range(n):
            job.attach_grads(w, arenas[w])
        torch.cuda.synchronize()
        if key_group is None:
            job.push_all()
        else:
            # backward order: each readiness group launches once its keys are in
            for k in reversed(range(len(KEYS))):
                for w in range(n):
                    job.push_key(w, k)
        job.step()
        g = [[h[o:o + m] for o, m in zip(offs, KEYS)] for h in host]
        if opt == "sgd":
            oracle.step_sgd(g, W, LR, WD)
        elif opt == "adam":
            oracle.step_adam(g, W, M, V, LR, B1, B2, EPS, WD, t + 1)
        else:
            oracle.step(g, W, M, LR, MU, WD, opt == "nesterov")
        Wg, Mg = job.state_arenas()
        for k, (o, m) in enumerate(zip(offs, KEYS)):
            assert _bits_equal(Wg[o:o + m], W[k]), f"step {t}: W key {k}"
            if opt != "sgd":
                assert _bits_equal(Mg[o:o + m], M[k]), f"step {t}: M key {k}"
        if opt == "adam":
            Vg = job.second_moment_arena()
            for k, (o, m) in enumerate(zip(offs, KEYS)):
                assert _bits_equal(Vg[o:o + m], V[k]), f"step {t}: V key {k}"
    job.destroy()


@pytest.mark.parametrize("n,opt", STASHED)
@pytest.mark.parametrize("workgroups,resident", [(1, 0), (3, 0), (1, "partial"), (None, 0),
                                                 (None, "partial")])
def test_burst_write_back_matches_the_oracle(lib, torch_dev, n, opt, workgroups, resident):
    _run(lib, torch_dev, n, opt, workgroups, resident)


@pytest.mark.parametrize("n,opt", [(16, "nesterov"), (13, "momentum"), (8, "nesterov"), (11, "sgd"),
                                   (24, "momentum"), (32, "sgd"), (20, "adam"), (14, "adam")])
@pytest.mark.parametrize("workgroups,resident", [(1, 0), (None, "partial")])
def test_burst_write_back_per_readiness_group(lib, torch_dev, n, opt, workgroups, resident):
    """Each readiness group's launch walks its own tiles: the stash is
    written back at the end of every group's bin."""
    _run(lib, torch_dev, n, opt, workgroups, resident,
         key_group=[k % 3 for k in range(len(KEYS))])


@pytest.mark.parametrize("n", [20, 24, 32])
@pytest.mark.parametrize("opt", ["momentum", "nesterov", "sgd", "adam"])
@pytest.mark.parametrize("workgroups,resident", [(1, 0), (None, "partial")])
def test_larger_fixed_worker_counts(lib, torch_dev, n, opt, workgroups, resident):
    """20, 24 and 32 workers have kernels of their own (phased ring of 6,
    burst write-back, resident ring below a whole tile); bit-exact against
    the oracle like the others."""
    _run(lib, torch_dev, n, opt, workgroups, resident)


@pytest.mark.parametrize("n,opt", [(8, "nesterov"), (16, "momentum"), (4, "nesterov"), (11, "sgd"),
                                   (14, "adam"), (3, "adam"), (24, "momentum")])
@pytest.mark.parametrize("workgroups,resident", [(1, 0), (3, 0), (5, "partial"), (None, 0)])
@pytest.mark.parametrize("grouped", [False, True])
def test_dynamic_schedule_matches_the_oracle(lib, torch_dev, n, opt, workgroups, resident, grouped):
    """The dynamic schedule: the streamed full tiles taken from a pool by the
    waves (with and without burst write-back), every launch of a step
    (readiness groups) and of the next step advancing the shared counter;
    bit-exact against the oracle over two steps."""
    _run(lib, torch_dev, n, opt, workgroups, resident,
         key_group=[k % 3 for k in range(len(KEYS))] if grouped else None,
         schedule=phub.PHUB_SCHEDULE_DYNAMIC)
