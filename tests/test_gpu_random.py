"""Seeded random combinations of the job options, each checked bit for bit
against the CPU oracle over two steps.

Every case draws: the worker count (1-20, so every fixed-N kernel with its
load window and, where it has one, its burst write-back; above 16 the any-N
kernel), a mix of key sizes (empty, ragged, around tile and chunk
boundaries, larger keys), the optimizer (momentum with or without Nesterov,
plain SGD, Adam), the schedule, the chunk size, the launch size, the cache
budget (none, partial, all, the default), readiness groups, pushpull and the
unfused ablation (only where it applies).  The draws come from a fixed seed, so a failure names a
reproducible case.
"""

import sys

import numpy as np
import pytest

import oracle
from paper_1805_07891_amd import phub
from paper_1805_07891_amd.job import TorchJob, load_library
from paper_1805_07891_amd.workloads import Job, key_offsets

pytestmark = pytest.mark.gpu

LR, MU, WD, B1, B2, EPS = 0.05, 0.9, 1e-3, 0.9, 0.999, 1e-8
CASES = 300


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


def draw_case(seed):
    rng = np.random.default_rng(1805_000 + seed)
    n = int(rng.integers(1, 21))
    k = int(rng.integers(1, 11))
    pool = [0, 1, 3, 4, 5, 63, 64, 65, 255, 1023, 1024, 1025, 2047, 4095, 4096, 4097, 8191,
            8193, 16384]
    keys = []
    for _ in range(k):
        if rng.random() < 0.7:
            keys.append(int(rng.choice(pool)))
        else:
            keys.append(int(rng.integers(1, 150_000)))
    opt = str(rng.choice(["momentum", "nesterov", "sgd", "adam"]))
    states = {"sgd": 1, "adam": 3}.get(opt, 2)
    state_bytes = 4 * states * sum(keys)
    resident = rng.choice([None, 0, 1 << 40, "partial"])
    if resident == "partial":
        resident = int(rng.integers(1, max(2, state_bytes)))
    groups = None
    if rng.random() < 0.4:
        ng = int(rng.integers(1, k + 2))
        groups = [int(g) for g in rng.integers(0, ng, size=k)]
    pushpull = bool(rng.random() < 0.3)
    unfused = bool(groups is None and not pushpull and rng.random() < 0.25)
    return dict(
        n=n, keys=tuple(keys), opt=opt, resident=resident, groups=groups, pushpull=pushpull,
        unfused=unfused,
        schedule=int(rng.choice([phub.PHUB_SCHEDULE_LPT, phub.PHUB_SCHEDULE_SPLIT])),
        chunk_bytes=int(16 * rng.integers(1, 1 << 16)),
        workgroups=None if rng.random() < 0.6 else int(rng.integers(1, 300)),
        seed=seed)


@pytest.mark.parametrize("seed", range(CASES))
def test_random_option_combination_matches_the_oracle(lib, torch_dev, seed):
    torch, dev = torch_dev
    c = draw_case(seed)
    _say("random case", c)
    n, keys, opt = c["n"], c["keys"], c["opt"]
    spec = Job("random", n, keys, lr=LR, momentum=MU, weight_decay=WD, nesterov=opt == "nesterov",
               chunk_elems=c["chunk_bytes"] // 4)
    job = TorchJob(spec, dev, lib=lib, chunk_bytes=c["chunk_bytes"], schedule=c["schedule"],
                   resident_bytes=c["resident"], key_group=c["groups"], unfused=c["unfused"],
                   optimizer={"momentum": None, "nesterov": None}.get(opt, opt), betas=(B1, B2),
                   eps=EPS, workgroups=c["workgroups"])
    offs, total = key_offsets(keys)
    rng = np.random.default_rng(seed)
    w0 = np.zeros(total, np.float32)
    for o, m in zip(offs, keys):
        w0[o:o + m] = rng.standard_normal(m, dtype=np.float32) * np.float32(0.05)
    job.set_weights(torch.from_numpy(w0).to(dev))
    W = [w0[o:o + m].copy() for o, m in zip(offs, keys)]
    M = [np.zeros(m, np.float32) for m in keys]
    V = [np.zeros(m, np.float32) for m in keys]
    models = None
    if c["pushpull"]:
        models = [torch.full((total,), float("nan"), device=dev) for _ in range(n)]
        for w in range(n):
            job.attach_models(w, models[w])
    for t in range(2):
        host = []
        for _ in range(n):
            a = np.zeros(total, np.float32)
            for o, m in zip(offs, keys):
                a[o:o + m] = rng.standard_normal(m, dtype=np.float32) * np.float32(1e-2)
            host.append(a)
        arenas = [torch.from_numpy(a).to(dev) for a in host]
        for w in range(n):
            job.attach_grads(w, arenas[w])
        torch.cuda.synchronize()
        if c["pushpull"]:
            job.pushpull_all()
        else:
            job.push_all()
        job.step()
        g = [[h[o:o + m] for o, m in zip(offs, keys)] for h in host]
        if opt == "sgd":
            oracle.step_sgd(g, W, LR, WD)
        elif opt == "adam":
            oracle.step_adam(g, W, M, V, LR, B1, B2, EPS, WD, t + 1)
        else:
            oracle.step(g, W, M, LR, MU, WD, opt == "nesterov")
        Wg, Mg = job.state_arenas()
        for k, (o, m) in enumerate(zip(offs, keys)):
            assert _bits_equal(Wg[o:o + m], W[k]), f"case {seed} step {t}: W key {k}"
            if opt != "sgd":
                assert _bits_equal(Mg[o:o + m], M[k]), f"case {seed} step {t}: M key {k}"
        if opt == "adam":
            Vg = job.second_moment_arena()
            for k, (o, m) in enumerate(zip(offs, keys)):
                assert _bits_equal(Vg[o:o + m], V[k]), f"case {seed} step {t}: V key {k}"
        if models is not None:
            for w in range(n):
                mh = models[w].cpu().numpy()
                for k, (o, m) in enumerate(zip(offs, keys)):
                    assert _bits_equal(mh[o:o + m], W[k]), f"case {seed} step {t}: model {w} key {k}"
    job.destroy()
