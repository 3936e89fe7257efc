"""GPU tests of the pluggable optimizers (paper section 3.2.2): plain SGD
and Adam in the fused pass, checked bit for bit against the CPU oracle over
several steps (Adam's step counter), with every launch variant."""

import sys

import numpy as np
import pytest

import oracle
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


LR, WD, B1, B2, EPS = 1e-3, 1e-2, 0.9, 0.999, 1e-8


class Case:
    def __init__(self, torch, dev, lib, optimizer, n_workers, key_elems, seed, **job_kw):
        self.torch, self.dev, self.opt = torch, dev, optimizer
        self.spec = Job("opt", n_workers, tuple(int(n) for n in key_elems), lr=LR, weight_decay=WD)
        self.job = TorchJob(self.spec, dev, lib=lib, optimizer=optimizer, betas=(B1, B2), eps=EPS,
                            **job_kw)
        self.offs, self.total = key_offsets(self.spec.key_elems)
        self.rng = np.random.default_rng(seed)
        w0 = np.zeros(self.total, np.float32)
        for o, n in zip(self.offs, self.spec.key_elems):
            w0[o:o + n] = self.rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
        self.job.set_weights(torch.from_numpy(w0).to(dev))
        self.W = [w0[o:o + n].copy() for o, n in zip(self.offs, self.spec.key_elems)]
        self.M = [np.zeros(n, np.float32) for n in self.spec.key_elems]
        self.V = [np.zeros(n, np.float32) for n in self.spec.key_elems]
        self.t = 0

    def new_grads(self):
        host = []
        for _ in range(self.spec.num_workers):
            a = np.zeros(self.total, np.float32)
            for o, n in zip(self.offs, self.spec.key_elems):
                a[o:o + n] = self.rng.standard_normal(n, dtype=np.float32) * np.float32(1e-2)
            host.append(a)
        arenas = [self.torch.from_numpy(a).to(self.dev) for a in host]
        for w, a in enumerate(arenas):
            self.job.attach_grads(w, a)
        self.torch.cuda.synchronize()
        return host, arenas

    def oracle_step(self, host):
        g = [[h[o:o + n] for o, n in zip(self.offs, self.spec.key_elems)] for h in host]
        self.t += 1
        if self.opt == "sgd":
            oracle.step_sgd(g, self.W, LR, WD)
        else:
            oracle.step_adam(g, self.W, self.M, self.V, LR, B1, B2, EPS, WD, self.t)

    def check(self, label):
        Wg, Mg = self.job.state_arenas()
        for k, wg in enumerate(self.job.split(Wg)):
            assert _bits_equal(wg, self.W[k]), f"{label}: W key {k}"
        if self.opt == "sgd":
            assert Mg is None and self.job.second_moment_arena() is None
        else:
            Vg = self.job.second_moment_arena()
            for k, (mg, vg) in enumerate(zip(self.job.split(Mg), self.job.split(Vg))):
                assert _bits_equal(mg, self.M[k]), f"{label}: M key {k}"
                assert _bits_equal(vg, self.V[k]), f"{label}: V key {k}"


KEYS = (5, 1024, 8193, 40000, 3, 70001, 2048, 131072, 1)


@pytest.mark.parametrize("optimizer", ["sgd", "adam"])
@pytest.mark.parametrize("n_workers", [1, 4, 8, 16, 17])
@pytest.mark.parametrize("resident", [0, 12 * 50000, 1 << 40])
def test_optimizer_matches_the_oracle(lib, torch_dev, optimizer, n_workers, resident):
    torch, dev = torch_dev
    _say(optimizer, "N", n_workers, "resident", resident)
    c = Case(torch, dev, lib, optimizer, n_workers, KEYS, seed=50 + n_workers,
             resident_bytes=resident)
    for t in range(3):
        host, _ = c.new_grads()
        c.job.push_all()
        c.job.step()
        c.oracle_step(host)
        c.check(f"{optimizer} N={n_workers} resident={resident} step {t + 1}")
    c.job.destroy()


@pytest.mark.parametrize("optimizer", ["sgd", "adam"])
@pytest.mark.parametrize("resident", [None, 12 * 30000])
def test_optimizer_with_groups_pushpull_and_unfused(lib, torch_dev, optimizer, resident):
    """Readiness groups + pushpull (every group of a step uses the same step
    number), then the unfused ablation; with the default budget (all state
    cached) and with a budget that ends inside a key (both bins in every
    group's launch)."""
    torch, dev = torch_dev
    _say(optimizer, "groups + pushpull, resident", resident)
    c = Case(torch, dev, lib, optimizer, 8, KEYS, seed=61, key_group=[k % 3 for k in range(len(KEYS))],
             resident_bytes=resident)
    frac = c.job.cached_fraction()
    if resident is not None:
        assert 0.0 < frac < 1.0
    else:  # the default budget; plain SGD with 8 workers streams all its state
        assert frac == (0.0 if optimizer == "sgd" else 1.0)
    models = [torch.full((c.total,), float("nan"), device=dev) for _ in range(8)]
    for w in range(8):
        c.job.attach_models(w, models[w])
    for t in range(3):
        host, _ = c.new_grads()
        c.job.pushpull_all()
        c.job.step()
        c.oracle_step(host)
        c.check(f"{optimizer} grouped pushpull step {t + 1}")
        for w in range(8):
            mh = models[w].cpu().numpy()
            for k, (o, n) in enumerate(zip(c.offs, c.spec.key_elems)):
                assert _bits_equal(mh[o:o + n], c.W[k]), f"model buffer {w} key {k}"
    c.job.destroy()
    # the unfused ablation with the same optimizer
    c = Case(torch, dev, lib, optimizer, 5, KEYS, seed=62, unfused=True, resident_bytes=resident)
    for t in range(2):
        host, _ = c.new_grads()
        c.job.push_all()
        c.job.step()
        c.oracle_step(host)
        c.check(f"{optimizer} unfused step {t + 1}")
    c.job.destroy()
