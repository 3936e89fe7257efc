"""GPU tests of PushPull (section 3.1): the fused step also writes each key's
updated weights into every worker's model buffer.  Every buffer must hold
exactly the oracle's W after the step, and W and M must match the oracle
as in a plain step."""

import sys

import numpy as np
import pytest

import oracle
from paper_1805_07891_amd import phub
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


class Case:
    def __init__(self, torch, dev, lib, n_workers, key_elems, seed, key_group=None,
                 resident_bytes=None, nesterov=True, schedule=None):
        self.torch = torch
        self.spec = Job("pushpull", n_workers, tuple(int(n) for n in key_elems), nesterov=nesterov)
        self.job = TorchJob(self.spec, dev, lib=lib, key_group=key_group,
                            resident_bytes=resident_bytes, schedule=schedule)
        self.offs, self.total = key_offsets(self.spec.key_elems)
        self.rng = np.random.default_rng(seed)
        w0 = np.zeros(self.total, np.float32)
        for o, n in zip(self.offs, self.spec.key_elems):
            w0[o:o + n] = self.rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
        self.job.set_weights(torch.from_numpy(w0).to(dev))
        self.W = [w0[o:o + n].copy() for o, n in zip(self.offs, self.spec.key_elems)]
        self.M = [np.zeros(n, np.float32) for n in self.spec.key_elems]
        # model buffers start as NaN so that an unwritten element shows
        self.models = [torch.full((self.total,), float("nan"), device=dev) for _ in range(n_workers)]
        for w in range(n_workers):
            self.job.attach_models(w, self.models[w])
        self.dev = dev

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
        s = self.spec
        oracle.step([[h[o:o + n] for o, n in zip(self.offs, s.key_elems)] for h in host],
                    self.W, self.M, s.lr, s.momentum, s.weight_decay, s.nesterov)

    def check(self, label, models_expected=True):
        Wg, Mg = self.job.state_arenas()
        for k, (wg, mg) in enumerate(zip(self.job.split(Wg), self.job.split(Mg))):
            assert _bits_equal(wg, self.W[k]) and _bits_equal(mg, self.M[k]), f"{label}: W/M key {k}"
        if models_expected:
            for w, m in enumerate(self.models):
                mh = m.cpu().numpy()
                for k, (o, n) in enumerate(zip(self.offs, self.spec.key_elems)):
                    assert _bits_equal(mh[o:o + n], self.W[k]), f"{label}: worker {w} key {k}"


KEYS = (5, 1024, 8193, 40000, 3, 70001, 2048, 131072, 1)


@pytest.mark.parametrize("n_workers", [1, 4, 8, 16, 17])
@pytest.mark.parametrize("resident", [0, 8 * 50000, 1 << 40])
@pytest.mark.parametrize("schedule", [None, phub.PHUB_SCHEDULE_DYNAMIC])
def test_pushpull_writes_the_updated_weights_to_every_worker(lib, torch_dev, n_workers, resident,
                                                             schedule):
    torch, dev = torch_dev
    _say("pushpull N", n_workers, "resident", resident, "schedule", schedule)
    c = Case(torch, dev, lib, n_workers, KEYS, seed=21 + n_workers, resident_bytes=resident,
             schedule=schedule)
    for t in range(2):
        host, arenas = c.new_grads()
        c.job.pushpull_all()
        c.job.step()
        c.oracle_step(host)
        c.check(f"N={n_workers} resident={resident} step {t}")
    c.job.destroy()


def test_pushpull_plain_nesterov_off_and_single_key_calls(lib, torch_dev):
    torch, dev = torch_dev
    c = Case(torch, dev, lib, 3, (777, 4096, 9), seed=31, nesterov=False)
    host, arenas = c.new_grads()
    for k in reversed(range(3)):
        for w in range(3):
            lib.phub_pushpull(c.job.handle, w, k, c.job.key_pointers(arenas[w])[k],
                              c.job.key_pointers(c.models[w])[k])
    c.job.step()
    c.oracle_step(host)
    c.check("single-key pushpull")
    c.job.destroy()


def test_pushpull_with_readiness_groups(lib, torch_dev):
    torch, dev = torch_dev
    c = Case(torch, dev, lib, 8, KEYS, seed=32, key_group=[k % 4 for k in range(len(KEYS))])
    for t in range(2):
        host, arenas = c.new_grads()
        c.job.pushpull_all()
        c.job.step()
        c.oracle_step(host)
        c.check(f"grouped pushpull step {t}")
    c.job.destroy()


def test_a_mix_of_push_and_pushpull_is_rejected(lib, torch_dev):
    torch, dev = torch_dev
    keys = (1024, 300)
    c = Case(torch, dev, lib, 2, keys, seed=33)
    host, arenas = c.new_grads()
    g = [c.job.key_pointers(a) for a in arenas]
    o = [c.job.key_pointers(m) for m in c.models]
    lib.phub_pushpull(c.job.handle, 0, 0, g[0][0], o[0][0])
    lib.phub_push(c.job.handle, 1, 0, g[1][0])
    for w in range(2):
        lib.phub_pushpull(c.job.handle, w, 1, g[w][1], o[w][1])
    assert lib.phub_step(c.job.handle, check=False) == phub.PHUB_EINVAL
    assert "worker 1" in lib.last_error() and "key 0" in lib.last_error()
    lib.phub_pushpull(c.job.handle, 1, 0, g[1][0], o[1][0])   # complete the registration
    c.job.step()
    c.oracle_step(host)
    c.check("after completing the registration")
    # a plain step next leaves the model buffers as they are
    before = [m.clone() for m in c.models]
    host, arenas = c.new_grads()
    c.job.push_all()
    c.job.step()
    c.oracle_step(host)
    c.check("plain step", models_expected=False)
    for b, m in zip(before, c.models):
        assert torch.equal(b.view(torch.int32), m.view(torch.int32))
    c.job.destroy()


def test_pushpull_rejects_bad_model_buffers(lib, torch_dev):
    torch, dev = torch_dev
    c = Case(torch, dev, lib, 2, (64,), seed=34)
    host, arenas = c.new_grads()
    gp = c.job.key_pointers(arenas[0])[0]
    op = c.job.key_pointers(c.models[0])[0]
    assert lib.phub_pushpull(c.job.handle, 0, 0, gp, None, check=False) == phub.PHUB_EINVAL
    assert lib.phub_pushpull(c.job.handle, 0, 0, gp, op + 4, check=False) == phub.PHUB_EINVAL
    c.job.destroy()
