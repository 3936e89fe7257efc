"""GPU tests of readiness groups and ready events (sections 3.2.2-3.2.3:
a chunk is aggregated as soon as all of its pieces have arrived).

Every case is checked bit for bit against the CPU oracle: grouping the keys,
launching groups as they complete, and waiting on producers' events must not
change a single result.
"""

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
    """A job with seeded weights, plus the oracle's copy of its state."""

    def __init__(self, torch, dev, lib, n_workers, key_elems, key_group=None, seed=0,
                 resident_bytes=None, ordered_events=False):
        self.torch, self.dev = torch, dev
        self.spec = Job("stream", n_workers, tuple(int(n) for n in key_elems), sigma_g=1e-2)
        self.job = TorchJob(self.spec, dev, lib=lib, key_group=key_group,
                            resident_bytes=resident_bytes, ordered_events=ordered_events)
        self.offs, self.total = key_offsets(self.spec.key_elems)
        self.rng = np.random.default_rng(seed)
        w0 = np.zeros(self.total, np.float32)
        for o, n in zip(self.offs, self.spec.key_elems):
            w0[o:o + n] = self.rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
        self.job.set_weights(torch.from_numpy(w0).to(dev))
        self.W = [w0[o:o + n].copy() for o, n in zip(self.offs, self.spec.key_elems)]
        self.M = [np.zeros(n, np.float32) for n in self.spec.key_elems]

    def host_grads(self):
        out = []
        for _ in range(self.spec.num_workers):
            a = np.zeros(self.total, np.float32)
            for o, n in zip(self.offs, self.spec.key_elems):
                a[o:o + n] = self.rng.standard_normal(n, dtype=np.float32) * np.float32(1e-2)
            out.append(a)
        return out

    def oracle_step(self, host):
        s = self.spec
        oracle.step([[h[o:o + n] for o, n in zip(self.offs, s.key_elems)] for h in host],
                    self.W, self.M, s.lr, s.momentum, s.weight_decay, s.nesterov)

    def check(self, label):
        Wg, Mg = self.job.state_arenas()
        for k, (wg, mg) in enumerate(zip(self.job.split(Wg), self.job.split(Mg))):
            assert _bits_equal(wg, self.W[k]) and _bits_equal(mg, self.M[k]), f"{label}: key {k}"


KEYS = (5, 1024, 8193, 40000, 3, 70001, 2048, 0, 131072)


@pytest.mark.parametrize("grouping", ["one", "per_key", "reversed", "sparse"])
def test_groups_launched_as_they_complete_match_the_oracle(lib, torch_dev, grouping):
    torch, dev = torch_dev
    K = len(KEYS)
    key_group = {"one": [0] * K, "per_key": list(range(K)),
                 "reversed": [K - 1 - k for k in range(K)],
                 "sparse": [3, 0, 3, 1, 0, 3, 1, 0, 3]}[grouping]   # group 2 has no key
    n_workers = 5
    _say("groups", grouping, key_group, "N", n_workers)
    c = Case(torch, dev, lib, n_workers, KEYS, key_group=key_group, seed=11)
    for t in range(3):
        host = c.host_grads()
        arenas = [torch.from_numpy(a).to(dev) for a in host]     # new buffers every step
        for w in range(n_workers):
            c.job.attach_grads(w, arenas[w])
        torch.cuda.synchronize()
        for k in reversed(range(K)):               # backward order, workers interleaved
            for w in reversed(range(n_workers)):
                c.job.push_key(w, k)
        c.job.step()
        c.oracle_step(host)
        c.check(f"{grouping} step {t}")
    c.job.destroy()


@pytest.mark.parametrize("grouped,batched,ordered,resident", [
    (False, False, False, None), (True, False, False, None), (True, True, False, None),
    (False, False, True, None), (True, False, True, None), (True, True, True, None),
    ("pairs", False, True, None), ("pairs", True, True, 8 * 100000), (False, False, True, 0)])
def test_ready_events_are_waited_on(lib, torch_dev, grouped, batched, ordered, resident):
    """Producers fill the gradient buffers on their own streams after a
    delay and record an event per key; the host pushes right away.  The step
    must read the produced values, not the zeros the buffers held.  Each
    worker's events are recorded on its own stream in push order, so the
    ordered-events option (a launch waits only for each worker's last event
    among its keys) holds too."""
    torch, dev = torch_dev
    keys = (300000, 70001, 8193, 1024, 5)
    n_workers = 4
    key_group = ([k // 2 for k in range(len(keys))] if grouped == "pairs" else
                 list(range(len(keys))) if grouped else None)
    _say("ready events,", "grouped" if grouped else "one launch", "batched" if batched else "per key",
         "ordered" if ordered else "")
    c = Case(torch, dev, lib, n_workers, keys, key_group=key_group, seed=12,
             ordered_events=ordered, resident_bytes=resident)
    host = c.host_grads()
    src = [torch.from_numpy(a).to(dev) for a in host]
    arenas = [torch.zeros(c.total, device=dev) for _ in range(n_workers)]
    for w in range(n_workers):
        c.job.attach_grads(w, arenas[w])
    delay = [torch.randn(2048, 2048, device=dev) * 1e-2 for _ in range(n_workers)]
    torch.cuda.synchronize()
    producers = [torch.cuda.Stream(device=dev) for _ in range(n_workers)]
    events = []
    for k in reversed(range(len(keys))):
        o, n = c.offs[k], keys[k]
        for w in range(n_workers):
            with torch.cuda.stream(producers[w]):
                d = delay[w]
                for _ in range(4):                 # the "backward" work of this layer
                    d = d @ d
                arenas[w][o:o + n].copy_(src[w][o:o + n])
                ev = torch.cuda.Event()
                ev.record(producers[w])
            events.append(ev)
            if batched:
                c.job.push_bucket(w, c.job.bucket(w, [k]), ev)
            else:
                c.job.push_key(w, k, ev)
    c.job.step()
    c.oracle_step(host)
    c.check("events")
    torch.cuda.synchronize()
    c.job.destroy()


def test_missing_push_leaves_completed_groups_applied(lib, torch_dev):
    torch, dev = torch_dev
    keys = (1024, 4096, 777)
    c = Case(torch, dev, lib, 3, keys, key_group=[0, 1, 1], seed=13)
    host = c.host_grads()
    arenas = [torch.from_numpy(a).to(dev) for a in host]
    for w in range(3):
        c.job.attach_grads(w, arenas[w])
    torch.cuda.synchronize()
    for k in range(3):
        for w in range(3):
            if (w, k) != (2, 2):
                c.job.push_key(w, k)
    # group 0 is complete and was enqueued: its keys cannot be pushed again
    rc = lib.phub_push(c.job.handle, 0, 0, c.job.key_pointers(arenas[0])[0], check=False)
    assert rc == phub.PHUB_ESTATE and "readiness group 0" in lib.last_error()
    assert lib.phub_step(c.job.handle, check=False) == phub.PHUB_ENOTREADY
    assert "worker 2" in lib.last_error() and "key 2" in lib.last_error()
    c.job.push_key(2, 2)
    c.job.step()
    c.oracle_step(host)
    c.check("completed after the missing push")
    # the next step starts clean: every key can be pushed again
    host = c.host_grads()
    for w in range(3):
        arenas[w].copy_(torch.from_numpy(host[w]))
    torch.cuda.synchronize()
    c.job.push_all()
    c.job.step()
    c.oracle_step(host)
    c.check("next step")
    c.job.destroy()


@pytest.mark.parametrize("resident", [1 << 40, 8 * 60000])
def test_grouped_job_with_cache_resident_state(lib, torch_dev, resident):
    """A grouped job whose state is wholly or partly cache-resident (both
    phases of the schedule in every group's launch) gives the same bits as
    the oracle too."""
    torch, dev = torch_dev
    c = Case(torch, dev, lib, 8, KEYS, key_group=[k % 3 for k in range(len(KEYS))], seed=14,
             resident_bytes=resident)
    frac = c.job.cached_fraction()
    assert frac == 1.0 if resident == 1 << 40 else 0.0 < frac < 1.0
    for t in range(2):
        host = c.host_grads()
        arenas = [torch.from_numpy(a).to(dev) for a in host]
        for w in range(8):
            c.job.attach_grads(w, arenas[w])
        torch.cuda.synchronize()
        c.job.push_all()
        c.job.step()
        c.oracle_step(host)
        c.check(f"resident={resident} grouped step {t}")
    c.job.destroy()
