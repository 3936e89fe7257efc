"""GPU tests of Pull (paper section 3.1): every key's state read through the
per-key pointers the library hands out, compared bit for bit with the oracle.

The other GPU tests read a job's state as whole arenas; here each key is
read on its own through phub_pull (W), phub_get_state (W, M) and
phub_get_second_moment (V), so a wrong per-key offset, a key left out of the
schedule, or a key whose cache-resident cut or readiness group misplaces it
fails.  Cases: a zero-length key, keys shorter than a float4, a key cut by
the cache-resident budget, keys in readiness groups, every optimizer, and a
read of the pulled pointer ordered after the step on the job's stream
without a host synchronisation.
"""

import ctypes
import sys

import numpy as np
import pytest

import oracle
from paper_1805_07891_amd.job import TorchJob, hip_runtime, load_library
from paper_1805_07891_amd.workloads import Job, key_offsets

pytestmark = pytest.mark.gpu

B1, B2, EPS = 0.9, 0.999, 1e-8
# a zero-length key, ragged keys, keys across several tiles and chunks
KEYS = (0, 5, 1, 1024, 8193, 3, 40000, 0, 70001, 64, 2 * 8192 + 3)


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


def _run(torch, dev, lib, n_workers, keys, steps, seed, optimizer="momentum", nesterov=True,
         resident_bytes=None, key_group=None):
    """`steps` steps on the GPU and in the oracle; returns the job (still
    live) and the oracle's per-key (W, M, V) lists."""
    spec = Job("pull", n_workers, tuple(keys), lr=0.1, momentum=0.9, weight_decay=1e-4,
               nesterov=nesterov, sigma_g=1e-2)
    job = TorchJob(spec, dev, lib=lib, resident_bytes=resident_bytes, key_group=key_group,
                   optimizer=None if optimizer == "momentum" else optimizer, betas=(B1, B2),
                   eps=EPS)
    offs, total = key_offsets(keys)
    rng = np.random.default_rng(seed)
    w0 = np.zeros(total, np.float32)
    for o, n in zip(offs, keys):
        w0[o:o + n] = rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
    job.set_weights(torch.from_numpy(w0).to(dev))
    W = [w0[o:o + n].copy() for o, n in zip(offs, keys)]
    M = [np.zeros(n, np.float32) for n in keys]
    V = [np.zeros(n, np.float32) for n in keys]
    for t in range(steps):
        host = []
        for _ in range(n_workers):
            a = np.zeros(total, np.float32)
            for o, n in zip(offs, keys):
                a[o:o + n] = rng.standard_normal(n, dtype=np.float32) * np.float32(1e-2)
            host.append(a)
        dev_g = [torch.from_numpy(a).to(dev) for a in host]
        for w in range(n_workers):
            job.attach_grads(w, dev_g[w])
        torch.cuda.synchronize()
        job.push_and_step()
        job.sync()
        g = [[h[o:o + n] for o, n in zip(offs, keys)] for h in host]
        if optimizer == "momentum":
            oracle.step(g, W, M, spec.lr, spec.momentum, spec.weight_decay, nesterov)
        elif optimizer == "sgd":
            oracle.step_sgd(g, W, spec.lr, spec.weight_decay)
        else:
            oracle.step_adam(g, W, M, V, spec.lr, B1, B2, EPS, spec.weight_decay, t + 1)
    return job, (W, None if optimizer == "sgd" else M, V if optimizer == "adam" else None)


def _check_pulled(job, ref, label):
    W, M, V = ref
    pulled = job.pulled_keys()
    assert len(pulled) == len(W)
    for k, (pw, pm, pv) in enumerate(pulled):
        n = job.spec.key_elems[k]
        assert pw is not None and pw.size == n, (label, k)
        assert _bits_equal(pw, W[k]), f"{label}: key {k} (n={n}) W through phub_pull differs"
        if M is None:
            assert pm is None, (label, k)
        else:
            assert _bits_equal(pm, M[k]), f"{label}: key {k} (n={n}) M differs"
        if V is None:
            assert pv is None, (label, k)
        else:
            assert _bits_equal(pv, V[k]), f"{label}: key {k} (n={n}) V differs"


def _check_layout(job):
    """Each key's pulled slice is 256-byte aligned, the slices of W (and of
    M, V) do not overlap, and the pointers do not move across steps."""
    spans = {0: [], 1: [], 2: []}
    for k, n in enumerate(job.spec.key_elems):
        w_pull, _, m, v = job.key_state_pointers(k)
        for i, p in enumerate((w_pull, m, v)):
            if p:
                assert p % 256 == 0, f"key {k}: state slice at {p:#x} is not 256-byte aligned"
                if n:
                    spans[i].append((p, p + 4 * n, k))
    for i, s in spans.items():
        s.sort()
        for (a0, a1, ka), (b0, b1, kb) in zip(s, s[1:]):
            assert a1 <= b0, f"state array {i}: keys {ka} and {kb} overlap"


@pytest.mark.parametrize("optimizer", ["momentum", "sgd", "adam"])
@pytest.mark.parametrize("resident", [None, 0, 8 * 9000])
def test_pull_every_key_matches_the_oracle(lib, torch_dev, optimizer, resident):
    """resident None: the default shared budget (all of this small state
    cached); 0: all of it streamed; 8 * 9000 bytes: a cut inside key 4
    (momentum, Adam) or key 6 (SGD), so that key is read partly with each
    policy."""
    torch, dev = torch_dev
    for n_workers in (1, 4, 8, 16, 17):
        _say("pull", optimizer, "resident", resident, "N", n_workers)
        job, ref = _run(torch, dev, lib, n_workers, KEYS, steps=3, seed=300 + n_workers,
                        optimizer=optimizer, resident_bytes=resident)
        before = [job.key_state_pointers(k) for k in range(len(KEYS))]
        _check_pulled(job, ref, f"{optimizer} N={n_workers} resident={resident}")
        _check_layout(job)
        job.push_and_step()  # the pointers stay where they were after another step
        job.sync()
        assert before == [job.key_state_pointers(k) for k in range(len(KEYS))]
        job.destroy()


@pytest.mark.parametrize("nesterov", [True, False])
def test_pull_with_readiness_groups(lib, torch_dev, nesterov):
    """Keys in readiness groups sit on the pointer table's rows in group
    order, not key order; pull must still give each key its own slice."""
    torch, dev = torch_dev
    key_group = [(3 * k + 1) % 4 for k in range(len(KEYS))]
    for n_workers in (2, 8):
        _say("pull groups N", n_workers, "nesterov", nesterov)
        job, ref = _run(torch, dev, lib, n_workers, KEYS, steps=2, seed=400 + n_workers,
                        nesterov=nesterov, key_group=key_group, resident_bytes=8 * 30000)
        _check_pulled(job, ref, f"groups N={n_workers}")
        _check_layout(job)
        job.destroy()


def test_pull_is_ordered_on_the_job_stream(lib, torch_dev):
    """A copy out of the pulled pointer enqueued on the job's stream right
    after phub_step (no host synchronisation between them) sees the step's
    result."""
    torch, dev = torch_dev
    keys = (70001, 5, 8193)
    n_workers = 4
    job, ref = _run(torch, dev, lib, n_workers, keys, steps=1, seed=501)
    W = ref[0]
    # one more step whose inputs are ready on the device before it is enqueued
    offs, total = key_offsets(keys)
    rng = np.random.default_rng(502)
    host = []
    for _ in range(n_workers):
        a = np.zeros(total, np.float32)
        for o, n in zip(offs, keys):
            a[o:o + n] = rng.standard_normal(n, dtype=np.float32) * np.float32(1e-2)
        host.append(a)
    dev_g = [torch.from_numpy(a).to(dev) for a in host]
    for w in range(n_workers):
        job.attach_grads(w, dev_g[w])
    outs = [torch.empty(n, dtype=torch.float32, device=dev) for n in keys]
    torch.cuda.synchronize()
    job.push_and_step()
    hip = hip_runtime()
    hip.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                   ctypes.c_int, ctypes.c_void_p]
    hip.hipMemcpyAsync.restype = ctypes.c_int
    for k, n in enumerate(keys):
        p = job.lib.phub_pull(job.handle, k)
        rc = hip.hipMemcpyAsync(outs[k].data_ptr(), p, 4 * n, 3, job.stream.cuda_stream)
        assert rc == 0
    job.sync()
    oracle.step([[h[o:o + n] for o, n in zip(offs, keys)] for h in host], W, ref[1],
                job.spec.lr, job.spec.momentum, job.spec.weight_decay, job.spec.nesterov)
    for k in range(len(keys)):
        assert _bits_equal(outs[k].cpu().numpy(), W[k]), f"key {k}"
    job.destroy()
