"""Many steps of one job against the oracle, bit for bit.  The burst
write-back stashes a wave's state and writes it when the device clock's
write window opens, so which tiles a write-back covers changes from step
to step; 300 steps (gradients fixed, state evolving) walk through many of
those patterns, on the default grid and on a grid of 3 workgroups where
every wave walks many tiles.  Any step whose result depended on when its
state was written back would leave W or M off by the end."""

import sys

import numpy as np
import pytest

import oracle
from paper_1805_07891_amd.job import TorchJob, load_library
from paper_1805_07891_amd.workloads import Job, key_offsets

pytestmark = pytest.mark.gpu

KEYS = (7, 4096, 100003, 1 << 17, 65, 50001)
STEPS = 300


@pytest.mark.parametrize("n_workers,workgroups", [(8, None), (8, 3), (16, None)])
def test_many_steps_bit_exact(n_workers, workgroups):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    dev = torch.device("cuda:0")
    print(f"long run: N={n_workers} workgroups={workgroups} steps={STEPS}", flush=True)
    sys.stdout.flush()
    lib = load_library()
    spec = Job("long", n_workers, KEYS, lr=0.01, momentum=0.9, weight_decay=1e-4,
               nesterov=True, sigma_g=1e-2)
    job = TorchJob(spec, dev, lib=lib, workgroups=workgroups)
    offs, total = key_offsets(KEYS)
    rng = np.random.default_rng(20 + n_workers)
    w0 = np.zeros(total, np.float32)
    for o, n in zip(offs, KEYS):
        w0[o:o + n] = rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
    job.set_weights(torch.from_numpy(w0).to(dev))
    host = [np.zeros(total, np.float32) for _ in range(n_workers)]
    for a in host:
        for o, n in zip(offs, KEYS):
            a[o:o + n] = rng.standard_normal(n, dtype=np.float32) * np.float32(1e-2)
    dev_g = [torch.from_numpy(a).to(dev) for a in host]
    for w in range(n_workers):
        job.attach_grads(w, dev_g[w])
    torch.cuda.synchronize()
    for _ in range(STEPS):
        job.push_and_step()
    W = [w0[o:o + n].copy() for o, n in zip(offs, KEYS)]
    M = [np.zeros(n, np.float32) for n in KEYS]
    g = [[h[o:o + n] for o, n in zip(offs, KEYS)] for h in host]
    for _ in range(STEPS):
        oracle.step(g, W, M, spec.lr, spec.momentum, spec.weight_decay, True)
    for k, (pw, pm, _) in enumerate(job.pulled_keys()):
        assert np.array_equal(pw.view(np.uint32), W[k].view(np.uint32)), f"key {k}: W differs"
        assert np.array_equal(pm.view(np.uint32), M[k].view(np.uint32)), f"key {k}: M differs"
    job.destroy()
