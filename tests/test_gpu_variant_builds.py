"""GPU parity of the ablation builds of the library: the build whose kernels
load the gradients cache-allocating (PHUB_GRADIENT_LOADS_CACHED; built by
``python -m paper_1805_07891_amd.build --gradients-cached``, run by
``bench.py --library``) must give the default's bits, since it changes only
the loads' cache policy.  Skipped where that build is absent (the default
build step does not make it)."""

import os
import sys

import numpy as np
import pytest

import oracle
from paper_1805_07891_amd import build as hip_build
from paper_1805_07891_amd.job import TorchJob, load_library
from paper_1805_07891_amd.workloads import Job, key_offsets

pytestmark = pytest.mark.gpu

# ragged keys across several tiles and chunks, a zero-length key
KEYS = (5, 1024, 8193, 0, 40000, 70001, 3, 2 * 8192 + 3)


def _bits_equal(a, b):
    return np.array_equal(np.asarray(a, np.float32).view(np.uint32),
                          np.asarray(b, np.float32).view(np.uint32))


@pytest.mark.skipif(not os.path.exists(hip_build.GRADIENTS_CACHED_LIB),
                    reason="the gradients-cached ablation build is not built")
@pytest.mark.parametrize("n_workers,resident_bytes", [(8, None), (8, 1 << 16), (4, None), (16, 0)])
def test_gradients_cached_build_matches_oracle(n_workers, resident_bytes):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    dev = torch.device("cuda:0")
    print(f"gradients-cached build: N={n_workers} resident={resident_bytes}", flush=True)
    sys.stdout.flush()
    lib = load_library(hip_build.GRADIENTS_CACHED_LIB)
    spec = Job("gc", n_workers, KEYS, lr=0.1, momentum=0.9, weight_decay=1e-4, nesterov=True,
               sigma_g=1e-2)
    job = TorchJob(spec, dev, lib=lib, resident_bytes=resident_bytes)
    offs, total = key_offsets(KEYS)
    rng = np.random.default_rng(1805 + n_workers)
    w0 = np.zeros(total, np.float32)
    for o, n in zip(offs, KEYS):
        w0[o:o + n] = rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
    job.set_weights(torch.from_numpy(w0).to(dev))
    W = [w0[o:o + n].copy() for o, n in zip(offs, KEYS)]
    M = [np.zeros(n, np.float32) for n in KEYS]
    for _ in range(3):
        host = [np.zeros(total, np.float32) for _ in range(n_workers)]
        for a in host:
            for o, n in zip(offs, KEYS):
                a[o:o + n] = rng.standard_normal(n, dtype=np.float32) * np.float32(1e-2)
        dev_g = [torch.from_numpy(a).to(dev) for a in host]
        for w in range(n_workers):
            job.attach_grads(w, dev_g[w])
        torch.cuda.synchronize()
        job.push_and_step()
        job.sync()
        oracle.step([[h[o:o + n] for o, n in zip(offs, KEYS)] for h in host], W, M,
                    spec.lr, spec.momentum, spec.weight_decay, True)
    for k, (pw, pm, _) in enumerate(job.pulled_keys()):
        assert _bits_equal(pw, W[k]), f"key {k}: W differs"
        assert _bits_equal(pm, M[k]), f"key {k}: M differs"
    job.destroy()
