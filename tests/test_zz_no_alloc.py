"""phub_step_noalloc (the entry point that allocates nothing) against the job
path (phub_init + phub_push_all + phub_step) on the same inputs: the updated
W and M must be bit for bit the same, and the oracle's.  Two calls in a
row, the second with a smaller input (fewer workers, fewer and smaller
keys), so the second call runs on what the first left in the library's
scratch array; then a call whose schedule does not fit the scratch array
must be refused with nothing changed."""

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


def _inputs(n_workers, keys, seed):
    offs, total = key_offsets(keys)
    rng = np.random.default_rng(seed)
    w0 = np.zeros(total, np.float32)
    grads = [np.zeros(total, np.float32) for _ in range(n_workers)]
    for o, n in zip(offs, keys):
        w0[o:o + n] = rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
        for g in grads:
            g[o:o + n] = rng.standard_normal(n, dtype=np.float32) * np.float32(1e-2)
    return offs, total, w0, grads


def _compare(torch, dev, lib, n_workers, keys, seed, nesterov):
    spec = Job("noalloc", n_workers, tuple(keys), nesterov=nesterov, sigma_g=1e-2)
    offs, total, w0, grads = _inputs(n_workers, keys, seed)
    dev_g = [torch.from_numpy(g).to(dev) for g in grads]
    # the job path
    job = TorchJob(spec, dev, lib=lib)
    job.set_weights(torch.from_numpy(w0).to(dev))
    for w in range(n_workers):
        job.attach_grads(w, dev_g[w])
    torch.cuda.synchronize()
    job.push_and_step()
    Wj, Mj = job.state_arenas()
    job.destroy()
    # the entry point without allocation, on caller arenas of the same layout
    W = torch.from_numpy(w0).to(dev)
    M = torch.zeros(total, dtype=torch.float32, device=dev)
    ptrs = [dev_g[w].data_ptr() + 4 * offs[k] for w in range(n_workers) for k in range(len(keys))]
    torch.cuda.synchronize()
    lib.phub_step_noalloc(n_workers, keys, spec.chunk_bytes, spec.lr, spec.momentum,
                          spec.weight_decay, nesterov, ptrs, W.data_ptr(), M.data_ptr(),
                          stream=torch.cuda.current_stream(dev).cuda_stream)
    torch.cuda.synchronize()
    Wn, Mn = W.cpu().numpy(), M.cpu().numpy()
    # the oracle
    Wo = [w0[o:o + n].copy() for o, n in zip(offs, keys)]
    Mo = [np.zeros(n, np.float32) for n in keys]
    oracle.step([[g[o:o + n] for o, n in zip(offs, keys)] for g in grads], Wo, Mo, spec.lr,
                spec.momentum, spec.weight_decay, nesterov)
    for k, (o, n) in enumerate(zip(offs, keys)):
        assert _bits_equal(Wn[o:o + n], Wj[o:o + n]), f"key {k}: W differs from the job path"
        assert _bits_equal(Mn[o:o + n], Mj[o:o + n]), f"key {k}: M differs from the job path"
        assert _bits_equal(Wn[o:o + n], Wo[k]), f"key {k}: W differs from the oracle"
        assert _bits_equal(Mn[o:o + n], Mo[k]), f"key {k}: M differs from the oracle"
    # padding between keys untouched
    pad = np.ones(total, bool)
    for o, n in zip(offs, keys):
        pad[o:o + n] = False
    assert not Wn[pad].any() and not Mn[pad].any()


def test_noalloc_step_matches_the_job_path_twice(lib, torch_dev):
    torch, dev = torch_dev
    big = (5, 1024, 8193, 40000, 3, 70001, 1 << 20, 0, 333)
    small = (7, 3000, 1)
    _say("noalloc: 8 workers, keys", big)
    _compare(torch, dev, lib, 8, big, seed=1, nesterov=True)
    _say("noalloc: 4 workers, keys", small)
    _compare(torch, dev, lib, 4, small, seed=2, nesterov=False)
    _say("noalloc: 16 workers, keys", small)
    _compare(torch, dev, lib, 16, small, seed=3, nesterov=True)


def test_noalloc_step_refuses_a_schedule_beyond_its_scratch(lib, torch_dev):
    torch, dev = torch_dev
    n = 300 << 20  # 300 M parameters: about 4.7 MB of tiles
    # full-size buffers, so that nothing could be out of bounds even if the
    # call were not refused
    W = torch.zeros(n, dtype=torch.float32, device=dev)
    M = torch.zeros(n, dtype=torch.float32, device=dev)
    g = torch.ones(n, dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    with pytest.raises(phub.PhubError) as err:
        lib.phub_step_noalloc(2, (n,), 32768, 0.1, 0.9, 1e-4, True, [g.data_ptr()] * 2,
                              W.data_ptr(), M.data_ptr())
    assert err.value.code == phub.PHUB_EINVAL
    assert "scratch" in lib.last_error()
    torch.cuda.synchronize()
    assert not W.any() and not M.any()
    del W, M, g
    torch.cuda.empty_cache()
