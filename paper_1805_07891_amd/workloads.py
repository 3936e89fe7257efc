"""Synthetic workloads and seeded input generators for the PHub exchange step.

This module holds no arithmetic of the method itself: it only describes the
key (layer) shapes of the models the paper trains (Table 3 in section 4.2),
the optimizer settings of each workload, and seeded random generators for
gradients and initial weights.  Both the HIP path and the CPU oracle take
their inputs from here, and nothing here depends on either of them.

A "key" is one layer's parameter tensor (the paper's key-value view of a
parameter server, section 2); only its element count matters to the exchange
step, so a model is described by the list of its key sizes in fp32 elements.

Inputs are synthetic, as in the paper's ZeroComputeEngine methodology
(section 4.4), where only the exchange runs: gradients are drawn from
N(0, sigma_g) and initial weights from N(0, sigma_w); momentum starts at 0.
"""

from __future__ import annotations

import dataclasses
import math
from typing import List, Sequence

import numpy as np

BASE_SEED = 180507891
ALIGN_ELEMS = 64  # key slices inside a worker arena start on 256-byte boundaries


# --------------------------------------------------------------------------
# Key shapes of the evaluated models (parameter tensors in model order).
# --------------------------------------------------------------------------

def resnet_v1_bottleneck_keys(blocks: Sequence[int], num_classes: int = 1000) -> List[int]:
    """ResNet v1 with bottleneck blocks: 7x7 stem, stages of widths
    64/128/256/512 with 4x expansion, a 1x1 projection on the first block of
    each stage, batch-norm gamma and beta after every convolution, and a
    final fully connected layer with bias.  Convolutions carry no bias."""
    keys = [64 * 3 * 7 * 7, 64, 64]
    in_ch = 64
    for stage, nblocks in enumerate(blocks):
        width = 64 << stage
        out_ch = 4 * width
        for b in range(nblocks):
            keys += [in_ch * width, width, width]          # 1x1 reduce + BN
            keys += [width * width * 9, width, width]      # 3x3 + BN
            keys += [width * out_ch, out_ch, out_ch]       # 1x1 expand + BN
            if b == 0:
                keys += [in_ch * out_ch, out_ch, out_ch]   # projection + BN
            in_ch = out_ch
    keys += [in_ch * num_classes, num_classes]
    return keys


def resnet50_keys() -> List[int]:
    return resnet_v1_bottleneck_keys([3, 4, 6, 3])


def resnet269_keys() -> List[int]:
    return resnet_v1_bottleneck_keys([3, 30, 48, 8])


def alexnet_keys() -> List[int]:
    """Five convolutions and three fully connected layers, each with bias;
    the FC layers (9216x4096, 4096x4096, 4096x1000) hold most parameters."""
    convs = [(3, 64, 11), (64, 192, 5), (192, 384, 3), (384, 256, 3), (256, 256, 3)]
    fcs = [(256 * 6 * 6, 4096), (4096, 4096), (4096, 1000)]
    keys: List[int] = []
    for cin, cout, k in convs:
        keys += [cout * cin * k * k, cout]
    for fin, fout in fcs:
        keys += [fout * fin, fout]
    return keys


def vgg19_keys() -> List[int]:
    """Sixteen 3x3 convolutions and three FC layers (25088x4096 first), each
    with bias."""
    chans = [64, 64, 128, 128, 256, 256, 256, 256, 512, 512, 512, 512, 512, 512, 512, 512]
    keys: List[int] = []
    cin = 3
    for cout in chans:
        keys += [cout * cin * 9, cout]
        cin = cout
    for fin, fout in [(512 * 7 * 7, 4096), (4096, 4096), (4096, 1000)]:
        keys += [fout * fin, fout]
    return keys


def inception_v3_keys() -> List[int]:
    """Inception-v3 without the auxiliary classifier: 94 bias-free
    convolutions each followed by batch-norm gamma and beta, then a 2048x1000
    FC layer with bias (284 keys)."""
    keys: List[int] = []

    def conv(cin, cout, kh, kw=None):
        kw = kh if kw is None else kw
        keys.extend([cout * cin * kh * kw, cout, cout])

    conv(3, 32, 3); conv(32, 32, 3); conv(32, 64, 3); conv(64, 80, 1); conv(80, 192, 3)

    def block_a(cin, pool):
        conv(cin, 64, 1)
        conv(cin, 48, 1); conv(48, 64, 5)
        conv(cin, 64, 1); conv(64, 96, 3); conv(96, 96, 3)
        conv(cin, pool, 1)

    def block_b(cin):
        conv(cin, 384, 3)
        conv(cin, 64, 1); conv(64, 96, 3); conv(96, 96, 3)

    def block_c(cin, c7):
        conv(cin, 192, 1)
        conv(cin, c7, 1); conv(c7, c7, 1, 7); conv(c7, 192, 7, 1)
        conv(cin, c7, 1); conv(c7, c7, 7, 1); conv(c7, c7, 1, 7); conv(c7, c7, 7, 1); conv(c7, 192, 1, 7)
        conv(cin, 192, 1)

    def block_d(cin):
        conv(cin, 192, 1); conv(192, 320, 3)
        conv(cin, 192, 1); conv(192, 192, 1, 7); conv(192, 192, 7, 1); conv(192, 192, 3)

    def block_e(cin):
        conv(cin, 320, 1)
        conv(cin, 384, 1); conv(384, 384, 1, 3); conv(384, 384, 3, 1)
        conv(cin, 448, 1); conv(448, 384, 3); conv(384, 384, 1, 3); conv(384, 384, 3, 1)
        conv(cin, 192, 1)

    block_a(192, 32); block_a(256, 64); block_a(288, 64)
    block_b(288)
    block_c(768, 128); block_c(768, 160); block_c(768, 160); block_c(768, 192)
    block_d(768)
    block_e(1280); block_e(2048)
    keys += [2048 * 1000, 1000]
    return keys


def tiny_keys(seed: int = 1805, num_keys: int = 32, lo_log2: int = 10, hi_log2: int = 17) -> List[int]:
    """Log-uniform key sizes in [2^lo, 2^hi] elements; most are not multiples
    of 4 or of the chunk size, so ragged tails are exercised."""
    rng = np.random.default_rng(seed)
    u = rng.random(num_keys)
    sizes = np.floor(2.0 ** (lo_log2 + (hi_log2 - lo_log2) * u)).astype(np.int64)
    sizes = np.clip(sizes, 1 << lo_log2, 1 << hi_log2)
    return [int(s) for s in sizes]


# --------------------------------------------------------------------------
# Workloads: key shapes plus optimizer settings and input scales.
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Job:
    """One training job (one tenant): N workers exchanging K keys."""
    name: str
    num_workers: int
    key_elems: tuple
    chunk_elems: int = 8192          # 32 KB chunks
    lr: float = 0.1
    momentum: float = 0.9
    weight_decay: float = 1e-4
    nesterov: bool = True
    sigma_g: float = 1e-3
    sigma_w: float = 0.05

    @property
    def num_keys(self) -> int:
        return len(self.key_elems)

    @property
    def num_params(self) -> int:
        return int(sum(self.key_elems))

    @property
    def chunk_bytes(self) -> int:
        return 4 * self.chunk_elems

    def hbm_bytes_per_step(self) -> int:
        """N gradient reads plus read and write of weights and momentum."""
        return (self.num_workers + 4) * self.num_params * 4

    def worker_grad_bytes_per_step(self) -> int:
        return self.num_workers * self.num_params * 4


@dataclasses.dataclass(frozen=True)
class Workload:
    """One or more concurrent jobs, stepped a fixed number of times."""
    name: str
    jobs: tuple
    steps: int
    seed_index: int

    def hbm_bytes_per_step(self) -> int:
        return sum(j.hbm_bytes_per_step() for j in self.jobs)

    def worker_grad_bytes_per_step(self) -> int:
        return sum(j.worker_grad_bytes_per_step() for j in self.jobs)


def _job(name, n, keys, **kw) -> Job:
    return Job(name=name, num_workers=n, key_elems=tuple(int(k) for k in keys), **kw)


def workload(name: str) -> Workload:
    """The five evaluation workloads by name."""
    if name == "tiny":
        return Workload("tiny", (_job("tiny", 4, tiny_keys(), sigma_g=1e-2),), steps=3, seed_index=0)
    if name == "resnet50":
        return Workload("resnet50", (_job("resnet50", 8, resnet50_keys()),), steps=10, seed_index=1)
    if name == "alexnet":
        return Workload("alexnet", (_job("alexnet", 8, alexnet_keys()),), steps=10, seed_index=2)
    if name == "resnet269":
        return Workload("resnet269", (_job("resnet269", 16, resnet269_keys()),), steps=10, seed_index=3)
    if name == "multitenant":
        jobs = (_job("resnet50.a", 8, resnet50_keys()),
                _job("resnet50.b", 8, resnet50_keys()),
                _job("inception_v3", 8, inception_v3_keys()),
                _job("vgg19", 8, vgg19_keys()))
        return Workload("multitenant", jobs, steps=5, seed_index=4)
    raise KeyError(f"unknown workload {name!r}")


WORKLOAD_NAMES = ("tiny", "resnet50", "alexnet", "resnet269", "multitenant")


# --------------------------------------------------------------------------
# Arena layout for inputs: one contiguous arena per worker, keys as aligned
# slices.  This is how the test and benchmark harness lay out gradients; the
# library itself accepts any 16-byte aligned pointer per (worker, key).
# --------------------------------------------------------------------------

def key_offsets(key_elems: Sequence[int], align: int = ALIGN_ELEMS) -> tuple:
    offs = []
    total = 0
    for n in key_elems:
        offs.append(total)
        total += (int(n) + align - 1) // align * align
    return tuple(offs), total


# --------------------------------------------------------------------------
# Seeds.
# --------------------------------------------------------------------------

def grad_seed(seed_index: int, job_index: int, step: int, worker: int) -> int:
    return BASE_SEED + 1_000_000 * seed_index + 100_000 * job_index + 1_000 * step + worker


def weight_seed(seed_index: int, job_index: int) -> int:
    return BASE_SEED + 1_000_000 * seed_index + 100_000 * job_index + 999


# --------------------------------------------------------------------------
# Host (numpy) generators: small cases that the oracle runs in full.
# --------------------------------------------------------------------------

def host_normal(seed: int, count: int, sigma: float) -> np.ndarray:
    """count fp32 values from N(0, sigma), PCG64 seeded."""
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(count, dtype=np.float32) * np.float32(sigma)).astype(np.float32)


def host_grad_arena(job: Job, seed_index: int, job_index: int, step: int, worker: int) -> np.ndarray:
    offs, total = key_offsets(job.key_elems)
    arena = np.zeros(total, dtype=np.float32)
    vals = host_normal(grad_seed(seed_index, job_index, step, worker), job.num_params, job.sigma_g)
    pos = 0
    for off, n in zip(offs, job.key_elems):
        arena[off:off + n] = vals[pos:pos + n]
        pos += n
    return arena


def host_weight_arena(job: Job, seed_index: int, job_index: int) -> np.ndarray:
    offs, total = key_offsets(job.key_elems)
    arena = np.zeros(total, dtype=np.float32)
    vals = host_normal(weight_seed(seed_index, job_index), job.num_params, job.sigma_w)
    pos = 0
    for off, n in zip(offs, job.key_elems):
        arena[off:off + n] = vals[pos:pos + n]
        pos += n
    return arena


# --------------------------------------------------------------------------
# Device (torch) generators: full-size cases.  Values come from torch's
# seeded device generator; a test that checks sampled outputs copies the
# sampled inputs back to the host for the oracle.
# --------------------------------------------------------------------------

def device_normal_arena(torch, device, seed: int, total: int, sigma: float):
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    t = torch.empty(total, dtype=torch.float32, device=device)
    t.normal_(0.0, sigma, generator=gen)
    return t


def device_grad_arena(torch, device, job: Job, seed_index: int, job_index: int, step: int, worker: int):
    _, total = key_offsets(job.key_elems)
    return device_normal_arena(torch, device, grad_seed(seed_index, job_index, step, worker), total, job.sigma_g)


def device_weight_arena(torch, device, job: Job, seed_index: int, job_index: int):
    _, total = key_offsets(job.key_elems)
    return device_normal_arena(torch, device, weight_seed(seed_index, job_index), total, job.sigma_w)


def describe(w: Workload) -> str:
    parts = []
    for j in w.jobs:
        parts.append(f"{j.name}: N={j.num_workers} K={j.num_keys} P={j.num_params:,} "
                     f"largest={max(j.key_elems):,}")
    return "; ".join(parts)


if __name__ == "__main__":
    for nm in WORKLOAD_NAMES:
        w = workload(nm)
        print(nm, describe(w), f"bytes/step={w.hbm_bytes_per_step()/1e9:.3f} GB")
