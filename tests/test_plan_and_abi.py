"""Host-side checks of the HIP library (no GPU needed).

The chunk schedule is pure host code exported through the C interface; it
is checked for exact coverage of every element, alignment, small-key
bundling, refinement and the LPT balance bound.  The library must export
every function the header declares, and calls that fail argument checks
must return their error code before touching the GPU.
"""

import itertools
import os
import re

import numpy as np
import subprocess

import pytest

from paper_1805_07891_amd import phub, workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "phub.h")
SEG_COST = 4096


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(phub.DEFAULT_LIB):
        from paper_1805_07891_amd import build
        build.build()
    return phub.load()


def test_header_symbols_are_exported(lib):
    with open(HEADER) as f:
        text = f.read()
    declared = set(re.findall(r"^\s*(?:int|const char \*)\s*(phub_\w+)\s*\(", text, re.M))
    assert declared, "no declarations parsed"
    assert declared == set(phub.EXPORTED)
    for name in declared:
        assert hasattr(lib.lib, name), name


def test_probe_header_symbols_are_exported():
    """The bandwidth probe library exports exactly what its header declares
    (loaded without calling anything: no GPU here)."""
    import ctypes
    from paper_1805_07891_amd import build
    if not os.path.exists(build.PROBE_LIB):
        build.build_probe()
    with open(os.path.join(ROOT, "include", "phub_probe.h")) as f:
        text = f.read()
    declared = set(re.findall(r"^\s*int\s*(phub_\w+)\s*\(", text, re.M))
    assert declared == {"phub_probe_read", "phub_probe_write", "phub_probe_mixed",
                        "phub_probe_tile_elems"}
    probe = ctypes.CDLL(build.PROBE_LIB)
    for name in declared:
        assert hasattr(probe, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", build.PROBE_LIB], capture_output=True,
                         text=True, check=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if " T " in ln and "phub_" in ln}
    assert exported == declared


LPT = phub.PHUB_SCHEDULE_LPT
SPLIT = phub.PHUB_SCHEDULE_SPLIT


def _check_plan(lib, n_workers, key_elems, chunk_bytes, groups, min_items=0, schedule=LPT):
    segs, gb, gc, item = lib.phub_plan_build(n_workers, key_elems, chunk_bytes, groups, min_items,
                                             schedule)
    used = len(gb) - 1
    assert gb[0] == 0 and gb[-1] == len(segs)
    assert all(b >= a for a, b in zip(gb, gb[1:]))
    assert used <= groups
    if schedule == LPT:
        assert all(gb[g + 1] > gb[g] for g in range(used)), "a bin without work"
    else:
        assert used == groups
    # coverage: every element of every key exactly once
    covered = [np.zeros(n, dtype=np.int8) for n in key_elems]
    for key, count, off in segs:
        assert count >= 1 and off >= 0 and off + count <= key_elems[key]
        assert off % 4 == 0, "segment start breaks 16-byte alignment"
        assert count <= chunk_bytes // 4 and (schedule == SPLIT or count <= item)
        covered[key][off:off + count] += 1
    for k, c in enumerate(covered):
        assert c.size == 0 or (c.min() == 1 and c.max() == 1), f"key {k} not covered exactly once"
    # costs add up
    per_elem = (n_workers + 4) * 4
    expect_total = sum(c * per_elem + SEG_COST for _, c, _ in segs)
    assert sum(gc) == expect_total
    for g in range(used):
        seg_cost = sum(segs[i][1] * per_elem + SEG_COST for i in range(gb[g], gb[g + 1]))
        assert gc[g] == seg_cost
        # segments of a workgroup in key, then offset, order
        keys = [(segs[i][0], segs[i][2]) for i in range(gb[g], gb[g + 1])]
        assert keys == sorted(keys)
    return segs, gb, gc, item


@pytest.mark.parametrize("name", workloads.WORKLOAD_NAMES)
@pytest.mark.parametrize("groups", [1, 7, 256, 1024])
@pytest.mark.parametrize("schedule", [LPT, SPLIT])
def test_plan_covers_workloads(lib, name, groups, schedule):
    for j in workloads.workload(name).jobs:
        _check_plan(lib, j.num_workers, j.key_elems, j.chunk_bytes, groups, min_items=512,
                    schedule=schedule)


@pytest.mark.parametrize("name", ["tiny", "resnet50", "alexnet", "resnet269"])
@pytest.mark.parametrize("bins", [1, 5, 1024])
def test_split_is_balanced_and_contiguous(lib, name, bins):
    j = workloads.workload(name).jobs[0]
    segs, bb, bc, item = _check_plan(lib, j.num_workers, j.key_elems, j.chunk_bytes, bins,
                                     schedule=SPLIT)
    # every bin holds the same number of float4 slots, to within one
    slots = [sum((c + 3) // 4 for _, c, _ in segs[bb[b]:bb[b + 1]]) for b in range(bins)]
    assert max(slots) - min(slots) <= 1
    # bins are contiguous runs in key order: concatenated, they walk the keys in order
    flat = [(k, o, c) for k, c, o in segs]
    for (k0, o0, c0), (k1, o1, c1) in zip(flat, flat[1:]):
        assert (k1 == k0 and o1 == o0 + c0) or (k1 > k0 and o1 == 0 and o0 + c0 == j.key_elems[k0])
    # no segment crosses a chunk boundary
    C = j.chunk_bytes // 4
    for k, o, c in flat:
        assert o // C == (o + c - 1) // C


def test_split_with_more_bins_than_float4_slots(lib):
    segs, bb, bc, item = _check_plan(lib, 3, [5, 2, 0, 1], 32768, 64, schedule=SPLIT)
    assert len(bb) == 65 and sum(1 for b in range(64) if bb[b + 1] > bb[b]) == 4


EDGE_SIZES = [1, 2, 3, 4, 5, 7, 8, 15, 16, 17, 1023, 1024, 1025, 8191, 8192, 8193, 2 * 8192 + 3, 0]


@pytest.mark.parametrize("chunk_bytes", [16, 48, 4096, 32768, 1 << 22])
@pytest.mark.parametrize("groups", [1, 3, 64])
@pytest.mark.parametrize("schedule", [LPT, SPLIT])
def test_plan_edge_shapes(lib, chunk_bytes, groups, schedule):
    _check_plan(lib, 3, EDGE_SIZES, chunk_bytes, groups, schedule=schedule)


def test_plan_bundles_small_keys(lib):
    # 100 keys of 100 elements with 8192-element chunks: bundles of <= 81 keys
    keys = [100] * 100
    segs, gb, gc, item = _check_plan(lib, 4, keys, 32768, 1 << 30)
    assert len(gb) - 1 == 2  # two items: 81 keys and 19 keys
    sizes = sorted(gb[g + 1] - gb[g] for g in range(2))
    assert sizes == [19, 81]


def test_plan_bundle_does_not_span_a_large_key(lib):
    keys = [10, 10, 20000, 10]
    segs, gb, gc, item = _check_plan(lib, 2, keys, 32768, 1 << 30)
    # items: {0,1}, three chunks of key 2, {3}
    assert len(gb) - 1 == 5


def test_plan_refines_to_reach_min_items(lib):
    keys = [8192 * 4]
    _, gb, _, item = _check_plan(lib, 2, keys, 32768, 1 << 30, min_items=16)
    assert item == 2048 and len(gb) - 1 == 16
    # never below 1024 elements
    _, gb, _, item = _check_plan(lib, 2, keys, 32768, 1 << 30, min_items=10 ** 6)
    assert item == 1024 and len(gb) - 1 == 32
    # min_items 0: chunks as given
    _, gb, _, item = _check_plan(lib, 2, keys, 32768, 1 << 30, min_items=0)
    assert item == 8192 and len(gb) - 1 == 4


def test_plan_one_item_per_group_is_in_decreasing_cost(lib):
    keys = [5000, 9000, 300, 20000, 7]
    segs, gb, gc, item = _check_plan(lib, 4, keys, 32768, 1 << 30)
    assert gc == sorted(gc, reverse=True)


def _lpt_opt_bruteforce(costs, groups):
    best = None
    for assign in itertools.product(range(groups), repeat=len(costs)):
        loads = [0] * groups
        for c, g in zip(costs, assign):
            loads[g] += c
        m = max(loads)
        best = m if best is None else min(best, m)
    return best


@pytest.mark.parametrize("seed", range(12))
def test_plan_lpt_within_graham_bound(lib, seed):
    rng = np.random.default_rng(seed)
    groups = int(rng.integers(2, 4))
    # keys of 1024..3072 elements with 1024-element chunks: every key is at
    # least one chunk, so nothing is bundled and each chunk is one item
    chunk = 1024
    keys, n_items = [], 0
    while True:
        n = int(rng.choice([1024, 1536, 2048, 2560, 3072]))
        c = -(-n // chunk)
        if n_items + c > 9:
            break
        keys.append(n)
        n_items += c
    assert n_items > groups
    segs, gb, gc, item = _check_plan(lib, 2, keys, chunk * 4, groups)
    assert len(segs) == n_items
    costs = [c * (2 + 4) * 4 + SEG_COST for _, c, _ in segs]
    opt = _lpt_opt_bruteforce(costs, groups)
    assert max(gc) <= (4 / 3 - 1 / (3 * groups)) * opt + 1e-9


@pytest.mark.parametrize("name", ["resnet50", "alexnet", "resnet269"])
def test_plan_list_scheduling_bound_on_workloads(lib, name):
    # any list schedule: makespan <= total / G + largest item; an item holds
    # at most `item` elements in at most item / (smallest key) segments
    j = workloads.workload(name).jobs[0]
    G = 256
    segs, gb, gc, item = _check_plan(lib, j.num_workers, j.key_elems, j.chunk_bytes, G)
    max_segs = -(-item // min(j.key_elems))
    largest = item * (j.num_workers + 4) * 4 + SEG_COST * max_segs
    assert max(gc) <= sum(gc) / G + largest


@pytest.mark.parametrize("args", [
    dict(num_workers=0), dict(num_workers=4097), dict(chunk_bytes=0), dict(chunk_bytes=8),
    dict(chunk_bytes=40), dict(chunk_bytes=(1 << 30) + 16), dict(key_elems=[5, -1]),
    dict(key_elems=[1 << 40]), dict(groups=0), dict(min_items=-1), dict(schedule=2),
    dict(schedule=-1),
])
def test_plan_rejects_bad_arguments(lib, args):
    a = dict(num_workers=2, key_elems=[5, 9], chunk_bytes=32768, groups=4, min_items=0,
             schedule=LPT)
    a.update(args)
    with pytest.raises(phub.PhubError) as e:
        lib.phub_plan_count(a["num_workers"], a["key_elems"], a["chunk_bytes"], a["groups"],
                            a["min_items"], a["schedule"])
    assert e.value.code == phub.PHUB_EINVAL
    assert lib.last_error()


def test_init_rejects_bad_arguments_before_touching_the_gpu(lib):
    for kw in [dict(num_workers=0), dict(chunk_bytes=20), dict(lr=float("nan")),
               dict(momentum=float("inf")), dict(schedule=7), dict(resident_bytes=-2),
               dict(key_group=[0, 2], num_groups=2), dict(key_group=[0, -1]),
               dict(key_group=[0, 1], num_groups=-1), dict(key_group=None, num_groups=3),
               dict(key_group=[0, 1], unfused=True), dict(optimizer=7),
               dict(optimizer=2, beta1=1.0), dict(optimizer=2, beta2=-0.5),
               dict(optimizer=2, eps=-1.0), dict(optimizer=2, eps=float("inf")),
               dict(workgroups=-1), dict(workgroups=1 << 17), dict(key_elems=[4, 1 << 34]),
               dict(ordered_events=2), dict(ordered_events=-1), dict(whole_chunks=2)]:
        a = dict(num_workers=2, key_elems=[4, 4], chunk_bytes=32768, lr=0.1, momentum=0.9,
                 weight_decay=1e-4, nesterov=True, schedule=None, resident_bytes=None,
                 key_group=None, num_groups=None, unfused=False, optimizer=None, beta1=0.9,
                 beta2=0.999, eps=1e-8, workgroups=None, ordered_events=0, whole_chunks=0)
        a.update(kw)
        rc, h = lib.phub_init(a["num_workers"], a["key_elems"], a["chunk_bytes"], a["lr"],
                              a["momentum"], a["weight_decay"], a["nesterov"], check=False,
                              schedule=a["schedule"], resident_bytes=a["resident_bytes"],
                              key_group=a["key_group"], num_groups=a["num_groups"],
                              unfused=a["unfused"], optimizer=a["optimizer"], beta1=a["beta1"],
                              beta2=a["beta2"], eps=a["eps"], workgroups=a["workgroups"],
                              ordered_events=a["ordered_events"], whole_chunks=a["whole_chunks"])
        assert rc == phub.PHUB_EINVAL and h is None, kw


def test_calls_on_a_dead_handle_return_estate(lib):
    for fn in (lambda: lib.phub_step(None, check=False),
               lambda: lib.phub_step(12345678, check=False),
               lambda: lib.phub_push(None, 0, 0, 0, check=False),
               lambda: lib.phub_push_event(None, 0, 0, 0, None, check=False),
               lambda: lib.phub_sync(None, check=False),
               lambda: lib.phub_destroy(None, check=False)):
        assert fn() == phub.PHUB_ESTATE
    assert "live job" in lib.last_error()


def test_noalloc_step_rejects_bad_arguments_before_touching_the_gpu(lib):
    """Every argument error of phub_step_noalloc, including a step whose
    schedule would not fit the library's scratch array, is found on the host
    before any HIP call (there is no GPU here): the pointers below are never
    dereferenced."""
    fake = 1 << 20  # a 16-byte aligned address that is never used
    for kw in [dict(num_workers=0), dict(chunk_bytes=20), dict(lr=float("nan")),
               dict(weight_decay=float("inf")), dict(key_elems=[4, 1 << 34]),
               dict(grads=[0, fake, fake, fake]), dict(grads=[fake + 4, fake, fake, fake]),
               dict(weights=0), dict(moments=fake + 8),
               dict(key_elems=[300 << 20, 4]),              # about 4.7 MB of tiles
               dict(num_workers=2, key_elems=[1] * 300000,  # 4.8 MB of gradient pointers
                    grads=[fake] * 600000)]:
        a = dict(num_workers=2, key_elems=[4, 4], chunk_bytes=32768, lr=0.1, momentum=0.9,
                 weight_decay=1e-4, nesterov=True, grads=[fake] * 4, weights=fake,
                 moments=fake)
        a.update(kw)
        rc = lib.phub_step_noalloc(a["num_workers"], a["key_elems"], a["chunk_bytes"], a["lr"],
                                   a["momentum"], a["weight_decay"], a["nesterov"], a["grads"],
                                   a["weights"], a["moments"], check=False)
        assert rc == phub.PHUB_EINVAL, (kw.keys(), rc, lib.last_error())
    assert "scratch" in lib.last_error()
