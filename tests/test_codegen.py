"""Code generation of the fused kernels (CPU only: the HIP source is
cross-compiled for gfx950 to assembly, and each kernel's metadata and body
are read).

The step is HBM-bound, so its kernels must keep every value in registers:
no scratch memory, no spilled vector registers, and no LDS (a stray LDS
copy of the launch scalars once cost plain SGD 3-6 points) except the
burst write-back stash of the streamed bin, in exactly the fixed-N kernels
that have it: those without pushpull with at least 6 workers for momentum
and plain SGD, at least 14 for Adam, each wave holding as many tiles' state
as fit 40 KB (4 waves per block).  Those kernels read the device's wall
clock (the write phases of the burst write-back) and no other kernel does.
The gradient loads must keep the non-temporal hint (gradients are read
once), and the fixed-N kernels must fit one wave per SIMD.
"""

import re

import pytest

from paper_1805_07891_amd import build


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    out = tmp_path_factory.mktemp("asm") / "fused_step.s"
    return open(build.device_assembly(str(out))).read()


def _kernels(asm):
    """name -> metadata dict of every kernel in the code object."""
    meta = {}
    for block in asm.split("  - .agpr_count:")[1:]:
        name = re.search(r"\.name:\s+(\S+)", block).group(1)
        fields = {}
        for key in ("group_segment_fixed_size", "private_segment_fixed_size", "vgpr_count",
                    "vgpr_spill_count", "sgpr_count"):
            fields[key] = int(re.search(rf"\.{key}:\s+(\d+)", block).group(1))
        meta[name] = fields
    return meta


def _body(asm, name):
    start = asm.index(name + ":")
    return asm[start:asm.index(".Lfunc_end", start)]


def _stash_lds(name):
    """LDS bytes the kernel should hold: its write-back stash, if any."""
    m = re.search(r"fused_step_fixedILi(\d+)ELi(\d)ELb(\d)E", name)
    if not m:
        return 0
    nw, opt, pull = int(m.group(1)), int(m.group(2)), m.group(3) == "1"
    s = {0: 2, 1: 2, 2: 1, 3: 3}[opt]
    least = {1: 6, 2: 6, 3: 14}[s]
    if pull or nw < least or not (nw <= 16 or nw in (20, 24, 32)):
        return 0
    tiles = (40 * 1024) // (s * 4 * 1024)
    return 4 * tiles * s * 4 * 1024


def test_stash_rule_covers_the_measured_cases():
    # momentum / Nesterov and plain SGD with 6-16 workers, Adam with 14-16;
    # never with pushpull
    with_stash = sorted((nw, opt) for nw in range(1, 17) for opt in range(4)
                        if _stash_lds(f"fused_step_fixedILi{nw}ELi{opt}ELb0E"))
    assert with_stash == sorted([(n, o) for n in range(6, 17) for o in (0, 1, 2)] +
                                [(n, 3) for n in range(14, 17)])
    assert _stash_lds("fused_step_fixedILi16ELi1ELb0E") == 160 * 1024
    assert _stash_lds("fused_step_fixedILi8ELi1ELb0E") == 160 * 1024
    assert _stash_lds("fused_step_fixedILi8ELi2ELb0E") == 160 * 1024
    assert _stash_lds("fused_step_fixedILi5ELi1ELb0E") == 0
    assert _stash_lds("fused_step_fixedILi13ELi3ELb0E") == 0
    assert _stash_lds("fused_step_fixedILi16ELi3ELb0E") == 144 * 1024
    assert _stash_lds("fused_step_fixedILi16ELi1ELb1E") == 0


def test_only_burst_kernels_read_the_wall_clock(asm):
    for name in _kernels(asm):
        reads = "s_memrealtime" in _body(asm, name)
        assert reads == bool(_stash_lds(name)), name


def test_every_kernel_keeps_its_data_in_registers(asm):
    meta = _kernels(asm)
    fixed = [n for n in meta if "fused_step_fixed" in n]
    # N = 1..16, 20, 24 and 32, four optimizer forms, with and without pushpull
    assert len(fixed) == 19 * 4 * 2
    assert any("fused_step_any" in n for n in meta)
    assert any("aggregate_only" in n for n in meta) and any("optimize_only" in n for n in meta)
    for name, m in meta.items():
        assert m["group_segment_fixed_size"] == _stash_lds(name), f"{name}: LDS size"
        assert m["private_segment_fixed_size"] == 0, f"{name} uses scratch"
        assert m["vgpr_spill_count"] == 0, f"{name} spills vector registers"
    for name in fixed:
        assert meta[name]["vgpr_count"] <= 512, name


def test_gradient_loads_are_non_temporal(asm):
    meta = _kernels(asm)
    for name in meta:
        if "fused_step_fixed" not in name:
            continue
        loads = re.findall(r"^\s+global_load_dwordx4\b.*$", _body(asm, name), re.M)
        nt = [line for line in loads if re.search(r"\bnt\b", line)]
        assert loads and nt, name


def test_the_only_atomics_are_vector_atomics_of_the_dynamic_schedule(asm):
    """The dynamic schedule's takes are vector atomics from one lane (the
    only read-modify-write the kernels do); no other kind appears."""
    meta = _kernels(asm)
    for name in meta:
        ops = {m.split()[0] for m in re.findall(r"^\s+(\S*atomic\S*)", _body(asm, name), re.M)}
        if "fused_step_fixed" in name:
            assert ops == {"global_atomic_add_x2"}, (name, ops)
        else:
            assert not ops, (name, ops)

