"""Code generation of the fused kernels (CPU only: the HIP source is
cross-compiled for gfx950 to assembly, and each kernel's metadata and body
are read).

The step is HBM-bound, so its kernels must keep every value in registers:
no LDS (the kernels have no use for it; a stray LDS copy of the launch
scalars once cost plain SGD 3-6 points), no scratch memory, no spilled
vector registers.  The gradient loads must keep the non-temporal hint
(gradients are read once), and the fixed-N kernels must fit one wave per
SIMD.
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


def test_every_kernel_keeps_its_data_in_registers(asm):
    meta = _kernels(asm)
    fixed = [n for n in meta if "fused_step_fixed" in n]
    # N = 1..16, four optimizer forms, with and without pushpull
    assert len(fixed) == 16 * 4 * 2
    assert any("fused_step_any" in n for n in meta)
    assert any("aggregate_only" in n for n in meta) and any("optimize_only" in n for n in meta)
    for name, m in meta.items():
        assert m["group_segment_fixed_size"] == 0, f"{name} uses LDS"
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
