"""The library used from C alone: tests/native/c_api_step.c drives a job
through include/phub.h (init, set_weights, push in reverse worker order,
step, sync, pull, get_state, destroy), with gradients copied in by the HIP
runtime, and compares every key with the C oracle bit for bit; it also
checks that a step without every push is refused.  The program is compiled
by gcc against the in-tree libphub.so and run in a process of its own."""

import os
import shutil
import subprocess
import sys

import pytest

from paper_1805_07891_amd import build as hip_build

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_c_program_matches_oracle(tmp_path):
    assert os.path.exists(hip_build.LIB), "libphub.so is not built"
    exe = tmp_path / "c_api_step"
    pkg = os.path.dirname(hip_build.LIB)
    subprocess.check_call([
        "gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-D__HIP_PLATFORM_AMD__",
        f"-I{ROCM}/include", f"-I{os.path.join(ROOT, 'include')}", "-o", str(exe),
        os.path.join(ROOT, "tests", "native", "c_api_step.c"),
        os.path.join(ROOT, "oracle", "phub_oracle.c"),
        f"-L{pkg}", "-lphub", f"-L{ROCM}/lib", "-lamdhip64",
        f"-Wl,-rpath,{pkg}", f"-Wl,-rpath,{ROCM}/lib", "-lm"])
    print("running the C program", flush=True)
    sys.stdout.flush()
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c api checks passed" in r.stdout, r.stdout
