"""The CPU code built with AddressSanitizer and UndefinedBehaviorSanitizer
(no GPU needed): the C oracle (oracle/phub_oracle.c) and the host chunk
schedule of the library (paper_1805_07891_amd/csrc/plan.cpp, section
3.2.4), each driven by a native checker under tests/sanitize/ that runs
the oracle's worked example and shape sweeps, and the schedule's coverage
and balance checks over the five workloads' key lists.  Any out-of-bounds
access, leak or undefined behaviour aborts the checker."""

import os
import shutil
import subprocess

import pytest

from paper_1805_07891_amd import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-g", "-O1"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(cmd, *args):
    r = subprocess.run([cmd, *args], capture_output=True, text=True, env=ENV, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "runtime error" not in r.stderr and "Sanitizer" not in r.stderr, r.stderr
    return r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers(tmp_path):
    exe = tmp_path / "oracle_check"
    subprocess.check_call(["gcc", "-std=c11", "-ffp-contract=off", "-fno-fast-math", *SAN, "-o",
                           str(exe), os.path.join(ROOT, "oracle", "phub_oracle.c"),
                           os.path.join(ROOT, "tests", "sanitize", "oracle_check.c"), "-lm"])
    out = _run(str(exe), os.path.join(ROOT, "tests", "golden", "worked_example.txt"))
    assert "oracle checks passed" in out


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_schedule_under_sanitizers(tmp_path):
    lists = tmp_path / "keys.txt"
    with open(lists, "w") as f:
        for name in workloads.WORKLOAD_NAMES:
            for job in workloads.workload(name).jobs:
                f.write(" ".join(str(x) for x in (job.num_workers, *job.key_elems)) + "\n")
        f.write("3 0 1 2 3 4 5 0 8191 8192 8193 1\n1 0\n17 4097 3 1024 1025\n")
    exe = tmp_path / "plan_check"
    csrc = os.path.join(ROOT, "paper_1805_07891_amd", "csrc")
    subprocess.check_call(["g++", "-std=c++17", *SAN, f"-I{csrc}", "-o", str(exe),
                           os.path.join(csrc, "plan.cpp"),
                           os.path.join(ROOT, "tests", "sanitize", "plan_check.cpp")])
    out = _run(str(exe), str(lists))
    assert "plan checks passed over 11 key lists" in out
