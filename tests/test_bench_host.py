"""Host logic of bench.py that runs without a GPU: what the five-workload
parent passes to each workload's process, the one-GPU rule, the kernel
source hash that ties profiles/ to the code, and the compact per-workload
block of the JSON line."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_child_args_drop_the_parents_own_flags():
    argv = ["--steps", "20", "--warmup=5", "--workload", "tiny", "--cpu-seconds", "3",
            "--config-cpu-seconds=1", "--min-timed-ms", "10", "--schedule", "dynamic",
            "--whole-chunks"]
    assert bench.child_args(argv) == ["--steps", "20", "--warmup=5", "--schedule", "dynamic",
                                      "--whole-chunks"]
    assert bench.child_args([]) == []
    # every flag the parent keeps for itself takes one value
    assert all(n == 1 for n in bench._OWN_FLAGS.values())


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_source_hash_follows_code_not_comments():
    code = 'int f(int x) {\n  return x + 1;  // one more\n}\n/* a block\n comment */\n'
    same = 'int f(int x) {  /* note */\n    return x + 1;\n}\n// trailing\n'
    other = 'int f(int x) {\n  return x + 2;\n}\n'
    assert bench._code_only(code) == bench._code_only(same)
    assert bench._code_only(code) != bench._code_only(other)
    # string literals are code, including ones that look like comments
    assert "// not a comment" in bench._code_only('const char* s = "// not a comment";')
    assert len(bench.kernel_source_hash()) == 16


def _line(cold, traffic, note=None):
    c = {"hbm_pct_of_peak_whole_step": 78.0, "jobs": [{"state_cached_fraction": 0.0}],
         "host_us_per_step": 5.0}
    if note:
        c["note"] = note
    return {
        "ms_per_step": 1.5, "value": 4000.0,
        "roofline": {"frac": 0.78, "cold": cold, "traffic": traffic,
                     "algorithmic_bytes_per_launch": 1000,
                     "frac_of_mixed_ceiling": 1.1,
                     "ceilings": {"read": {"frac_of_peak": 0.92}, "mixed": {"frac_of_peak": 0.71},
                                  "phase_separated": {"frac_of_peak": 0.88}}},
        "config": c,
        "cpu_baseline": {"value": 5.0, "sample": "s"},
    }


@pytest.mark.parametrize("cold,traffic,note", [
    ({"frac": 0.77, "isolated_warm_frac": 0.775}, 1001, None),
    (None, None, "cache-resident"),
])
def test_compact_block(cold, traffic, note):
    out = bench.compact(_line(cold, traffic, note))
    assert out["kernel_frac"] == 0.78 and out["whole_step_pct"] == 78.0
    assert out["kernel_frac_cold"] == (cold["frac"] if cold else None)
    assert out["traffic_over_algorithmic"] == (1.001 if traffic else None)
    assert out["state_cached_fraction"] == [0.0]
    assert out.get("note") == note
