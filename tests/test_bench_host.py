"""Host-side checks of bench.py that need no GPU: the one-GPU refusal, argument checks, the
lookup of committed profile counters, and the CPU oracle baseline on a tiny budget."""

import glob
import json
import os
import subprocess
import sys

import bench
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_per_tensor_layout_needs_an_opt_workload():
    r = _run("--workload", "tiny", "--layout", "tensors", "--no-cpu-baseline")
    assert r.returncode == 2
    assert "model-shaped" in r.stderr


def test_committed_counters_match_the_sweep_source():
    """Every profile summary carries a counters-json line for the current sweep source, and the
    bench finds it by workload, K, dtype and layout (so `traffic` is not null)."""
    digest = bench.sweep_source_digest()
    found = []
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        lines = [ln for ln in open(path) if ln.startswith("counters-json:")]
        assert len(lines) == 1, path
        d = json.loads(lines[0].split(":", 1)[1])
        assert d["source_sha256"] == digest, f"{path} was taken with other sweep sources"
        got = bench.measured_counters(d["workload"], d["K"], d["dtype"], d.get("layout", "flat"))
        assert got == d
        sweep = 2 * 2 * workloads.WORKLOADS[d["workload"]].n
        for kernel, traffic in d["traffic_bytes_per_launch"].items():
            assert abs(traffic / sweep - 1) < 1e-3, (path, kernel)
        found.append((d["workload"], d["K"], d.get("layout", "flat")))
    assert ("opt13b", 16, "flat") in found  # the benchmark's default workload


def test_binding_unit_is_the_busiest_measured_unit():
    assert bench.binding_unit(0.81) == "hbm"
    assert bench.binding_unit(0.81, 0.19, 0.50) == "hbm"  # the K = 16 update
    assert bench.binding_unit(0.68, 0.71, 0.87) == "alu"  # the K = 32 update at a lowered clock
    assert bench.binding_unit(0.35, 0.96, 0.75) == "lds"  # a shared-table update at K = 64
    assert bench.binding_unit(0.42, 0.74, 0.86) == "alu"  # the K = 64 update on 16-copy tables
    assert bench.binding_unit(0.84, None, 0.39) == "hbm"  # the perturb (no LDS)


def test_committed_counters_name_the_expected_bounds():
    """With the committed counters, the K = 16 update is memory-bound and K = 32 and K = 64
    VALU-bound (the 16-copy tables took K = 64 off the LDS bound; the HBM fractions are those
    the profiles' traces give)."""
    for wl, K, hbm, want in [("opt13b", 16, 0.81, "hbm"), ("opt30b", 32, 0.68, "alu"), ("opt1.3b", 64, 0.42, "alu")]:
        c = bench.measured_counters(wl, K, "bf16")
        assert bench.binding_unit(hbm, c["lds_per_launch"]["zo_update"]["lds_busy"], c["valu_busy"]["zo_update"]) == want


def test_counters_absent_for_an_unprofiled_configuration():
    assert bench.measured_counters("opt13b", 7, "bf16") == {}
    assert bench.measured_counters("opt1.3b", 64, "bf16", "tensors") == {}


def test_cpu_baseline_reports_the_oracle_on_a_bounded_sample():
    w = workloads.WORKLOADS["tiny"]
    one = bench.cpu_baseline(w, 4, budget_s=0.5)
    assert one["kind"] == "oracle" and one["cores"] == 1 and one["value"] > 0
    assert "tiny" in one["sample"]
    many = bench.cpu_baseline(w, 4, budget_s=0.5, procs=2)
    assert many["cores"] == 2 and many["value"] > 0
