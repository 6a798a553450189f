"""Host-side logic of bench.py that needs no GPU: one GPU only, and the
traffic figure reported only for the kernel source it was measured on."""

import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_traffic_only_for_the_measured_source():
    sys.path.insert(0, ROOT)
    import bench

    names = [n for n in os.listdir(os.path.join(ROOT, "profiles")) if n.endswith("_traffic.json")]
    assert names
    for name in names:
        with open(os.path.join(ROOT, "profiles", name)) as fh:
            rec = json.load(fh)
        wl, variant = rec["workload"], rec.get("variant", "")
        got = bench.measured_profile(rec["kernel"], wl, variant)
        if rec["kernel_source_sha256_16"] == bench.kernel_source_hash():
            assert got == rec
            if not variant:
                # within 0.1% of the algorithmic bytes: no re-reads
                assert abs(rec["hbm_bytes_per_launch"] / rec["algorithmic_bytes_per_launch"]
                           - 1.0) < 1e-3
        else:
            assert got is None
    assert bench.measured_profile(bench.DOMINANT, "tiny", "no-such-variant") is None


def test_cpu_baseline_sample_is_whole_steps():
    """Workloads above the sample size are cut to their first whole steps; the
    cut keeps every per-token input of those rows and the step offsets."""
    sys.path.insert(0, ROOT)
    import numpy as np

    import bench
    import synth

    wl = synth.make_workload("microbatch")
    sub, n = bench._steps_prefix(wl, bench.CPU_SAMPLE_MAX_ROWS)
    assert 0 < sub.T <= bench.CPU_SAMPLE_MAX_ROWS and sub.S == n
    assert sub.T == int(wl.off[n]) and int(wl.off[n + 1]) > bench.CPU_SAMPLE_MAX_ROWS
    assert np.array_equal(sub.off, wl.off[:n + 1])
    for k in ("target", "adv", "old_offset", "roll_offset", "kind", "src_row", "spike_col",
              "spike_val"):
        assert np.array_equal(getattr(sub, k), getattr(wl, k)[:sub.T])
    # a first step longer than the sample is still taken whole
    one, n1 = bench._steps_prefix(wl, 1)
    assert n1 == 1 and one.T == int(wl.off[1])


def test_cpu_baseline_runs_on_the_small_workload():
    sys.path.insert(0, ROOT)
    import bench
    import synth

    r = bench.cpu_baseline(synth.make_workload("tiny"), threads=2, min_seconds=0.05, max_passes=3)
    assert r["kind"] == "oracle" and r["cores"] == 2 and r["value"] > 0
    assert 1 <= r["passes"] <= 3 and r["sample"].startswith("whole workload")
