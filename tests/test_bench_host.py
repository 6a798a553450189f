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

    for wl in ("vlm7b", "longhorizon"):
        path = os.path.join(ROOT, "profiles", f"tis_grad_kernel_{wl}_traffic.json")
        rec = json.load(open(path))
        got = bench.measured_traffic(wl)
        if rec["kernel_source_sha256_16"] == bench.kernel_source_hash():
            assert got == rec["hbm_bytes_per_launch"]
            # within 0.1% of the algorithmic bytes: no re-reads
            assert abs(got / rec["algorithmic_bytes_per_launch"] - 1.0) < 1e-3
        else:
            assert got is None
    assert bench.measured_traffic("tiny") is None
