"""CPU checks of the benchmark's bookkeeping: the algorithmic FLOP count that
the roofline fraction divides by, the guard that drops stale traffic counters,
and the one-GPU limit of the command line."""
import json
import os
import subprocess
import sys

import pytest

import bench
from paper_1506_09067_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# Multiply-adds per sample written out layer by layer from the shapes of
# Table I (valid stride-1 convolutions, non-overlapping pools):
#   forward          conv: maps x out positions x in maps x k^2; FC: out x in
#   backward data    the same count for every layer above the input
#   weight gradient  the forward count plus one bias add per output value
#   update           one multiply-add per parameter
# The training count is 2 x (forward + backward data + weight gradient +
# update); the forward count is 2 x forward.
HAND = {
    # conv5 k4 26x26 | max2 | conv10 k5 9x9 | max3 | FC50 (90 in) | FC10
    "small": dict(
        fwd=[5 * 676 * 16, 10 * 81 * 5 * 25, 50 * 90, 10 * 50],
        out=[5 * 676, 10 * 81, 50, 10],
        params=6405),
    # conv20 k4 26x26 | max2 | conv40 k5 9x9 | max3 | FC150 (360 in) | FC10
    "medium": dict(
        fwd=[20 * 676 * 16, 40 * 81 * 20 * 25, 150 * 360, 10 * 150],
        out=[20 * 676, 40 * 81, 150, 10],
        params=76040),
    # conv20 k4 26x26 | max2 | conv60 k3 11x11 | conv100 k6 6x6 | max2 | FC150 (900 in) | FC10
    "large": dict(
        fwd=[20 * 676 * 16, 60 * 121 * 20 * 9, 100 * 36 * 60 * 36, 150 * 900, 10 * 150],
        out=[20 * 676, 60 * 121, 100 * 36, 150, 10],
        params=363960),
    # conv20 k4 26x26 | max1 | conv60 k5 22x22 | max2 | conv100 k6 6x6 | max2 | FC150 | FC10
    "large_table1": dict(
        fwd=[20 * 676 * 16, 60 * 484 * 20 * 25, 100 * 36 * 60 * 36, 150 * 900, 10 * 150],
        out=[20 * 676, 60 * 484, 100 * 36, 150, 10],
        params=383160),
}

# the per-sample totals as printed in the design tables (MFLOP, rounded)
PRINTED = {"small": (0.875, 0.321), "medium": (11.10, 3.784), "large": (56.96, 18.87),
           "large_table1": (136.3, 45.30)}


@pytest.mark.parametrize("name", sorted(HAND))
def test_train_flops_per_sample(name):
    h = HAND[name]
    fwd = sum(h["fwd"])
    bwd = fwd - h["fwd"][0]  # no backward-data pass into the input
    wgrad = fwd + sum(h["out"])
    train, forward = bench.train_flops_per_sample(wl.NETS[name])
    assert forward == 2 * fwd
    assert train == 2 * (fwd + bwd + wgrad + h["params"])
    t, f = PRINTED[name]
    assert train / 1e6 == pytest.approx(t, rel=6e-3)
    assert forward / 1e6 == pytest.approx(f, rel=6e-3)


def test_large_net_flops_exact():
    # the figure the headline roofline fraction divides by
    assert bench.train_flops_per_sample(wl.NETS["large"]) == (56_958_080, 18_871_240)


def _traffic(tmp_path, **over):
    t = {"net": "large", "workers": 256, "samples_per_launch": 60000,
         "bytes_per_launch": 1.5e11, "source_sha256": bench.kernel_source_hash()}
    t.update(over)
    p = tmp_path / "traffic.json"
    p.write_text(json.dumps(t))
    return str(p)


def test_traffic_only_for_the_profiled_kernel_and_configuration(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILE_TRAFFIC", _traffic(tmp_path))
    assert bench.measured_traffic("large", 256, 60000) == 1.5e11
    assert bench.measured_traffic("large", 512, 60000) is None
    assert bench.measured_traffic("large", 256, 30000) is None
    assert bench.measured_traffic("medium", 256, 60000) is None
    monkeypatch.setattr(bench, "PROFILE_TRAFFIC", _traffic(tmp_path, source_sha256="0" * 64))
    assert bench.measured_traffic("large", 256, 60000) is None
    monkeypatch.setattr(bench, "PROFILE_TRAFFIC", str(tmp_path / "absent.json"))
    assert bench.measured_traffic("large", 256, 60000) is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in (r.stdout + r.stderr)
    assert not r.stdout.strip().startswith("{")
