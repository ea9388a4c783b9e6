"""CPU: the benchmark's command line and its threshold calibration (no GPU)."""
import json
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120, cwd=ROOT)
    assert out.returncode == 2
    msg = json.loads(out.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_calibrated_threshold_hits_the_target_fraction():
    rng = np.random.default_rng(3)
    T, N, s_max = 8, 35, 8
    u = 10.0 ** rng.uniform(-4, -2, size=(T, N))
    embed = np.zeros(N, bool)
    embed[0] = True
    for target in (0.15, 0.2, 0.3):
        k0 = bench.calibrate_k0(u, embed, s_max, target)
        # replay the rule over the same horizon the calibration uses
        K = k0 * np.where(embed, 10.0, 1.0)
        delta, last, tot, horizon = np.zeros(N), np.zeros(N, np.int64), 0, max(8 * s_max, 4 * T)
        for t in range(1, horizon + 1):
            delta += u[(t - 1) % T]
            sel = (delta >= K) | (t - last >= s_max)
            delta[sel] = 0.0
            last[sel] = t
            tot += int(sel.sum())
        assert abs(tot / (horizon * N) - target) < 0.05, (target, tot / (horizon * N))
    # a larger target never needs a larger threshold
    assert bench.calibrate_k0(u, embed, s_max, 0.3) <= bench.calibrate_k0(u, embed, s_max, 0.15)
