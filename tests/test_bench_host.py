"""Host-side logic of bench.py (no GPU): the per-step statistics and the
one-GPU guard."""
import subprocess
import sys
from pathlib import Path

import bench

ROOT = Path(__file__).resolve().parents[1]


def test_filtered_mean_drops_outliers_iteratively():
    # 10 is above mean + 1.5 sd of [1, 1, 1, 1, 10] (mean 2.8, sd 3.6); then nothing more
    assert bench.filtered_mean([1, 1, 1, 1, 10]) == 1.0
    # two rounds: 1000 goes first, then 100 against [1, 2, 3, 4, 100]
    assert bench.filtered_mean([1, 2, 3, 4, 100, 1000]) == 2.5
    # nothing above the bar: the plain mean
    assert bench.filtered_mean([5, 6, 7]) == 6.0


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, str(ROOT / "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
