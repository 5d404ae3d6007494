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


def test_cpu_baseline_reports_stages_and_host():
    """The CPU leg on the tiny workload: one pass of the oracle's stages, each
    timed, with the host's core count and CPU model."""
    from paper_2608_28511_amd.workloads import TINY, make_inputs
    rec = bench.cpu_baseline(TINY, make_inputs(TINY), 0, min_seconds=0.0, max_runs=1)
    assert rec["kind"] == "oracle" and rec["unit"] == "slots/s" and rec["value"] > 0
    assert rec["nproc"] >= 1 and isinstance(rec["cpu_model"], str)
    assert set(rec["stage_seconds_per_pass"]) == {"router_logits", "route", "permutation", "dispatch",
                                                  "expert_ffn", "combine"}
