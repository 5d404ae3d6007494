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


def test_gemm_roofline_takes_the_bound_of_its_intensity():
    """The grouped GEMM's roofline: below the ridge (2500 TFLOP/s over 8 TB/s =
    312.5 flop per byte) HBM bounds it, above it the MFMA pipes; the 256-expert
    layer's projection (2.8 GB of weights for 65,536 rows) falls below, the
    64-expert one above."""
    from paper_2608_28511_amd.workloads import WORKLOADS
    ce, base = WORKLOADS["ce_s8192_d2048_e256_k8"], WORKLOADS["base_s8192_d2048_e64_k6"]
    fl = 2.0 * ce.R * ce.D * ce.F
    nb = bench.gemm_bytes(ce, ce.E)
    assert nb == ce.R * (ce.D + ce.F) * 2 + ce.E * ce.D * ce.F * 2
    r = bench.gemm_roofline("grouped_up", fl, nb, 1e-3)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert abs(r["achieved"] - nb / 1e-3 / 1e9) < 0.1 and abs(r["frac"] - r["hbm_frac"]) < 1e-9
    assert r["intensity_flop_per_byte"] < 312.5 == r["ridge_flop_per_byte"]
    assert abs(r["mfma_frac"] - fl / 1e-3 / 2.5e15) < 1e-4
    fl_b = 2.0 * base.R * base.D * base.F
    r = bench.gemm_roofline("grouped_up", fl_b, bench.gemm_bytes(base, base.E), 2e-4)
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s" and abs(r["frac"] - r["mfma_frac"]) < 1e-9
