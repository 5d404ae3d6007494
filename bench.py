"""Benchmark of one routed MoE layer forward on one MI355X.

Prints ONE JSON line on stdout (progress goes to stderr):
  value        routed token-slots per second of moe_layer_fwd (S*K / layer time)
               on the 256-expert CE-MoE-style layer (8192 tokens, D 2048, top-8,
               F 2688: the largest forward of the five workloads by flops and
               weight bytes), inputs resident in HBM, input sets rotated between
               steps so the 256 MB last-level cache cannot hold a step's weights
  other_workloads  the same layer measurement (value, ms per step, the
               dominant GEMM's fraction of the MFMA peak) on the other full-size
               workloads
  roofline     the dominant kernel (the larger of the two grouped GEMMs), each
               launch timed with its own HIP events on the stream it is launched
               on, inside the layer's own launch sequence, against the roofline
               that bounds it: HBM (8 TB/s) when its flops per algorithmic byte
               fall below the ridge (312.5), else the dense bf16 MFMA peak; both
               fractions are reported
  stages       per-stage times and algorithmic GB/s or TFLOP/s; each launch of
               a stage is timed alone with its own events, after an untimed
               512 MB write that evicts its inputs from the last-level cache
  cpu_baseline the CPU oracle on the same workload, with its per-stage times

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time
from pathlib import Path

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

METRIC = ("routed token-slots/sec per MoE layer fwd; HBM GB/s (route/dispatch/combine), "
          "MFMA % peak")
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, GB/s
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, TFLOP/s
PEAK_FP32_TFLOPS = 157.3       # MI355X fp32 vector, TFLOP/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--settle-seconds", type=float, default=0.3,
                   help="run the layer this long before the warm-up steps, so the GPU is at its "
                        "sustained clock when the timed steps start")
    p.add_argument("--workload", default="ce_s8192_d2048_e256_k8")
    p.add_argument("--others", default="base_s8192_d2048_e64_k6,latent_s16384_h4096_d1024_e128_k6,"
                                       "skew_s16384_d2048_e128_k8_bwd",
                   help="comma-separated workloads measured after the headline one (layer rate and the "
                        "dominant GEMM only); empty for none")
    p.add_argument("--other-steps", type=int, default=20)
    p.add_argument("--sets", type=int, default=3, help="rotating input sets")
    p.add_argument("--payload", default="bf16", choices=("bf16", "mxfp8"),
                   help="dispatch payload of the timed layer (MX-FP8: b_x = 1 + 1/32)")
    p.add_argument("--stage-reps", type=int, default=20)
    p.add_argument("--cpu-tokens", type=int, default=0,
                   help="tokens of the batch the CPU oracle runs (0: the whole batch)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--ep-share", type=int, default=0, metavar="G",
                   help="also time the expert-local grouped GEMMs one GPU would run under expert "
                        "parallelism over G GPUs (E/G experts, the same S*K rows); reported apart")
    p.add_argument("--route-sweep", action="store_true",
                   help="also time the route alone over token counts 1K..128K (the workload's E and K) "
                        "and report its algorithmic GB/s; reported apart")
    p.add_argument("--flush-bytes", type=int, default=512 << 20,
                   help="bytes written between stage launches so no stage reads its inputs from the "
                        "256 MB last-level cache")
    p.add_argument("--calib-bytes", type=int, default=1 << 30,
                   help="size of the plain copy run once for counter calibration")
    p.add_argument("--traffic-from", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                   help="summarise two rocprofv3 counter passes into profiles/ and exit")
    p.add_argument("--traffic-kernel", default="grouped_down", choices=sorted(KERNEL_NAME))
    p.add_argument("--traffic-bench-args", default="--others= --no-cpu-baseline --steps 10 --warmup 2 --stage-reps 5",
                   help="the bench arguments the two counter passes ran with (recorded in the summary)")
    return p.parse_args()


# ---- HBM traffic of the dominant kernel, from hardware counters ----------------
# Two profiler passes of this same command, one per counter:
#   rocprofv3 --pmc FETCH_SIZE --output-format csv -d <dir_fetch> -o p -- python bench.py --no-cpu-baseline
#   rocprofv3 --pmc WRITE_SIZE --output-format csv -d <dir_write> -o p -- python bench.py --no-cpu-baseline
# then `python bench.py --traffic-from <dir_fetch> <dir_write>` writes the summary
# profiles/traffic_<kernel>_<workload>.txt.  Each counter (KiB per dispatch) is
# scaled by what it reads for the plain 1 GiB device copy this script runs at
# start-up (a copy reads and writes exactly 1 GiB).  The summary records a
# digest of the GEMM sources; once they change, `traffic` is reported as null.
GEMM_SOURCES = ("gemm.hip", "tile_dma.h", "kernels.h", "common.h")
# The grouped GEMM's symbol carries its operand layout, epilogue and k-tail
# flag (up: squared-ReLU epilogue; down: plain bf16); the tile height is
# chosen inside the kernel.
KERNEL_NAME = {"grouped_up": ("gemm_rows_kernel<false, 1, false>",),
               "grouped_down": ("gemm_rows_kernel<false, 0, false>",),
               "grouped_up_mxfp8": ("gemm_rows_mx_kernel<1, false>",)}


def kernel_match(kernel, name):
    return all(part in name for part in KERNEL_NAME[kernel])


def gemm_digest():
    import hashlib
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        h.update((ROOT / "paper_2608_28511_amd" / "csrc" / f).read_bytes())
    return h.hexdigest()


def traffic_path(kernel, workload):
    return ROOT / "profiles" / f"traffic_{kernel}_{workload}.txt"


def load_traffic(kernel, workload):
    p = traffic_path(kernel, workload)
    if not p.exists():
        return None
    rec = json.loads(p.read_text().split("\n", 1)[1])
    if rec.get("gemm_sources_sha256") != gemm_digest():
        log(f"{p.name}: GEMM sources changed since the counters were taken; traffic null")
        return None
    return rec["bytes_per_launch"]


def counter_rows(d):
    """Rows of the newest counter_collection.csv under d (one profiler run)."""
    import csv
    files = sorted(Path(d).rglob("*counter_collection.csv"), key=lambda f: f.stat().st_mtime)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    if len(files) > 1:
        log(f"{d}: {len(files)} counter files, using the newest ({files[-1].name})")
    return list(csv.DictReader(open(files[-1])))


def per_dispatch(rows, counter, match):
    vals = {}
    for r in rows:
        if r["Counter_Name"] == counter and match(r["Kernel_Name"]):
            vals[r["Dispatch_Id"]] = vals.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    return list(vals.values())


def write_traffic(d_fetch, d_write, workload, kernel, calib_bytes, bench_args):
    out = {"kernel": kernel, "kernel_symbol": "...".join(KERNEL_NAME[kernel]), "workload": workload,
           "gemm_sources_sha256": gemm_digest()}
    total = 0.0
    for d, counter in ((d_fetch, "FETCH_SIZE"), (d_write, "WRITE_SIZE")):
        rows = counter_rows(d)
        cal = per_dispatch(rows, counter, lambda n: "copyBuffer" in n)
        if not cal:
            raise SystemExit(f"{d}: no device copy dispatch to calibrate {counter}")
        factor = calib_bytes / (max(cal) * 1024.0)
        ks = per_dispatch(rows, counter, lambda n: kernel_match(kernel, n))
        if not ks:
            raise SystemExit(f"{d}: no {kernel} dispatches")
        kib = sum(ks) / len(ks)
        out[counter] = {"kib_per_dispatch": round(kib, 1), "dispatches": len(ks),
                        "copy_kib": round(max(cal), 1), "factor": round(factor, 4),
                        "bytes": round(kib * 1024.0 * factor)}
        total += kib * 1024.0 * factor
    out["bytes_per_launch"] = round(total)
    p = traffic_path(kernel, workload)
    cmd = f"python3 -u bench.py --workload {workload} {bench_args}"
    out["commands"] = [f"rocprofv3 --pmc FETCH_SIZE --output-format csv -d {d_fetch} -o f -- {cmd}",
                       f"rocprofv3 --pmc WRITE_SIZE --output-format csv -d {d_write} -o wr -- {cmd}",
                       f"python bench.py --traffic-from {d_fetch} {d_write} --workload {workload} "
                       f"--traffic-kernel {kernel}"]
    p.write_text(f"HBM traffic of {kernel} on {workload} from rocprofv3 FETCH_SIZE / WRITE_SIZE "
                 f"passes (commands below), each scaled by what it reads for a 1 GiB device copy\n"
                 + json.dumps(out, indent=1) + "\n")
    print(p.read_text())


def gemm_bytes(s, e_used):
    """Algorithmic bytes of one grouped-GEMM launch (either projection): the
    A rows read, the output rows written and the weights of the experts that
    received rows, R*Kd*2 + R*N*2 + E_used*Kd*N*2 with {Kd, N} = {D, F}."""
    return s.R * s.D * 2 + s.R * s.F * 2 + e_used * s.D * s.F * 2


def gemm_roofline(kernel, flops, nbytes, t, traffic=None, per_launch=""):
    """The dominant grouped GEMM against the roofline that bounds it: an
    algorithmic intensity (flops per algorithmic byte) below the ridge (peak
    MFMA rate over peak HBM bandwidth, 312.5 flop/B) bounds it by HBM, above
    it by the MFMA pipes.  Both fractions are reported."""
    ridge = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    ai = flops / nbytes
    tf, gbs = flops / t / 1e12, nbytes / t / 1e9
    if ai < ridge:
        r = {"bound": "hbm", "kernel": kernel, "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
             "frac": round(gbs / PEAK_HBM_GBS, 4)}
    else:
        r = {"bound": "mfma", "kernel": kernel, "achieved": round(tf, 1), "peak": PEAK_BF16_TFLOPS,
             "unit": "TFLOP/s", "frac": round(tf / PEAK_BF16_TFLOPS, 4)}
    r.update(traffic=traffic, intensity_flop_per_byte=round(ai, 1), ridge_flop_per_byte=round(ridge, 1),
             mfma_frac=round(tf / PEAK_BF16_TFLOPS, 4), hbm_frac=round(gbs / PEAK_HBM_GBS, 4),
             algorithmic_bytes=int(nbytes), flops=flops, per_launch=per_launch)
    return r


def stage_bytes(s):
    S, D, E, K, F, R = s.S, s.D, s.E, s.K, s.F, s.R
    return {
        # x read, Wr read and split into three bf16 planes, planes re-read per
        # 64-token tile from L2 (not counted), logits written
        "router_logits": S * D * 2 + D * E * 4 + 3 * D * E * 2 + S * E * 4,
        "route": S * E * 4 + R * 16 + (2 * E + 1) * 4,
        "dispatch": S * D * 2 + R * 8 + R * (2 * D + 4),
        # with a shared expert its fp32 output is read as the addend
        "combine": R * (2 * D + 8) + S * D * 2 + (S * D * 4 if s.Fs else 0),
        # dy read once per slot, y_disp and p read, dy_disp written, dp written
        "combine_bwd": S * D * 2 + R * (2 * D + 8) + R * 2 * D + R * 4,
        # plus the router's fp32 input gradient read as the addend
        "dispatch_bwd": R * (2 * D + 4) + S * D * 2 + S * D * 4,
        # logits read once per 64-token chunk, topk_idx read, partials written
        "seq_aux_loss": S * E * 4 + R * 4,
        # MX-FP8 payload: x read once, codes + scales + p written per routed row
        "dispatch_mxfp8": S * D * 2 + R * 8 + R * (D + D // 32 + 4),
        "mxfp8_dequant": R * (D + D // 32) + R * D * 2,
    }


def time_region(fn, reps, stream):
    """Average duration of fn() over reps back-to-back launches, bracketed by
    HIP events recorded on `stream` (the stream the kernels run on)."""
    import torch
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(reps):
        fn(i)
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / reps * 1e-3   # seconds


def time_flushed(fn, reps, stream, flush):
    """Average duration (s) of fn(i) over reps launches, each bracketed by its
    own HIP events on `stream`, with flush() (an untimed write of more bytes
    than the last-level cache holds) enqueued before each, so every launch
    reads its inputs from HBM."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    torch.cuda.synchronize()
    for i in range(reps):
        flush()
        ev[i][0].record(stream)
        fn(i)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in ev) / reps * 1e-3


def step_times(fn, reps, stream):
    """Durations (us) of reps back-to-back calls fn(i), one HIP event pair
    per call on `stream`."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    torch.cuda.synchronize()
    for i in range(reps):
        ev[i][0].record(stream)
        fn(i)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) * 1e3 for a, b in ev]


def filtered_mean(xs):
    """Mean after iteratively dropping samples above mean + 1.5 standard
    deviations, until none is dropped."""
    xs = list(xs)
    while len(xs) > 2:
        m = sum(xs) / len(xs)
        sd = (sum((x - m) ** 2 for x in xs) / len(xs)) ** 0.5
        kept = [x for x in xs if x <= m + 1.5 * sd]
        if len(kept) == len(xs):
            break
        xs = kept
    return sum(xs) / len(xs)


def route_sweep(_lib, s, reps, stream, dev):
    """The route (top-K, histogram and scan, permutation) alone over token
    counts S = 1K .. 128K with the workload's E and K: duration and
    algorithmic bytes (read S*E*4, write R*16 + (2E+1)*4) per S, to show where
    its two launches stop being latency-bound."""
    import torch
    out = []
    for S in (1 << k for k in range(10, 18)):
        R = S * s.K
        g = torch.Generator(device=dev).manual_seed(S)
        logits = torch.randn((S, s.E), generator=g, device=dev)
        bufs = [torch.empty((S, s.K), dtype=torch.int32, device=dev), torch.empty((S, s.K), device=dev),
                torch.empty((s.E,), dtype=torch.int32, device=dev),
                torch.empty((s.E + 1,), dtype=torch.int32, device=dev),
                torch.empty((R,), dtype=torch.int32, device=dev), torch.empty((R,), dtype=torch.int32, device=dev)]
        ws = torch.empty(max(1, _lib.moe_route_workspace_bytes(S, s.E, s.K)), dtype=torch.uint8, device=dev)
        fn = lambda i: _lib.moe_route_topk(logits, S, s.E, s.K, *bufs, ws)
        for i in range(3):
            fn(i)
        t = time_region(fn, reps, stream)
        nbytes = S * s.E * 4 + R * 16 + (2 * s.E + 1) * 4
        out.append({"S": S, "us": round(t * 1e6, 2), "bytes": nbytes, "GBps": round(nbytes / t / 1e9, 1)})
    return out


def ep_share(_lib, s, G, reps, stream, dev):
    """Up and down grouped GEMM of one GPU's share under expert parallelism
    over G GPUs: its E/G experts receive, on balanced routing, all S*K rows
    (each of the G GPUs sends it S*K/G).  Seeded balanced segments, fresh
    weights of the workload's widths."""
    import torch
    from paper_2608_28511_amd.workloads import make_segments
    if s.E % G:
        return {"G": G, "skipped": f"E = {s.E} is not a multiple of G"}
    E_loc, R = s.E // G, s.S * s.K
    g = torch.Generator(device=dev).manual_seed(s.seed)
    off = make_segments(R, E_loc, seed=s.seed).to(dev)
    x = torch.randn((R, s.D), generator=g, device=dev).to(torch.bfloat16)
    W1 = [(torch.randn((E_loc, s.D, s.F), generator=g, device=dev) / math.sqrt(s.D)).to(torch.bfloat16)
          for _ in range(2)]
    W2 = [(torch.randn((E_loc, s.F, s.D), generator=g, device=dev) / math.sqrt(s.F)).to(torch.bfloat16)
          for _ in range(2)]
    h = torch.empty((R, s.F), dtype=torch.bfloat16, device=dev)
    y = torch.empty((R, s.D), dtype=torch.bfloat16, device=dev)
    sched = torch.empty(_lib.moe_grouped_schedule_bytes(E_loc, R) // 4 + 1, dtype=torch.int32, device=dev)
    _lib.moe_grouped_schedule(off, E_loc, R, sched)
    up = lambda i: _lib.moe_grouped_gemm(x, sched, E_loc, R, s.D, s.F, W1[i % 2], 1, h, None)
    down = lambda i: _lib.moe_grouped_gemm(h, sched, E_loc, R, s.F, s.D, W2[i % 2], 0, y, None)
    for i in range(3):
        up(i); down(i)
    t_up, t_down = time_region(up, reps, stream), time_region(down, reps, stream)
    fl = 2.0 * R * s.D * s.F
    return {"G": G, "E_local": E_loc, "rows": R, "rows_per_expert": R // E_loc,
            "up_us": round(t_up * 1e6, 1), "down_us": round(t_down * 1e6, 1),
            "up_TFLOPs": round(fl / t_up / 1e12, 1), "down_TFLOPs": round(fl / t_down / 1e12, 1)}


def time_layer_gemms(_lib, sets, out, s, reps, stream, ws_router, ws_route, r_bufs, xd, pd, h, yd, mx=None):
    """Average durations (s) of the up and down grouped GEMM launches inside
    the layer's launch sequence, one HIP event pair per launch on `stream`:
    router, route, tile schedule, up projection gathering its rows from x
    (the dispatch fused into its operand copy, as the layer runs it), down
    projection, combine.  mx = (codes, scales): the MX-FP8 payload instead,
    dispatched and read as sent by the up GEMM."""
    import torch
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(reps)]
    lg = torch.empty_like(out["logits"])
    y = torch.empty_like(out["y"])
    sched = torch.empty(_lib.moe_grouped_schedule_bytes(s.E, s.R) // 4 + 1, dtype=torch.int32, device=lg.device)
    torch.cuda.synchronize()
    for i in range(reps):
        inp = sets[i % len(sets)]
        _lib.moe_router_logits(inp["x"], inp["Wr"], inp["bias"], s.S, s.D, s.E, lg, ws_router)
        _lib.moe_route_topk(lg, s.S, s.E, s.K, r_bufs["topk_idx"], r_bufs["topk_prob"], r_bufs["counts"],
                            r_bufs["offsets"], r_bufs["perm"], r_bufs["inv_perm"], ws_route)
        if mx is not None:
            _lib.moe_dispatch_mxfp8(inp["x"], r_bufs["topk_prob"], r_bufs["inv_perm"], s.S, s.D, s.K, *mx, pd)
        _lib.moe_grouped_schedule(r_bufs["offsets"], s.E, s.R, sched)
        ev[i][0].record(stream)
        if mx is None:
            _lib.moe_grouped_gemm_gather(inp["x"], r_bufs["perm"], s.S, s.K, sched, s.E, s.R, s.D, s.F, inp["W1"], 1,
                                         h, None)
        else:
            _lib.moe_grouped_gemm_mxfp8(*mx, sched, s.E, s.R, s.D, s.F, inp["W1"], 1, h, None)
        ev[i][1].record(stream)
        ev[i][2].record(stream)
        _lib.moe_grouped_gemm(h, sched, s.E, s.R, s.F, s.D, inp["W2"], 0, yd, None)
        ev[i][3].record(stream)
        _lib.moe_combine(yd, pd if mx is not None else None, r_bufs["inv_perm"], s.S, s.D, s.K, y)
    torch.cuda.synchronize()
    up = sum(e[0].elapsed_time(e[1]) for e in ev) / reps * 1e-3
    down = sum(e[2].elapsed_time(e[3]) for e in ev) / reps * 1e-3
    return up, down


def host_info():
    """nproc and the CPU model of the host this runs on."""
    model = "unknown"
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "cpu_model": model}


def cpu_baseline(s, inp, tokens, payload="bf16", min_seconds=10.0, max_runs=8):
    """The float64 oracle on the first `tokens` tokens (0: all) of the same
    workload, repeated until about min_seconds of CPU work.  For the softmax
    layers the oracle's stage functions are called one by one, in the order
    its layer forward calls them, and each is timed."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info

    from oracle import moe_oracle as O

    T = s.S if tokens <= 0 else min(tokens, s.S)
    x = inp["x"][:T].cpu().to(torch.float64).numpy()
    Wr = inp["Wr"].cpu().to(torch.float64).numpy()
    bias = None if inp["bias"] is None else inp["bias"].cpu().to(torch.float64).numpy()
    W1c, W2c = inp["W1"].cpu(), inp["W2"].cpu()

    class Experts:
        def __init__(self, W):
            self.W = W

        def __getitem__(self, e):
            return self.W[int(e)].to(torch.float64).numpy()

    f64 = lambda t: t.cpu().to(torch.float64).numpy()
    extra = {}
    if s.H:
        extra = dict(Wdown=f64(inp["Wdown"]), Wup=f64(inp["Wup"]))
    staged = s.score == "softmax" and not s.Fs and payload == "bf16"
    if s.score == "sigmoid":
        extra.update(score="sigmoid", sel_bias=f64(inp["sel_bias"]))
        if s.seq_len and T % s.seq_len == 0:   # the balance loss needs whole sequences
            extra.update(seq_len=s.seq_len, aux_coeff=s.aux_coeff)
    if s.Fs:
        extra.update(Ws1=f64(inp["Ws1"]), Ws2=f64(inp["Ws2"]))
    if payload != "bf16":
        extra["payload"] = payload
    stage_s = {}

    def timed(name, fn, *a, **kw):
        t0 = time.perf_counter()
        r = fn(*a, **kw)
        stage_s[name] = stage_s.get(name, 0.0) + time.perf_counter() - t0
        return r

    def staged_layer():
        # the oracle's layer forward, stage by stage
        x_r = timed("latent_down", O.latent_down, x, extra["Wdown"]) if s.H else x
        logits = timed("router_logits", O.router_logits, x_r, Wr, bias)
        idx, prob = timed("route", O.route, logits, s.K)
        _, off, _, inv = timed("permutation", O.expert_permutation, idx, s.E)
        x_disp, p_disp = timed("dispatch", O.dispatch, x_r, prob, inv, s.K)
        _, _, y_disp = timed("expert_ffn", O.expert_ffn, x_disp, off, Experts(W1c), Experts(W2c))
        y = timed("combine", O.combine, y_disp, p_disp, inv, T, s.K)
        if s.H:
            timed("latent_up", O.latent_up, y, extra["Wup"])

    runs, dt = 0, 0.0
    while runs < max_runs and (runs == 0 or dt < min_seconds):
        t0 = time.perf_counter()
        if staged:
            staged_layer()
        else:
            O.layer_fwd(x, Wr, Experts(W1c), Experts(W2c), s.K, bias=bias, **extra)
        dt += time.perf_counter() - t0
        runs += 1
    blas = [d.get("num_threads", 1) for d in threadpool_info() if d.get("user_api") == "blas"]
    rec = {
        "value": runs * T * s.K / dt, "unit": "slots/s", "cores": int(max(blas) if blas else 1),
        "kind": "oracle",
        "sample": f"{runs} pass(es) over the first {T} of {s.S} tokens of the same workload through the "
                  f"float64 oracle layer forward ({T * s.K} routed rows per pass, {dt:.1f} s in all; BLAS "
                  f"matmuls threaded, routing and permutation single-threaded Python)",
        **host_info(),
    }
    if stage_s:
        rec["stage_seconds_per_pass"] = {k: round(v / runs, 3) for k, v in stage_s.items()}
    return rec


def settle_and_time(step, steps, warmup, settle_seconds, stream):
    """Run the layer for settle_seconds and `warmup` steps, then time `steps`
    steps with one pair of HIP events: seconds per step.  A GPU that has just
    started work runs its first tens of steps ~10% slower (measured: 0.642 ms
    per step after 5 warm-up steps, 0.579 ms after 100); a training or
    serving loop runs at the sustained rate."""
    import torch
    t_end, i = time.perf_counter() + settle_seconds, 0
    while time.perf_counter() < t_end:
        step(i)
        i += 1
        if i % 8 == 0:
            torch.cuda.synchronize()
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    return time_region(step, steps, stream)


def other_workload(name, args, dev, stream):
    """Layer rate and the dominant grouped GEMM of another workload: value,
    ms per step and the GEMM's fraction of the bf16 MFMA peak, measured as
    for the headline (rotating input sets, sustained clock, GEMM launches
    timed inside the layer's own launch sequence where the layer has no
    latent projection)."""
    import torch
    from paper_2608_28511_amd import _lib, layer
    from paper_2608_28511_amd.workloads import PAPER_SHAPES, PRODUCTION, WORKLOADS, make_inputs
    s = {**WORKLOADS, **PRODUCTION, **PAPER_SHAPES}[name]
    log(f"other workload {name}: {args.sets} input sets")
    sets = [make_inputs(s, device=dev, seed=s.seed + 1000 * i) for i in range(args.sets)]
    modes = dict(score=s.score, Fs=s.Fs, seq_len=s.seq_len, aux_coeff=s.aux_coeff)
    lf = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, H=s.H, device=dev, export=False, **modes)

    def call(l, i):
        inp = sets[i % len(sets)]
        return l(inp["x"], inp["Wr"], inp["W1"], inp["W2"], bias=inp["bias"], Wdown=inp.get("Wdown"),
                 Wup=inp.get("Wup"), sel_bias=inp.get("sel_bias"), Ws1=inp.get("Ws1"), Ws2=inp.get("Ws2"))

    t_layer = settle_and_time(lambda i: call(lf, i), args.other_steps, args.warmup, args.settle_seconds, stream)
    # the intermediates the GEMM timings read, from one exporting call
    lfx = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, H=s.H, device=dev, export=True, **modes)
    out = call(lfx, 0)
    reps = args.stage_reps
    h2 = torch.empty_like(out["h"])
    yd2 = torch.empty_like(out["y_disp"])
    if s.score == "softmax" and not s.H:
        ws_router = torch.empty(max(1, _lib.moe_router_logits_workspace_bytes(s.D, s.E)), dtype=torch.uint8,
                                device=dev)
        ws_route = torch.empty(max(1, _lib.moe_route_workspace_bytes(s.S, s.E, s.K)), dtype=torch.uint8,
                               device=dev)
        r_bufs = {k: torch.empty_like(out[k]) for k in ("topk_idx", "topk_prob", "counts", "offsets",
                                                          "perm", "inv_perm")}
        xd2 = torch.empty_like(out["x_disp"])
        pd2 = torch.empty_like(out["p_disp"])
        t_up, t_down = time_layer_gemms(_lib, sets, out, s, reps, stream, ws_router, ws_route, r_bufs, xd2, pd2,
                                        h2, yd2)
    else:
        sched = layer.grouped_schedule(out["offsets"], s.E, s.R)
        t_up = time_region(lambda i: _lib.moe_grouped_gemm(out["x_disp"], sched, s.E, s.R, s.D, s.F,
                                                           sets[i % len(sets)]["W1"], 1, h2, None), reps, stream)
        t_down = time_region(lambda i: _lib.moe_grouped_gemm(out["h"], sched, s.E, s.R, s.F, s.D,
                                                             sets[i % len(sets)]["W2"], 0, yd2, None), reps, stream)
    fl = 2.0 * s.R * s.D * s.F
    e_used = int((out["counts"] > 0).sum().item())
    dom, t_dom = ("grouped_up", t_up) if t_up >= t_down else ("grouped_down", t_down)
    rec = {"value": round(s.R / t_layer, 1), "unit": "slots/s", "ms_per_step": round(t_layer * 1e3, 4),
           "steps": args.other_steps,
           "grouped_up_us": round(t_up * 1e6, 1), "grouped_down_us": round(t_down * 1e6, 1),
           "roofline": gemm_roofline(dom, fl, gemm_bytes(s, e_used), t_dom)}
    del sets, lf, lfx, out, h2, yd2
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return rec


def main():
    args = parse()
    if args.traffic_from:
        write_traffic(*args.traffic_from, args.workload, args.traffic_kernel, args.calib_bytes,
                      args.traffic_bench_args)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: this build has no multi-GPU path "
              f"(--gpus {args.gpus} requested).", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2608_28511_amd import _lib, layer
    from paper_2608_28511_amd.workloads import PAPER_SHAPES, PRODUCTION, WORKLOADS, make_inputs

    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        sys.exit(1)
    _lib.load(build_if_missing=True)
    s = {**WORKLOADS, **PRODUCTION, **PAPER_SHAPES}[args.workload]
    prod = s.score == "sigmoid"
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()

    log(f"generating {args.sets} input sets for {s.name}")
    sets = [make_inputs(s, device=dev, seed=s.seed + 1000 * i) for i in range(args.sets)]
    modes = dict(score=s.score, Fs=s.Fs, seq_len=s.seq_len, aux_coeff=s.aux_coeff)
    # the timed layer exports nothing but y, as a training or serving step
    # would call it (with the bf16 payload the dispatch is then fused into the
    # up projection's operand copy); stage timings read the intermediates of
    # one more, exporting call
    lf = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, H=s.H, device=dev, export=False, payload=args.payload, **modes)
    lfx = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, H=s.H, device=dev, export=True, payload=args.payload, **modes)
    mx_run = args.payload == "mxfp8"
    if mx_run:
        lfx.out["x_disp"] = None   # the up projection reads the payload as sent: no decode pass

    # a plain device copy of known size, once, so hardware byte counters can be
    # calibrated against it in profiler runs of this same command
    n = args.calib_bytes // 2
    a = torch.empty(n, dtype=torch.bfloat16, device=dev).fill_(1.0)
    b = torch.empty_like(a)
    b.copy_(a)
    del a, b
    torch.cuda.synchronize()

    def step(i):
        inp = sets[i % len(sets)]
        lf(inp["x"], inp["Wr"], inp["W1"], inp["W2"], bias=inp["bias"], Wdown=inp.get("Wdown"),
           Wup=inp.get("Wup"), sel_bias=inp.get("sel_bias"), Ws1=inp.get("Ws1"), Ws2=inp.get("Ws2"))

    log(f"settle {args.settle_seconds} s, warmup {args.warmup}, timed {args.steps}")
    t_layer = settle_and_time(step, args.steps, args.warmup, args.settle_seconds, stream)
    slots = s.S * s.K
    value = slots / t_layer
    # the same steps once more, each with its own events, for the paper's
    # per-step statistics (median and the mean after iteratively dropping
    # samples above mean + 1.5 sigma); not part of the timed region above
    per_step = step_times(step, args.steps, stream)

    # ---- per-stage timings on the same stream, same launch configuration ----
    i0 = sets[0]
    out = lfx(i0["x"], i0["Wr"], i0["W1"], i0["W2"], bias=i0["bias"], Wdown=i0.get("Wdown"), Wup=i0.get("Wup"),
              sel_bias=i0.get("sel_bias"), Ws1=i0.get("Ws1"), Ws2=i0.get("Ws2"))
    reps = args.stage_reps
    st = {}
    # an untimed write of more bytes than the 256 MB last-level cache holds,
    # enqueued before each timed launch of an HBM-bound stage
    fbuf = torch.empty(max(1, args.flush_bytes), dtype=torch.uint8, device=dev)
    flush = lambda: fbuf.fill_(0)  # noqa: E731
    ws_router = torch.empty(max(1, _lib.moe_router_logits_workspace_bytes(s.D, s.E)), dtype=torch.uint8,
                            device=dev)
    st["router_logits"] = time_flushed(
        lambda i: _lib.moe_router_logits(sets[i % len(sets)]["x"] if not s.H else out["x_lat"],
                                         sets[i % len(sets)]["Wr"], sets[i % len(sets)]["bias"],
                                         s.S, s.D, s.E, out["logits"], ws_router), reps, stream, flush)
    ws_route = torch.empty(max(1, _lib.moe_route_workspace_bytes(s.S, s.E, s.K)), dtype=torch.uint8,
                           device=dev)
    r_bufs = {k: torch.empty_like(out[k]) for k in ("topk_idx", "topk_prob", "counts", "offsets",
                                                      "perm", "inv_perm")}
    if prod:
        st["route"] = time_flushed(
            lambda i: _lib.moe_route_sigmoid(out["logits"], sets[i % len(sets)]["sel_bias"], s.S, s.E, s.K,
                                             r_bufs["topk_idx"], r_bufs["topk_prob"], r_bufs["counts"],
                                             r_bufs["offsets"], r_bufs["perm"], r_bufs["inv_perm"], ws_route),
            reps, stream, flush)
    else:
        st["route"] = time_flushed(
            lambda i: _lib.moe_route_topk(out["logits"], s.S, s.E, s.K, r_bufs["topk_idx"],
                                          r_bufs["topk_prob"], r_bufs["counts"], r_bufs["offsets"],
                                          r_bufs["perm"], r_bufs["inv_perm"], ws_route), reps, stream, flush)
    if s.seq_len:
        ws_aux = torch.empty(max(1, _lib.moe_seq_aux_loss_workspace_bytes(s.S, s.E, s.seq_len)),
                             dtype=torch.uint8, device=dev)
        loss2 = torch.empty(1, dtype=torch.float32, device=dev)
        cnt2 = torch.empty((s.S // s.seq_len, s.E), dtype=torch.int32, device=dev)
        st["seq_aux_loss"] = time_flushed(
            lambda i: _lib.moe_seq_aux_loss(out["logits"], out["topk_idx"], s.S, s.E, s.K, s.seq_len, s.aux_coeff,
                                            loss2, cnt2, ws_aux), reps, stream, flush)
    xd2 = torch.empty((s.R, s.D), dtype=torch.bfloat16, device=dev)
    pd2 = torch.empty_like(out["p_disp"])
    x_r = [(st_["x"] if not s.H else out["x_lat"]) for st_ in sets]
    st["dispatch"] = time_flushed(
        lambda i: _lib.moe_dispatch(x_r[i % len(x_r)], out["topk_prob"], out["inv_perm"], s.S, s.D,
                                    s.K, xd2, pd2), reps, stream, flush)
    if s.D % 32 == 0:
        xq2 = torch.empty((s.R, s.D), dtype=torch.uint8, device=dev)
        xs2 = layer.mx_scales(s.R, s.D, dev)
        st["dispatch_mxfp8"] = time_flushed(
            lambda i: _lib.moe_dispatch_mxfp8(x_r[i % len(x_r)], out["topk_prob"], out["inv_perm"], s.S, s.D, s.K,
                                              xq2, xs2, pd2), reps, stream, flush)
        st["mxfp8_dequant"] = time_flushed(lambda i: _lib.moe_mxfp8_dequant(xq2, xs2, s.R, s.D, xd2), reps, stream, flush)
    sched = layer.grouped_schedule(out["offsets"], s.E, s.R)
    h2 = torch.empty_like(out["h"])
    if s.D % 32 == 0:
        # the up projection reading the MX-FP8 payload as sent (decode in its operand path)
        _lib.moe_dispatch_mxfp8(x_r[0], out["topk_prob"], out["inv_perm"], s.S, s.D, s.K, xq2, xs2, pd2)
        st["grouped_up_mxfp8"] = time_region(
            lambda i: _lib.moe_grouped_gemm_mxfp8(xq2, xs2, sched, s.E, s.R, s.D, s.F, sets[i % len(sets)]["W1"],
                                                  1, h2, None), reps, stream)
    yd2 = torch.empty_like(out["y_disp"])
    # the two grouped GEMMs inside the layer's own launch sequence (router,
    # route, dispatch, schedule, up, down, combine per input set), each GEMM
    # launch bracketed by its own events, so they run under the cache and
    # clock conditions of the timed layer steps
    if not prod and not s.H:
        st["grouped_up"], st["grouped_down"] = time_layer_gemms(
            _lib, sets, out, s, reps, stream, ws_router, ws_route, r_bufs, xd2, pd2, h2, yd2,
            mx=(xq2, xs2) if mx_run else None)
    else:
        if mx_run:
            st["grouped_up"] = st["grouped_up_mxfp8"]
        else:
            st["grouped_up"] = time_region(
                lambda i: _lib.moe_grouped_gemm(out["x_disp"], sched, s.E, s.R, s.D, s.F,
                                                sets[i % len(sets)]["W1"], 1, h2, None), reps, stream)
        st["grouped_down"] = time_region(
            lambda i: _lib.moe_grouped_gemm(out["h"], sched, s.E, s.R, s.F, s.D,
                                            sets[i % len(sets)]["W2"], 0, yd2, None), reps, stream)
    y2 = torch.empty((s.S, s.D), dtype=torch.bfloat16, device=dev)
    if s.Fs:
        hs2 = torch.empty_like(out["h_s"])
        ys2 = torch.empty_like(out["y_s"])
        st["shared_fwd"] = time_region(
            lambda i: _lib.moe_shared_expert_fwd(sets[i % len(sets)]["x"], sets[i % len(sets)]["Ws1"],
                                                 sets[i % len(sets)]["Ws2"], s.S, s.D, s.Fs, hs2, None, ys2),
            reps, stream)
        st["combine"] = time_flushed(
            lambda i: _lib.moe_combine_add(out["y_disp"], out["p_disp"], out["inv_perm"], out["y_s"], s.S, s.D,
                                           s.K, y2), reps, stream, flush)
    else:
        st["combine"] = time_flushed(
            lambda i: _lib.moe_combine(out["y_disp"], out["p_disp"], out["inv_perm"], s.S, s.D, s.K, y2),
            reps, stream, flush)
    if s.H:
        st["latent_down"] = time_region(
            lambda i: _lib.moe_latent_proj(sets[i % len(sets)]["x"], sets[i % len(sets)]["Wdown"],
                                           s.S, s.H, s.D, out["x_lat"]), reps, stream)

    if s.backward:
        # backward stages (reported per stage; `value` stays the forward rate)
        lb = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, H=s.H, device=dev, export=True, save_u=True, **modes)
        i0 = sets[0]
        ob = lb(i0["x"], i0["Wr"], i0["W1"], i0["W2"], bias=i0["bias"], sel_bias=i0.get("sel_bias"),
                Ws1=i0.get("Ws1"), Ws2=i0.get("Ws2"))
        dy = sets[0]["dy"]
        dy_disp = torch.empty_like(ob["x_disp"])
        dp = torch.empty((s.S, s.K), dtype=torch.float32, device=dev)
        dx_disp = torch.empty_like(ob["x_disp"])
        dW1 = torch.empty((s.E, s.D, s.F), dtype=torch.float32, device=dev)
        dW2 = torch.empty((s.E, s.F, s.D), dtype=torch.float32, device=dev)
        dx = torch.empty((s.S, s.D), dtype=torch.bfloat16, device=dev)
        ws_bwd = torch.empty(max(1, _lib.moe_grouped_ffn_bwd_workspace_bytes(s.E, s.R, s.D, s.F)),
                             dtype=torch.uint8, device=dev)
        st["combine_bwd"] = time_flushed(
            lambda i: _lib.moe_combine_bwd(dy, ob["y_disp"], ob["p_disp"], ob["inv_perm"], s.S, s.D, s.K,
                                           dy_disp, dp), reps, stream, flush)
        st["grouped_ffn_bwd"] = time_region(
            lambda i: _lib.moe_grouped_ffn_bwd(ob["x_disp"], ob["u_save"], ob["h"], dy_disp, ob["offsets"],
                                               s.E, s.R, s.D, s.F, sets[0]["W1"], sets[0]["W2"], dx_disp,
                                               dW1, dW2, ws_bwd), max(2, reps // 4), stream)
        dWr = torch.empty((s.D, s.E), dtype=torch.float32, device=dev)
        dbias = torch.empty((s.E,), dtype=torch.float32, device=dev)
        dx_r = torch.empty((s.S, s.D), dtype=torch.float32, device=dev)
        if prod:
            ws_rb = torch.empty(max(1, _lib.moe_router_bwd_sigmoid_workspace_bytes(s.S, s.D, s.E)), dtype=torch.uint8,
                                device=dev)
            st["router_bwd"] = time_region(
                lambda i: _lib.moe_router_bwd_sigmoid(i0["x"], i0["Wr"], ob["logits"], ob["topk_idx"],
                                                      ob["topk_prob"], dp, ob["seq_counts"], s.seq_len, s.aux_coeff,
                                                      s.S, s.D, s.E, s.K, None, dWr, dbias, dx_r, ws_rb),
                reps, stream)
        else:
            ws_rb = torch.empty(max(1, _lib.moe_router_bwd_workspace_bytes(s.S, s.D, s.E)), dtype=torch.uint8,
                                device=dev)
            st["router_bwd"] = time_region(
                lambda i: _lib.moe_router_bwd(i0["x"], i0["Wr"], ob["topk_idx"], ob["topk_prob"], dp, s.S, s.D,
                                              s.E, s.K, None, dWr, None if i0["bias"] is None else dbias, dx_r,
                                              ws_rb), reps, stream)
        if s.Fs:
            dWs1 = torch.empty((s.D, s.Fs), dtype=torch.float32, device=dev)
            dWs2 = torch.empty((s.Fs, s.D), dtype=torch.float32, device=dev)
            ws_sb = torch.empty(max(1, _lib.moe_shared_expert_bwd_workspace_bytes(s.S, s.D, s.Fs)),
                                dtype=torch.uint8, device=dev)
            st["shared_bwd"] = time_region(
                lambda i: _lib.moe_shared_expert_bwd(i0["x"], ob["u_s"], ob["h_s"], dy, i0["Ws1"], i0["Ws2"], s.S,
                                                     s.D, s.Fs, dx_r, True, dWs1, dWs2, ws_sb),
                max(2, reps // 4), stream)
        st["dispatch_bwd"] = time_flushed(
            lambda i: _lib.moe_dispatch_bwd_add(dx_disp, ob["inv_perm"], dx_r, s.S, s.D, s.K, dx), reps, stream, flush)
        del lb, ob, dy_disp, dx_disp, dW1, dW2, ws_bwd

    bytes_ = stage_bytes(s)
    gemm_flops = 2.0 * s.R * s.D * s.F
    stages = {}
    for k, t in st.items():
        e = {"us": round(t * 1e6, 2)}
        if k in ("route", "dispatch", "combine", "combine_bwd", "dispatch_bwd", "seq_aux_loss", "dispatch_mxfp8",
                 "mxfp8_dequant"):
            gbs = bytes_[k] / t / 1e9
            e.update(bytes=bytes_[k], GBps=round(gbs, 1), hbm_frac=round(gbs / PEAK_HBM_GBS, 4))
        elif k == "router_logits":
            # fp32 products computed as three bf16 MFMAs; bounded by HBM
            tf = 2.0 * s.S * s.D * s.E / t / 1e12
            gbs = bytes_[k] / t / 1e9
            e.update(TFLOPs_fp32_equiv=round(tf, 2), bytes=bytes_[k], GBps=round(gbs, 1),
                     hbm_frac=round(gbs / PEAK_HBM_GBS, 4))
        elif k == "router_bwd":
            # dWr (x^T against three bf16 planes of dlogits) and dx_r, in fp32-equivalent flops
            tf = 4.0 * s.S * s.D * s.E / t / 1e12
            e.update(TFLOPs_fp32_equiv=round(tf, 2))
        else:
            if k == "grouped_ffn_bwd":
                fl = 4.0 * gemm_flops      # dgrad and wgrad of both projections
            elif k == "shared_fwd":
                fl = 4.0 * s.S * s.D * s.Fs
            elif k == "shared_bwd":
                fl = 8.0 * s.S * s.D * s.Fs  # two dgrads, two wgrads
            else:
                fl = gemm_flops if k.startswith("grouped") else 2.0 * s.S * s.H * s.D
            tf = fl / t / 1e12
            e.update(flops=fl, TFLOPs=round(tf, 1), mfma_frac=round(tf / PEAK_BF16_TFLOPS, 4))
        stages[k] = e

    dom = max(("grouped_up", "grouped_down"), key=lambda k: st[k])
    # on the MX payload the timed up projection is the kernel that decodes it
    dom_kernel = "grouped_up_mxfp8" if mx_run and dom == "grouped_up" else dom
    e_used = int((out["counts"] > 0).sum().item())
    gb = gemm_bytes(s, e_used)
    roofline = gemm_roofline(
        dom_kernel, gemm_flops, gb, st[dom], traffic=load_traffic(dom_kernel, s.name),
        per_launch=(f"2*R*D*F = {gemm_flops:.4g} flop and R*D*2 + R*F*2 + E_used*D*F*2 = {gb:.4g} bytes "
                    f"per launch (R = S*K = {s.R}, E_used = {e_used})"))

    cpu = None
    if not args.no_cpu_baseline:
        log(f"cpu baseline: oracle on {args.cpu_tokens or s.S} tokens")
        cpu = cpu_baseline(s, sets[0], args.cpu_tokens, args.payload)

    # the other full-size workloads, after the headline's buffers are freed
    route_sw = route_sweep(_lib, s, reps, stream, dev) if args.route_sweep else None
    ep = ep_share(_lib, s, args.ep_share, reps, stream, dev) if args.ep_share > 1 else None
    del sets, lf, lfx, out, fbuf
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    others = {}
    for name in [n for n in args.others.split(",") if n and n != s.name]:
        others[name] = other_workload(name, args, dev, stream)

    rec = {
        "metric": METRIC, "value": round(value, 1), "unit": "slots/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(t_layer * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": s.name, "S": s.S, "D": s.D, "E": s.E, "K": s.K, "F": s.F,
                   "H": s.H, "rotating_input_sets": args.sets, "parallelism": "none (1 GPU)",
                   **({"payload": "mxfp8"} if args.payload == "mxfp8" else {}),
                   **({"score": s.score, "Fs": s.Fs, "seq_len": s.seq_len, "aux_coeff": s.aux_coeff}
                      if prod else {})},
        "roofline": roofline, "stages": stages, "cpu_baseline": cpu,
        **({"ep_share": ep} if ep is not None else {}),
        **({"route_sweep": route_sw} if route_sw is not None else {}),
        **({"other_workloads": others} if others else {}),
        "layer_step_us": {"n": len(per_step), "median": round(statistics.median(per_step), 2),
                          "filtered_mean": round(filtered_mean(per_step), 2),
                          "min": round(min(per_step), 2), "max": round(max(per_step), 2)},
        # Eq. 1: forward dispatch payload with bf16 and with MX-FP8 hidden elements
        "payload": {"timed": args.payload, "eq1_dispatch_bytes_bf16": _lib.moe_payload_bytes(s.S, s.K, s.D),
                    "eq1_dispatch_bytes_mxfp8": _lib.moe_mx_payload_bytes(s.S, s.K, s.D),
                    "mxfp8_over_bf16": round(_lib.moe_mx_payload_bytes(s.S, s.K, s.D)
                                             / _lib.moe_payload_bytes(s.S, s.K, s.D), 4)},
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
