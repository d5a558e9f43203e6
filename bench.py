"""Benchmark: fused training step vs the unfused eager step on one MI355X.

Workload (default): the 8-layer fp32 MLP of width 1024, batch 256, Adam
(mlp8x1024).  A step is one training iteration over one resident batch.  All
three orderings run on the same inputs in the same process:
  eager  forward, backward writing every gradient, one multi-tensor optimizer launch
  ff     forward-fusion (update applied while the next forward loads W)
  bf     backward-fusion (update in the weight-gradient epilogue, second stream)
The headline is backward-fusion.  `value` is its update bandwidth: the
parameter and optimizer-state bytes the fused step must move, over its step
time.

The dominant kernel of the fused step is timed live with HIP events on the
stream it runs on, during the timed steps, and set against its roofline
(algorithmic bytes or flops per launch over MI355X peaks: HBM 8 TB/s, fp32
MFMA 157.3 TFLOP/s).  The CPU baseline is the float64 oracle's eager step on
this host, timed on a bounded sample of steps.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from workloads import get_config, make_params, make_batch  # noqa: E402

PEAK_HBM = 8.0e12          # bytes/s
PEAK_FP32_MFMA = 157.3e12  # flop/s

METRIC = "fused train-step time & update GB/s vs unfused eager; % of HBM/MFMA roofline"


# ----------------------------------------------------------------- cost model
def state_bytes_per_param(kind, ordering):
    """Parameter + optimizer-state bytes one parameter costs per step (fp32).

    Reads and writes of theta, its gradient and its history across the stages
    (Fig. 2 accounting): eager = fwd R theta, dgrad R theta, wgrad W g, opt
    R theta,g,hist W theta,hist; ff = fused fwd R theta,g,hist W theta,hist,
    dgrad R theta, wgrad W g; bf = fwd R theta, dgrad R theta, fused wgrad
    R theta,hist W theta,hist.
    """
    h = 2 if kind != "sgd" else 1          # history tensors (m, v) or (momentum)
    upd = 4 * (2 + 2 * h)                  # R theta,hist + W theta,hist
    if ordering == "eager":
        return 4 + 4 + 4 + (upd + 4)
    if ordering == "ff":
        return (upd + 4) + 4 + 4
    return 4 + 4 + upd


def linear_launches(cfg):
    """Per-launch algorithmic (flops, bytes) of each kernel class, by layer."""
    M = cfg["batch"]
    dims = cfg["dims"]
    kind = cfg["opt"]["kind"]
    h = 2 if kind != "sgd" else 1
    out = []
    for i in range(1, len(dims)):
        K, N = dims[i - 1], dims[i]
        act_prev = i > 1 and cfg["act"] != "none"
        w, xb, yb = 4 * N * K, 4 * M * K, 4 * M * N
        bias = 4 * N if cfg["bias"] else 0
        upd_w = 4 * N * K * (2 + 2 * h)          # R W,hist + W W,hist
        upd_b = 4 * N * (2 + 2 * h) if cfg["bias"] else 0
        f = 2 * M * N * K
        out.append(dict(
            layer=i, N=N, K=K,
            fwd=(f, xb + w + yb + bias),
            fwd_ff=(f, xb + yb + w * 2 + upd_w + bias * 2 + upd_b),   # + R g_W, g_b
            dgrad=(f, yb + w + xb + (xb if act_prev else 0)) if i > 1 else None,
            wgrad=(f, yb + xb + w + bias),
            wgrad_bf=(f, yb + xb + upd_w + upd_b),
        ))
    return out


def step_cost(cfg, ordering):
    """Whole-step algorithmic flops and bytes (kernels as implemented)."""
    L = linear_launches(cfg)
    F = B = 0
    for d in L:
        fk = "fwd_ff" if ordering == "ff" else "fwd"
        wk = "wgrad_bf" if ordering == "bf" else "wgrad"
        for k in (fk, "dgrad", wk):
            if d[k] is not None:
                F += d[k][0]
                B += d[k][1]
    n = sum(d["N"] * d["K"] + (d["N"] if cfg["bias"] else 0) for d in L)
    h = 2 if cfg["opt"]["kind"] != "sgd" else 1
    if ordering == "eager":
        B += n * 4 * (3 + 2 * h)           # R w, g, hist; W w, hist
    M, C = cfg["batch"], cfg["dims"][-1]
    B += 4 * M * C * 2
    return F, B


def kernel_roofline(flops, nbytes, seconds):
    t_hbm, t_mfma = nbytes / PEAK_HBM, flops / PEAK_FP32_MFMA
    if t_hbm >= t_mfma:
        ach = nbytes / seconds / 1e9
        return dict(bound="hbm", achieved=round(ach, 1), peak=PEAK_HBM / 1e9, unit="GB/s",
                    frac=round(ach / (PEAK_HBM / 1e9), 4))
    ach = flops / seconds / 1e12
    return dict(bound="mfma", achieved=round(ach, 2), peak=PEAK_FP32_MFMA / 1e12,
                unit="TFLOP/s", frac=round(ach / (PEAK_FP32_MFMA / 1e12), 4))


def traffic_for(kernel_class, workload):
    """HBM bytes per launch measured by rocprofv3 counters, if recorded for the
    current kernel source (profiles/traffic.json keyed by the source hash)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    src = os.path.join(ROOT, "paper_2104_00237_amd", "csrc", "gemm_f32.hip")
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    rec = json.load(open(path)).get(f"{workload}:{kernel_class}")
    if not rec or rec.get("source_sha") != digest:
        return None
    return rec.get("bytes_per_launch")


# ------------------------------------------------------------------ timing
def time_ordering(torch, cfg, ordering, batches, warmup, steps, timer_classes=(), graph=True):
    """Mean step time of one ordering.  graph: every step is a replay of a HIP graph
    captured once per resident batch (the step-dependent optimizer constants are
    read from the device step counter); else each step is launched from Python."""
    from paper_2104_00237_amd.trainer import Trainer, KernelTimer
    tr = Trainer(cfg, make_params(cfg), "cuda:0")
    n = len(batches)
    for t in range(max(warmup, 1)):
        x, y = batches[t % n]
        tr.step(x, y, ordering)
    timer = KernelTimer(timer_classes) if timer_classes else None
    if graph and timer is None:
        runs = [tr.capture(x, y, ordering) for x, y in batches]
        for t in range(n):          # each graph once before timing
            runs[t]()
    else:
        tr.timer = timer
        runs = [(lambda xy=xy: tr.step(xy[0], xy[1], ordering)) for xy in batches]
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(tr.stream)
    t_host = time.perf_counter()
    for t in range(steps):
        runs[(warmup + t) % n]()
    e1.record(tr.stream)
    torch.cuda.synchronize()
    host_s = time.perf_counter() - t_host
    ms = e0.elapsed_time(e1) / steps
    losses = tr.loss_history()
    tr.timer = None
    return ms, host_s / steps * 1e3, timer, losses


def cpu_baseline(cfg, budget_s=15.0):
    import oracle
    from oracle.train import new_model
    model = new_model(cfg)
    t0 = time.perf_counter()
    n = 0
    while True:
        x, y = make_batch(cfg, n + 1)
        y = y if y.dtype == np.int64 else y.astype(np.float64)
        model.step_eager(x.astype(np.float64), y)
        n += 1
        if time.perf_counter() - t0 >= budget_s or n >= cfg["steps"]:
            break
    dt = (time.perf_counter() - t0) / n
    del oracle
    return dt, n


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="mlp8x1024")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (HBM counter calibration)")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        n = args.calibrate_copy << 18  # floats
        src = torch.ones(n, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 3}))
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch
    cfg = get_config(args.workload)
    if cfg["kind"] != "mlp" or cfg["dtype"] != "f32":
        print(f"workload {args.workload} has no GPU path in this build", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    nb = 4
    batches = []
    for t in range(1, nb + 1):
        x, y = make_batch(cfg, t)
        batches.append((torch.as_tensor(x).to(dev), torch.as_tensor(y).to(dev)))
    torch.cuda.synchronize()

    res = {}
    for o in ("eager", "ff", "bf"):
        ms, host_ms, _, _ = time_ordering(torch, cfg, o, batches, args.warmup, args.steps,
                                          graph=False)
        ms_g = None
        if not args.no_graph:
            ms_g, _, _, _ = time_ordering(torch, cfg, o, batches, args.warmup, args.steps,
                                          graph=True)
        res[o] = dict(ms=ms, host_ms=host_ms, ms_graph=ms_g)
        print(f"[bench] {o}: {ms:.4f} ms/step launched (host {host_ms:.4f}), "
              f"graph replay {ms_g} ms/step", file=sys.stderr, flush=True)

    # Dominant kernel of the fused (bf) step: one instrumented pass finds the class
    # with the largest total time; the timed pass then brackets only that class.
    classes = ("fwd", "dgrad", "wgrad_bf", "loss")
    _, _, probe, _ = time_ordering(torch, cfg, "bf", batches, 2, 3, classes)
    totals = {c: sum(d for d, _ in probe.durations(c)) for c in classes}
    dom = max(totals, key=totals.get)
    ms_dom_step, _, timer, _ = time_ordering(torch, cfg, "bf", batches, args.warmup, args.steps,
                                             (dom,))
    launches = linear_launches(cfg)
    recs = timer.durations(dom)
    # Group by layer shape: report the largest shape's launches (the repeated hidden layer).
    by_shape = {}
    for d_ms, op in recs:
        by_shape.setdefault((op.N, op.K), []).append(d_ms)
    shape = max(by_shape, key=lambda s: s[0] * s[1])
    durs = by_shape[shape]
    per = next(d for d in launches if (d["N"], d["K"]) == shape)[dom]
    # Each launch is bracketed by an event pair on its own stream; the pair's own
    # cost (an empty pair on the same stream) is taken off.
    from paper_2104_00237_amd.trainer import KernelTimer
    dom_stream = torch.cuda.Stream() if dom == "wgrad_bf" else torch.cuda.current_stream()
    marker_ms = KernelTimer.marker_overhead_ms(dom_stream)
    avg_s = (float(np.mean(durs)) - marker_ms) / 1e3
    roof = kernel_roofline(per[0], per[1], avg_s)
    roof.update(kernel=dom, shape=f"M={cfg['batch']} N={shape[0]} K={shape[1]}",
                avg_us=round(avg_s * 1e6, 3), launches=len(durs),
                bracketed_avg_us=round(float(np.mean(durs)) * 1e3, 3),
                marker_us=round(marker_ms * 1e3, 3),
                algorithmic_bytes=per[1], algorithmic_flops=per[0],
                traffic=traffic_for(dom, args.workload))

    n_params = sum(d["N"] * d["K"] + (d["N"] if cfg["bias"] else 0) for d in launches)
    kind = cfg["opt"]["kind"]
    upd_bytes = n_params * state_bytes_per_param(kind, "bf")
    bf_s = res["bf"]["ms"] / 1e3
    value = upd_bytes / bf_s / 1e9
    F, B = step_cost(cfg, "bf")
    step_roof_s = max(B / PEAK_HBM, F / PEAK_FP32_MFMA)

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(res["bf"]["ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "global_batch": cfg["batch"],
                   "layers": f"{len(cfg['dims']) - 1}x{cfg['dims'][1]}",
                   "optimizer": kind, "ordering": "backward-fusion",
                   "parallelism": "single-gpu"},
        "eager_ms_per_step": round(res["eager"]["ms"], 4),
        "ff_ms_per_step": round(res["ff"]["ms"], 4),
        "bf_ms_per_step": round(res["bf"]["ms"], 4),
        "speedup_bf_vs_eager": round(res["eager"]["ms"] / res["bf"]["ms"], 4),
        "speedup_ff_vs_eager": round(res["eager"]["ms"] / res["ff"]["ms"], 4),
        "ms_per_step_graph_replay": {o: (round(r["ms_graph"], 4) if r["ms_graph"] else None)
                                     for o, r in res.items()},
        "host_ms_per_step": {o: round(r["host_ms"], 4) for o, r in res.items()},
        "timing": "steps launched from the host scheduler; graph replay reported beside",
        "step_roofline": {"flops": F, "bytes": B, "roofline_ms": round(step_roof_s * 1e3, 5),
                          "frac": round(step_roof_s / bf_s, 4)},
        "update_bytes_per_step": {o: n_params * state_bytes_per_param(kind, o)
                                  for o in ("eager", "ff", "bf")},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        dt, n = cpu_baseline(cfg, args.cpu_budget)
        cores = len(os.sched_getaffinity(0))
        try:
            from threadpoolctl import threadpool_info
            blas = [i["num_threads"] for i in threadpool_info() if i.get("user_api") == "blas"]
            cores = min(cores, max(blas)) if blas else cores
        except Exception:
            pass
        eager_bytes = n_params * state_bytes_per_param(kind, "eager")
        out["cpu_baseline"] = {"value": round(eager_bytes / dt / 1e9, 4), "unit": "GB/s",
                               "cores": cores, "kind": "oracle",
                               "ms_per_step": round(dt * 1e3, 2),
                               "sample": f"{n} eager float64 steps of {args.workload} "
                                         f"(oracle, numpy, {cores} host threads)"}
    print(json.dumps(out))


if __name__ == "__main__":
    main()
