"""Benchmark: fused training step vs the unfused eager step on one MI355X.

Workload (default): the parameter-bound stack of four 8192 x 8192 fp32 linear
layers, 64 tokens, Adam (linear4x8192), the largest single-GPU configuration
at the paper's fp32 precision.  The 8-layer width-1024 MLP (mlp8x1024) is
timed beside it and reported under extra keys.  A step is one training
iteration over one resident batch.  All three orderings run on the same
inputs in the same process:
  eager  forward, backward writing every gradient, one multi-tensor optimizer launch
  ff     forward-fusion (update applied while the next forward loads W)
  bf     backward-fusion (update in the weight-gradient epilogue, second stream)
  bfm    backward-fusion with each layer's data gradient merged into the update's
         read of W (fp32 linear layers with at most 64 rows; linear4x8192)
The headline is backward-fusion (the faster of bf and bfm where bfm applies).  `value` is its update bandwidth: the
parameter and optimizer-state bytes the fused step must move, over its step
time.

The dominant kernel of the fused step is timed live with HIP events on the
stream it runs on, during the timed steps, and set against its roofline
(algorithmic bytes or flops per launch over MI355X peaks: HBM 8 TB/s, fp32
MFMA 157.3 TFLOP/s).  The HBM rates this device reaches with the library's
own streaming kernels (read only, and copy) are reported beside it
(`hbm_ceiling`).  The CPU baseline is the float64 oracle's eager step on this
host, timed on a bounded sample of steps.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
import argparse
import gc
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
PEAK_BF16_MFMA = 2.5e15    # flop/s, dense

METRIC = "fused train-step time & update GB/s vs unfused eager; % of HBM/MFMA roofline"

# --optimizer: the workload with another of the optimizers Fig. 7 compares
# (PyTorch's default hyperparameters; weight decay applied, as in the figure).
FIG7_OPTIMIZERS = {
    "sgd": dict(kind="sgd", lr=0.01, momentum=0.0, weight_decay=1e-4),
    "sgd_momentum": dict(kind="sgd", lr=0.01, momentum=0.9, weight_decay=1e-4),
    "adagrad": dict(kind="adagrad", lr=0.01, eps=1e-10, weight_decay=1e-4),
    "rmsprop": dict(kind="rmsprop", lr=0.01, alpha=0.99, eps=1e-8, weight_decay=1e-4),
    "adam": dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-4),
    "adadelta": dict(kind="adadelta", lr=1.0, rho=0.9, eps=1e-6, weight_decay=1e-4),
}


# ----------------------------------------------------------------- cost model
def n_state(hyper):
    """Optimizer state tensors the kernels stream per parameter: the momentum
    buffer (SGD), m and v (Adam, AdamW, Adadelta, RMSprop with momentum), or v
    alone (Adagrad, RMSprop without momentum)."""
    k = hyper["kind"]
    if k == "sgd" or k == "adagrad" or (k == "rmsprop" and not hyper.get("momentum", 0.0)):
        return 1
    return 2


def state_bytes_per_param(kind, ordering):
    """Parameter + optimizer-state bytes one parameter costs per step (fp32).

    Reads and writes of theta, its gradient and its history across the stages
    (Fig. 2 accounting): eager = fwd R theta, dgrad R theta, wgrad W g, opt
    R theta,g,hist W theta,hist; ff = fused fwd R theta,g,hist W theta,hist,
    dgrad R theta, wgrad W g; bf = fwd R theta, dgrad R theta, fused wgrad
    R theta,hist W theta,hist; bfm = fwd R theta, merged dgrad + update
    R theta,hist W theta,hist.
    """
    h = kind if isinstance(kind, int) else (2 if kind != "sgd" else 1)   # state tensors
    upd = 4 * (2 + 2 * h)                  # R theta,hist + W theta,hist
    if ordering == "eager":
        return 4 + 4 + 4 + (upd + 4)
    if ordering in ("ff", "ffp"):
        return (upd + 4) + 4 + 4
    if ordering == "bfm":
        return 4 + upd
    return 4 + 4 + upd


def layer_launches(cfg):
    """Per-launch algorithmic (flops, bytes) of each kernel class, by layer.

    Linear [M,K] -> [M,N]: 2MNK flops; bytes = operands read + results written
    once.  A 3x3 convolution counts as its implicit GEMM (M = N*H*W pixels,
    N = Cout, K = 9*Cin) for flops, with the activation tensors (not the
    gathered im2col matrix) for bytes.  Convolutions apply forward-fusion's
    pending update in an element-wise pass before the forward, counted in
    fwd_ff.  `extra` holds the max-pool bytes (forward, backward) after a layer.
    """
    h = n_state(cfg["opt"])

    def upd(n):                      # R theta,hist + W theta,hist
        return 4 * n * (2 + 2 * h)

    layers = []                      # (name, kind, M, N, K, in_elems, out_elems, bias, act_prev, pool)
    if cfg["kind"] == "tblock":
        return tblock_launches(cfg)
    if cfg["kind"] == "mbv2":
        return mbv2_launches(cfg)
    if cfg["kind"] == "mlp":
        M, dims = cfg["batch"], cfg["dims"]
        for i in range(1, len(dims)):
            layers.append((f"fc{i}", "linear", M, dims[i], dims[i - 1], M * dims[i - 1],
                           M * dims[i], cfg["bias"], i > 1 and cfg["act"] != "none", None))
    elif cfg["kind"] == "vgg":
        B, s, c = cfg["batch"], cfg["image"], cfg["in_channels"]
        pooled = False
        for i, co in enumerate(cfg["channels"], start=1):
            pool = i in cfg["pool_after"]
            layers.append((f"conv{i}", "conv", B * s * s, co, 9 * c, B * s * s * c, B * s * s * co,
                           True, i > 1 and not pooled, B * s * s * co if pool else None))
            pooled = pool
            if pool:
                s //= 2
            c = co
        layers.append(("fc", "linear", B, cfg["classes"], c, B * c, B * cfg["classes"], True,
                       False, None))
    out = []
    for j, (name, lk, M, N, K, nin, nout, bias, act_prev, pool) in enumerate(layers):
        w, xb, yb = 4 * N * K, 4 * nin, 4 * nout
        bb = 4 * N if bias else 0
        f = 2 * M * N * K
        if lk == "linear":
            fwd_ff = (f, xb + yb + w * 2 + upd(N * K) + bb * 2 + (upd(N) if bias else 0))
        else:
            el = upd(N * K) + w + (upd(N) + bb if bias else 0)      # + R g
            fwd_ff = (f, xb + w + yb + bb + el)
        extra = 0
        if pool:                                           # fwd R y W p,arg; bwd R gp,arg,y W gz
            q = pool // 4
            extra = (4 * pool + 5 * q) + (4 * q + q + 4 * pool + 4 * pool)
        out.append(dict(
            name=name, kind=lk, M=M, N=N, K=K, nparams=N * K + (N if bias else 0),
            fwd=(f, xb + w + yb + bb),
            fwd_ff=fwd_ff,
            dgrad=(f, yb + w + xb + (xb if act_prev else 0)) if j > 0 else None,
            wgrad=(f, yb + xb + w + bb),
            wgrad_bf=(f, yb + xb + upd(N * K) + (upd(N) if bias else 0)),
            # merged data gradient + update: dZ, X, the state once, dX (+ the saved
            # tensor for the activation derivative)
            wgrad_bfm=((2 * f, yb + xb + upd(N * K) + (upd(N) if bias else 0) + xb
                        + (xb if act_prev else 0)) if j > 0 else
                       (f, yb + xb + upd(N * K) + (upd(N) if bias else 0))),
            extra=extra,
        ))
    return out


def tblock_launches(cfg):
    """Per-launch costs of the bf16 Transformer blocks.  Contractions take bf16
    operands: the weight is read as its 2-byte shadow, activations and
    gradients as fp32; the fused update also rewrites the shadow.  LayerNorm
    and the residual adds count as `extra` bytes of their block."""
    M, d, f, nb = cfg["batch"], cfg["hidden"], cfg["ffn"], cfg["blocks"]
    h = n_state(cfg["opt"])
    G = min(64, max(1, (M + 63) // 64))
    out = []
    for b in range(1, nb + 1):
        p = f"blk{b}."
        for name, N, K, act_prev, gelu in (("qkv", 3 * d, d, False, False),
                                           ("proj", d, d, False, False),
                                           ("fc1", f, d, False, True),
                                           ("fc2", d, f, True, False)):
            wb, xb, yb = 2 * N * K, 4 * M * K, 4 * M * N
            upd_w = 4 * N * K * (2 + 2 * h) + 2 * N * K
            upd_b = 4 * N * (2 + 2 * h)
            fl = 2 * M * N * K
            out.append(dict(
                name=p + name, kind="linear", M=M, N=N, K=K, nparams=N * K + N, dtype="bf16",
                fwd=(fl, xb + wb + yb * (2 if gelu else 1) + 4 * N),
                fwd_ff=(fl, xb + wb + yb * (2 if gelu else 1) + 4 * N + upd_w + 4 * N * K + upd_b),
                dgrad=(fl, yb + wb + xb + (xb if act_prev else 0)),
                wgrad=(fl, yb + xb + 4 * N * K + 4 * N),
                wgrad_bf=(fl, yb + xb + upd_w + upd_b),
                extra=0,
            ))
        for name in ("ln1", "ln2"):
            md = 4 * M * d
            # fwd R x W y, mean, rstd; bwd R dy, x, dres W dx (+ the parameter pass
            # R dy, x W 2 G d); residual add R 2 W 1
            extra = (2 * md + 8 * M) + (4 * md + 8 * M) + (2 * md + 8 * G * d) + 3 * md
            out.append(dict(name=p + name, kind="ln", M=M, N=d, K=0, nparams=2 * d, dtype="f32",
                            fwd=None, fwd_ff=None, dgrad=None, wgrad=None, wgrad_bf=None,
                            extra=extra))
    return out


def mbv2_launches(cfg):
    """Per-launch costs of the MobileNetV2-like network.  1x1 convolutions are
    linears over the pixel rows; a depthwise layer moves its input and output
    once per pass (fwd: R x W y; dgrad: R dy (+ the saved ReLU output) W dx;
    filter gradient: R dy, x, plus the slice partials) and does 2*9 flops per
    output element and pass.  Residual adds and the average pool count as
    `extra` bytes of the layer they follow (forward and backward)."""
    h = n_state(cfg["opt"])

    def upd(n):
        return 4 * n * (2 + 2 * h)

    B, H = cfg["batch"], cfg["image"]
    out = []

    def linear(name, M, N, K, act_prev, first=False, extra=0):
        w, xb, yb, bb = 4 * N * K, 4 * M * K, 4 * M * N, 4 * N
        f = 2 * M * N * K
        out.append(dict(
            name=name, kind="linear", M=M, N=N, K=K, nparams=N * K + N,
            fwd=(f, xb + w + yb + bb),
            fwd_ff=(f, xb + yb + w * 2 + upd(N * K) + bb * 2 + upd(N)),
            dgrad=None if first else (f, yb + w + xb + (xb if act_prev else 0)),
            wgrad=(f, yb + xb + w + bb),
            wgrad_bf=(f, yb + xb + upd(N * K) + upd(N)),
            extra=extra))

    c, s = cfg["stem"], H
    conv_in, conv_out = B * s * s * cfg["in_channels"], B * s * s * c
    out.append(dict(
        name="stem", kind="conv", M=B * s * s, N=c, K=9 * cfg["in_channels"],
        nparams=9 * cfg["in_channels"] * c + c,
        fwd=(2 * B * s * s * c * 9 * cfg["in_channels"], 4 * (conv_in + conv_out) + 4 * 9 * cfg["in_channels"] * c),
        fwd_ff=(2 * B * s * s * c * 9 * cfg["in_channels"], 4 * (conv_in + conv_out)
                + upd(9 * cfg["in_channels"] * c) + 4 * 9 * cfg["in_channels"] * c),
        dgrad=None,
        wgrad=(2 * B * s * s * c * 9 * cfg["in_channels"], 4 * (conv_in + conv_out)),
        wgrad_bf=(2 * B * s * s * c * 9 * cfg["in_channels"], 4 * (conv_in + conv_out)
                  + upd(9 * cfg["in_channels"] * c + c)),
        extra=0))
    k = 0
    cin, s = cfg["stem"], H
    for t, co, n, st in cfg["blocks"]:
        for r in range(n):
            k += 1
            stride = st if r == 0 else 1
            so = (s - 1) // stride + 1
            hid = t * cin
            p = f"blk{k}."
            if t != 1:
                linear(p + "expand", B * s * s, hid, cin, act_prev=k == 1)
            nin, nout = B * s * s * hid, B * so * so * hid
            dwf = 2 * 9 * nout
            out.append(dict(
                name=p + "dw", kind="dw", M=B * so * so, N=hid, K=9, nparams=10 * hid,
                fwd=(dwf, 4 * (nin + nout) + 40 * hid),
                fwd_ff=(dwf, 4 * (nin + nout) + 40 * hid + upd(10 * hid) + 40 * hid),
                dgrad=(dwf, 4 * (nout + 2 * nin) + 40 * hid),
                wgrad=(dwf, 4 * (nout + nin) + 40 * hid),
                wgrad_bf=(dwf, 4 * (nout + nin) + upd(10 * hid)),
                extra=0))
            res = stride == 1 and cin == co
            linear(p + "project", B * so * so, co, hid, act_prev=True,
                   extra=(3 + 3) * 4 * B * so * so * co if res else 0)
            cin, s = co, so
    linear("head", B * s * s, cfg["head"], cin, act_prev=False,
           extra=4 * (B * s * s * cfg["head"] + B * cfg["head"]) * 2)
    linear("fc", B, cfg["classes"], cfg["head"], act_prev=False)
    return out


def step_cost(cfg, ordering):
    """Whole-step algorithmic flops and bytes (kernels as implemented)."""
    L = layer_launches(cfg)
    F = B = 0
    for d in L:
        fk = "fwd_ff" if ordering == "ff" else "fwd"
        wk = {"bf": "wgrad_bf", "bfm": "wgrad_bfm"}.get(ordering, "wgrad")
        for k in ((fk, wk) if ordering == "bfm" else (fk, "dgrad", wk)):
            if d.get(k) is not None:
                F += d[k][0]
                B += d[k][1]
        B += d["extra"]
    n = sum(d["nparams"] for d in L)
    h = n_state(cfg["opt"])
    if ordering == "eager":
        B += n * 4 * (3 + 2 * h)           # R w, g, hist; W w, hist
    B += 4 * L[-1]["M"] * L[-1]["N"] * 2   # loss: R logits, W their gradient
    return F, B


def describe_layers(cfg):
    if cfg["kind"] == "mbv2":
        nb = sum(r[2] for r in cfg["blocks"])
        return (f"MobileNetV2-like: stem conv3x3 {cfg['stem']}, {nb} inverted-residual blocks "
                f"(1x1 expand, depthwise 3x3, 1x1 project), 1x1 head {cfg['head']}, avg-pool, "
                f"linear classifier; {cfg['image']}x{cfg['image']} input")
    if cfg["kind"] == "tblock":
        return (f"{cfg['blocks']} pre-LN blocks, hidden {cfg['hidden']}, FFN {cfg['ffn']}, "
                f"bf16 operands")
    if cfg["kind"] == "mlp":
        return f"{len(cfg['dims']) - 1} linear, width {cfg['dims'][1]}"
    return (f"{len(cfg['channels'])} conv3x3 ({','.join(map(str, cfg['channels']))}), "
            f"max-pool after {cfg['pool_after']}, linear classifier, {cfg['image']}x{cfg['image']}")


def mfma_peak(cfg):
    return PEAK_BF16_MFMA if cfg["dtype"] == "bf16" else PEAK_FP32_MFMA


def kernel_roofline(flops, nbytes, seconds, peak_mfma=PEAK_FP32_MFMA):
    t_hbm, t_mfma = nbytes / PEAK_HBM, flops / peak_mfma
    if t_hbm >= t_mfma:
        ach = nbytes / seconds / 1e9
        return dict(bound="hbm", achieved=round(ach, 1), peak=PEAK_HBM / 1e9, unit="GB/s",
                    frac=round(ach / (PEAK_HBM / 1e9), 4))
    ach = flops / seconds / 1e12
    return dict(bound="mfma", achieved=round(ach, 2), peak=peak_mfma / 1e12,
                unit="TFLOP/s", frac=round(ach / (peak_mfma / 1e12), 4))


def traffic_for(kernel_class, workload):
    """HBM bytes per launch measured by rocprofv3 counters, if recorded for the
    current kernel source (profiles/traffic.json keyed by the source hash)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    srcfile = "merged.hip" if kernel_class == "merged_bwd" else "gemm_f32.hip"
    src = os.path.join(ROOT, "paper_2104_00237_amd", "csrc", srcfile)
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
    merge = ordering == "bfm"
    if merge:
        ordering = "bf"
    prologue = ordering == "ffp"
    if prologue:
        ordering = "ff"
    tr = Trainer(cfg, make_params(cfg), "cuda:0", merge_dgrad=merge, conv_prologue=prologue,
                 linear_prologue=prologue)
    n = len(batches)
    for t in range(max(warmup, 1)):
        x, y = batches[t % n]
        tr.step(x, y, ordering)
    # events for the bracketed launches are made before the timed region (one
    # step's bracket count, measured on an extra untimed step, times the steps)
    timer = None
    if timer_classes:
        count = KernelTimer(timer_classes)
        tr.timer = count
        x, y = batches[max(warmup, 1) % n]
        tr.step(x, y, ordering)
        tr.timer = None
        per_step = sum(len(r) for r in count.records.values())
        timer = KernelTimer(timer_classes, pool=min(2 * per_step * (steps + 1) + 16, 60000))
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
    gc.collect()    # a collection now rather than inside the timed region
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


def median_step_ms(torch, cfg, ordering, batches, warmup, steps):
    """Median step time of one ordering, each launched step bracketed by its own
    event pair on the step's stream (a pass of its own, so the mean above is
    timed without per-step markers)."""
    from paper_2104_00237_amd.trainer import Trainer
    merge = ordering == "bfm"
    prologue = ordering == "ffp"
    o = "bf" if merge else "ff" if prologue else ordering
    tr = Trainer(cfg, make_params(cfg), "cuda:0", merge_dgrad=merge, conv_prologue=prologue,
                 linear_prologue=prologue)
    n = len(batches)
    for t in range(max(warmup, 1)):
        tr.step(*batches[t % n], o)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    evs[0].record(tr.stream)
    for t in range(steps):
        tr.step(*batches[(warmup + t) % n], o)
        evs[t + 1].record(tr.stream)
    torch.cuda.synchronize()
    return float(np.median([evs[t].elapsed_time(evs[t + 1]) for t in range(steps)]))


STAGES = {"forward": ("fwd", "fwd_ff", "loss"),
          "backward": ("dgrad", "wgrad", "wgrad_bf", "ln_bwd", "add"),
          "optimizer": ("opt", "clip")}


def stage_breakdown(torch, cfg, batches, ordering, steps, marker_ms):
    """Fig. 3-style split of one ordering's step into forward, backward and
    optimizer kernel time (ms per step): every launch class bracketed by events
    on its own stream, the event pair's cost taken off each launch.  Kernels
    that overlap on two streams (backward-fusion's updates) are both counted, so
    the stages can sum to more than the step."""
    classes = [c for cs in STAGES.values() for c in cs]
    ms, _, timer, _ = time_ordering(torch, cfg, ordering, batches, 3, steps, classes)
    out = {}
    for stage, cs in STAGES.items():
        tot = 0.0
        for c in cs:
            durs = timer.durations(c)
            tot += sum(max(d - marker_ms, 0.0) for d, _ in durs)
        out[stage] = round(tot / steps, 4)
    out["step_bracketed"] = round(ms, 4)
    return out


# MobileNetV2's 17 depthwise 3x3 layers (H = W, C) at their output resolution; the
# stride-2 ones are taken at stride 1 on their output size (the kernels are stride 1).
MBV2_DEPTHWISE = [(112, 32), (56, 96), (56, 144), (28, 144), (28, 192), (28, 192), (14, 192),
                  (14, 384), (14, 384), (14, 384), (14, 384), (14, 576), (14, 576), (7, 576),
                  (7, 960), (7, 960), (7, 960)]


def depthwise_stack(torch, batch, steps, warmup):
    """Backward of MobileNetV2's depthwise layers (batch 32, SGD with momentum): eager
    (data gradient, filter gradient written, one multi-tensor optimizer launch over all
    filters and biases) against backward-fusion (data gradient, filter gradient whose
    reduction applies the update), plus the forward's HBM rate.  Returns milliseconds
    per pass over the 17 layers."""
    from paper_2104_00237_amd import _lib as L
    dev = "cuda:0"
    hyper = dict(kind="sgd", lr=0.05, momentum=0.9, weight_decay=4e-5)
    g = torch.Generator(device=dev).manual_seed(0)
    layers = []
    for hw, c in MBV2_DEPTHWISE:
        d = L.OfConvDesc(batch, hw, hw, c, c, L.OF_ACT_RELU, 1)
        t = dict(d=d, x=torch.randn((batch, hw, hw, c), device=dev, generator=g),
                 dy=torch.randn((batch, hw, hw, c), device=dev, generator=g) * 0.1)
        t["y"], t["dx"] = torch.empty_like(t["x"]), torch.empty_like(t["x"])
        t["ws"] = torch.empty(max(4, L.of_dwconv_workspace_size(d) // 4), device=dev)
        for nm, shape in (("W", (3, 3, c)), ("b", (c,))):
            w, m = torch.randn(shape, device=dev, generator=g) * 0.1, torch.zeros(shape, device=dev)
            t[nm] = (w, m, L.OfParam(w.data_ptr(), m.data_ptr(), None, None, w.numel()),
                     torch.empty(shape, device=dev))
        layers.append(t)
    s = torch.cuda.current_stream().cuda_stream
    opt = L.make_opt(hyper, 1)

    def fwd():
        for t in layers:
            L.of_dwconv_fwd(t["d"], t["x"].data_ptr(), t["W"][0].data_ptr(), t["b"][0].data_ptr(),
                            t["y"].data_ptr(), s)

    def eager():
        for t in layers:
            L.of_dwconv_bwd_data(t["d"], t["dy"].data_ptr(), t["W"][0].data_ptr(),
                                 t["x"].data_ptr(), L.OF_ACT_RELU, t["dx"].data_ptr(), s)
            L.of_dwconv_bwd_weight(t["d"], t["dy"].data_ptr(), t["x"].data_ptr(),
                                   t["W"][3].data_ptr(), t["b"][3].data_ptr(), 0,
                                   t["ws"].data_ptr(), t["ws"].numel() * 4, s)
        ps = [t[k][2] for t in layers for k in ("W", "b")]
        gs = [t[k][3].data_ptr() for t in layers for k in ("W", "b")]
        L.of_optimizer_step(len(ps), (L.OfParam * len(ps))(*ps), (L.c_void_p * len(gs))(*gs),
                            opt, s)

    def bf():
        for t in layers:
            L.of_dwconv_bwd_data(t["d"], t["dy"].data_ptr(), t["W"][0].data_ptr(),
                                 t["x"].data_ptr(), L.OF_ACT_RELU, t["dx"].data_ptr(), s)
            L.of_dwconv_wgrad_fused(t["d"], t["dy"].data_ptr(), t["x"].data_ptr(), t["W"][2],
                                    t["b"][2], None, None, opt, t["ws"].data_ptr(),
                                    t["ws"].numel() * 4, s)

    res = {}
    for name, fn in (("forward", fwd), ("eager_backward", eager), ("bf_backward", bf)):
        for _ in range(warmup):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        res[name] = e0.elapsed_time(e1) / steps
    act_bytes = sum(2 * batch * hw * hw * c * 4 for hw, c in MBV2_DEPTHWISE)
    n_params = sum(10 * c for _, c in MBV2_DEPTHWISE)
    return {"layers": len(MBV2_DEPTHWISE), "batch": batch, "params": n_params,
            "optimizer": "sgd_momentum",
            **{k + "_ms": round(v, 4) for k, v in res.items()},
            "bf_speedup_backward": round(res["eager_backward"] / res["bf_backward"], 3),
            "forward_GBps": round(act_bytes / (res["forward"] * 1e-3) / 1e9, 1)}


def hbm_ceiling(torch, nbytes=1 << 30, reps=20):
    """Read, copy and in-place read-modify-write rates of the library's
    streaming kernels over `nbytes` (copy and read-modify-write: nbytes read and
    nbytes written; rmw3: three arrays of a third each, updated side by side as
    W, m and v are), GB/s of bytes moved: the best over launches of 2048, 16384
    and 65535 workgroups (measured on MI355X: many short-lived workgroups
    reach 6.1 TB/s read-modify-write where 2048 grid-striding ones reach 5.4).
    rmw3_columns: three 8192 x 8192 arrays in the merged backward kernel's
    4-byte column layout and grid (its own streaming ceiling)."""
    from paper_2104_00237_amd import _lib as L
    n = nbytes // 4
    src = torch.ones(n, device="cuda:0")
    dst = torch.empty_like(src)
    s = torch.cuda.current_stream()
    out = {}
    n3 = n // 12 * 12
    chunk = 3 * 8192 * 32
    ncol = min(3 * 8192 * 8192, n // chunk * chunk)
    for name, mode, cnt, moved in (("read_GBps", L.OF_STREAM_READ, n, nbytes),
                                   ("copy_GBps", L.OF_STREAM_COPY, n, 2 * nbytes),
                                   ("rmw_GBps", L.OF_STREAM_RMW, n, 2 * nbytes),
                                   ("rmw3_GBps", L.OF_STREAM_RMW3, n3, 8 * n3),
                                   ("rmw3_columns_GBps", L.OF_STREAM_RMW3_COLUMNS, ncol, 8 * ncol)):
        if cnt <= 0:
            continue
        best = 0.0
        for blocks in ((0,) if mode == L.OF_STREAM_RMW3_COLUMNS else (2048, 16384, 65535)):
            for _ in range(3):
                L.of_hbm_stream(mode, src.data_ptr(), dst.data_ptr(), cnt, blocks, s.cuda_stream)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            for _ in range(reps):
                L.of_hbm_stream(mode, src.data_ptr(), dst.data_ptr(), cnt, blocks, s.cuda_stream)
            e1.record(s)
            torch.cuda.synchronize()
            best = max(best, moved * reps / (e0.elapsed_time(e1) / 1e3) / 1e9)
        out[name] = round(best, 1)
    out["bytes"] = nbytes
    del src, dst
    torch.cuda.empty_cache()
    return out


def extra_workload(torch, name, steps, warmup):
    """Eager, forward- and backward-fusion step times of another workload."""
    cfg = get_config(name)
    dev = torch.device("cuda:0")
    batches = []
    for t in range(1, 5):
        x, y = make_batch(cfg, t)
        batches.append((torch.as_tensor(x).to(dev), torch.as_tensor(y).to(dev)))
    mergeable = cfg["kind"] == "mlp" and cfg["dtype"] == "f32" and cfg["batch"] <= 64
    # forward-fusion in the weight-tile prologue with a second buffer set
    # (fp32 layers of more than 64 rows)
    prologue = cfg["dtype"] == "f32" and cfg["batch"] > 64
    res = {}
    for o in ("eager", "ff", "bf") + (("bfm",) if mergeable else ()) + (("ffp",) if prologue else ()):
        ms, _, _, _ = time_ordering(torch, cfg, o, batches, warmup, steps, graph=False)
        res[f"{o}_ms_per_step"] = round(ms, 4)
        print(f"[bench] {name} {o}: {ms:.4f} ms/step", file=sys.stderr, flush=True)
    for o in ("ff", "bf") + (("bfm",) if mergeable else ()) + (("ffp",) if prologue else ()):
        res[f"speedup_{o}_vs_eager"] = round(res["eager_ms_per_step"] / res[f"{o}_ms_per_step"], 4)
    res["global_batch"] = cfg["batch"]
    res["layers"] = describe_layers(cfg)
    res["optimizer"] = cfg["opt"]["kind"]
    return res


def cpu_baseline(cfg, budget_s=15.0):
    """Oracle eager steps on this host, seconds per step of `cfg`.  The 12-block
    Transformer stack is sampled as one block (same width and tokens) and its
    time scaled by the block count."""
    import oracle
    from oracle.train import new_model
    scale = 1
    if cfg["kind"] == "tblock":
        scale = cfg["blocks"]
        cfg = dict(cfg, blocks=1)
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
    dt = (time.perf_counter() - t0) / n * scale
    del oracle
    return dt, n


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="linear4x8192")
    ap.add_argument("--extra-workloads", default="mlp8x1024",
                    help="comma-separated workloads timed beside the main one (eager, ff, bf; "
                         "'' for none)")
    ap.add_argument("--optimizer", choices=sorted(FIG7_OPTIMIZERS), default=None,
                    help="replace the workload's optimizer (Fig. 7's set)")
    ap.add_argument("--batch", type=int, default=None,
                    help="replace the workload's batch (rows per step; Figs. 4-5 sweep)")
    ap.add_argument("--dims", default=None, metavar="WIDTHxDEPTH",
                    help="MLP workloads: DEPTH hidden layers of WIDTH (parameters per layer, "
                         "Fig. 6 sweep); the input and output widths follow WIDTH and the classes")
    ap.add_argument("--ff-prologue", "--conv-ff-prologue", dest="ff_prologue",
                    action="store_true",
                    help="also time forward-fusion with every update in its own forward's "
                         "weight-tile prologue (ffp: convolutions and linear layers of more "
                         "than 64 rows write a second buffer set)")
    ap.add_argument("--depthwise", action="store_true",
                    help="also time MobileNetV2's depthwise 3x3 layers (batch 32): eager "
                         "vs backward-fusion backward, and the forward's HBM rate")
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
    if args.optimizer:
        cfg = dict(cfg, opt=FIG7_OPTIMIZERS[args.optimizer])
    if args.batch:
        cfg = dict(cfg, batch=args.batch)
    if args.dims:
        if cfg["kind"] != "mlp":
            print("--dims applies to MLP workloads", file=sys.stderr)
            sys.exit(2)
        w, dpt = (int(v) for v in args.dims.lower().split("x"))
        out = cfg["classes"] if cfg["loss"] == "xent" else w
        cfg = dict(cfg, dims=[w] * (dpt + 1) + ([out] if cfg["loss"] == "xent" else []))
    if cfg["kind"] not in ("mlp", "vgg", "tblock", "mbv2"):
        print(f"workload {args.workload} has no GPU path in this build", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    nb = 4
    batches = []
    for t in range(1, nb + 1):
        x, y = make_batch(cfg, t)
        batches.append((torch.as_tensor(x).to(dev), torch.as_tensor(y).to(dev)))
    torch.cuda.synchronize()

    # the merged backward applies to fp32 linear chains of at most 64 rows
    mergeable = cfg["kind"] == "mlp" and cfg["dtype"] == "f32" and cfg["batch"] <= 64
    res = {}
    extra = (("bfm",) if mergeable else ()) + (("ffp",) if args.ff_prologue else ())
    for o in ("eager", "ff", "bf") + extra:
        ms, host_ms, _, _ = time_ordering(torch, cfg, o, batches, args.warmup, args.steps,
                                          graph=False)
        ms_g = None
        if not args.no_graph:
            ms_g, _, _, _ = time_ordering(torch, cfg, o, batches, args.warmup, args.steps,
                                          graph=True)
        res[o] = dict(ms=ms, host_ms=host_ms, ms_graph=ms_g)
        print(f"[bench] {o}: {ms:.4f} ms/step launched (host {host_ms:.4f}), "
              f"graph replay {ms_g} ms/step", file=sys.stderr, flush=True)

    # The headline backward-fusion variant: the faster one.
    head = "bfm" if mergeable and res["bfm"]["ms"] < res["bf"]["ms"] else "bf"
    # Dominant kernel of the fused step: one instrumented pass finds the class
    # with the largest total time; the timed pass then brackets only that class
    # (bfm brackets each layer's merged pass -- its kernel and the data-gradient
    # sum -- as wgrad_bf).
    classes = ("fwd", "dgrad", "wgrad_bf", "loss")
    _, _, probe, _ = time_ordering(torch, cfg, head, batches, 2, 3, classes)
    totals = {c: sum(d for d, _ in probe.durations(c)) for c in classes}
    dom = max(totals, key=totals.get)
    print("[bench] launch-class totals (ms over the probe steps): " +
          ", ".join(f"{c} {t:.3f}" for c, t in totals.items()), file=sys.stderr, flush=True)
    ms_dom_step, _, timer, _ = time_ordering(torch, cfg, head, batches, args.warmup, args.steps,
                                             (dom,))
    cost_key = "wgrad_bfm" if (head == "bfm" and dom == "wgrad_bf") else dom
    launches = {d["name"]: d for d in layer_launches(cfg)}
    recs = timer.durations(dom)
    # Group launches by layer shape (the repeated hidden layers of an MLP share
    # one) and report the group with the largest total time.
    by_shape = {}
    for d_ms, op in recs:
        if op is not None:
            by_shape.setdefault((op.kind, op.M, op.N, op.K), []).append((d_ms, op.name, op))
    costed = [k for k in by_shape if launches[by_shape[k][0][1]].get(cost_key)]
    shape = max(costed, key=lambda s: sum(d for d, _, _ in by_shape[s]))
    if cost_key == "wgrad_bfm":
        # the first layer has no data gradient: its merged pass is the plain update
        grp = [(d, n, o) for d, n, o in by_shape[shape] if launches[n]["dgrad"] is not None]
        by_shape[shape] = grp or by_shape[shape]
    durs = [d for d, _, _ in by_shape[shape]]
    per = launches[by_shape[shape][0][1]][cost_key]
    # Each launch is bracketed by an event pair on its own stream; the pair's own
    # cost (an empty pair on the same stream) is taken off.
    from paper_2104_00237_amd.trainer import KernelTimer, device_stream
    on_side = (dom == "wgrad_bf" and head == "bf"
               and getattr(by_shape[shape][0][2], "overlap_update", False))
    dom_stream = (device_stream(torch.device("cuda:0"), "side") if on_side
                  else torch.cuda.current_stream())
    marker_ms = KernelTimer.marker_overhead_ms(dom_stream)
    avg_s = (float(np.mean(durs)) - marker_ms) / 1e3
    roof = kernel_roofline(per[0], per[1], avg_s, mfma_peak(cfg))
    roof.update(kernel=("merged_bwd" if cost_key == "wgrad_bfm" else dom),
                layers=sorted({n for _, n, _ in by_shape[shape]}),
                shape=f"{shape[0]} GEMM M={shape[1]} N={shape[2]} K={shape[3]}",
                avg_us=round(avg_s * 1e6, 3), launches=len(durs),
                bracketed_avg_us=round(float(np.mean(durs)) * 1e3, 3),
                marker_us=round(marker_ms * 1e3, 3),
                algorithmic_bytes=per[1], algorithmic_flops=per[0],
                traffic=traffic_for("merged_bwd" if cost_key == "wgrad_bfm" else dom,
                                    args.workload))

    medians = {o: round(median_step_ms(torch, cfg, o, batches, args.warmup, args.steps), 4)
               for o in res}
    # Fig. 3 analogue: forward / backward / optimizer kernel time of each ordering
    main_marker = KernelTimer.marker_overhead_ms(torch.cuda.current_stream())
    breakdown = {o: stage_breakdown(torch, cfg, batches, o, 10, main_marker) for o in res}

    n_params = sum(d["nparams"] for d in launches.values())
    kind = cfg["opt"]["kind"]
    nst = n_state(cfg["opt"])
    upd_bytes = n_params * state_bytes_per_param(nst, head)
    bf_s = res[head]["ms"] / 1e3
    value = upd_bytes / bf_s / 1e9
    F, B = step_cost(cfg, head)
    step_roof_s = max(B / PEAK_HBM, F / mfma_peak(cfg))

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(res[head]["ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg["dtype"] == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "global_batch": cfg["batch"],
                   "layers": describe_layers(cfg),
                   "optimizer": args.optimizer or kind,
                   "ordering": ("backward-fusion, data gradient merged into the update"
                                if head == "bfm" else "backward-fusion"),
                   "parallelism": "single-gpu"},
        "eager_ms_per_step": round(res["eager"]["ms"], 4),
        "ff_ms_per_step": round(res["ff"]["ms"], 4),
        "bf_ms_per_step": round(res["bf"]["ms"], 4),
        "speedup_bf_vs_eager": round(res["eager"]["ms"] / res["bf"]["ms"], 4),
        "speedup_ff_vs_eager": round(res["eager"]["ms"] / res["ff"]["ms"], 4),
        **({"ffp_ms_per_step": round(res["ffp"]["ms"], 4),
            "speedup_ffp_vs_eager": round(res["eager"]["ms"] / res["ffp"]["ms"], 4)}
           if "ffp" in res else {}),
        **({"bfm_ms_per_step": round(res["bfm"]["ms"], 4),
            "speedup_bfm_vs_eager": round(res["eager"]["ms"] / res["bfm"]["ms"], 4)}
           if mergeable else {}),
        "ms_per_step_graph_replay": {o: (round(r["ms_graph"], 4) if r["ms_graph"] else None)
                                     for o, r in res.items()},
        "host_ms_per_step": {o: round(r["host_ms"], 4) for o, r in res.items()},
        "median_ms_per_step": medians,
        "timing": "steps launched from the host scheduler; graph replay reported beside",
        "step_roofline": {"flops": F, "bytes": B, "roofline_ms": round(step_roof_s * 1e3, 5),
                          "frac": round(step_roof_s / bf_s, 4)},
        "update_bytes_per_step": {o: n_params * state_bytes_per_param(nst, o) for o in res},
        "roofline": roof,
        "stage_breakdown_ms": breakdown,
        "optimizer_share_eager": round(breakdown["eager"]["optimizer"] / res["eager"]["ms"], 4),
        # the separate optimizer pass alone: R w, g, state and W w, state per parameter
        "eager_optimizer_GBps": (round(n_params * 4 * (3 + 2 * nst) /
                                       (breakdown["eager"]["optimizer"] / 1e3) / 1e9, 1)
                                 if breakdown["eager"]["optimizer"] > 0 else None),
        "tflops_per_s": round(F / bf_s / 1e12, 3),
        # the speedup model's inputs (Section 4): t_opt of the eager step and, per
        # fused ordering, t_saved = eager - fused step time and the share of t_opt saved
        "t_opt_ms": breakdown["eager"]["optimizer"],
        "t_saved_ms": {o: round(res["eager"]["ms"] - res[o]["ms"], 4) for o in res if o != "eager"},
        "t_opt_saved_frac": ({o: round((res["eager"]["ms"] - res[o]["ms"]) /
                                       breakdown["eager"]["optimizer"], 3)
                              for o in res if o != "eager"}
                             if breakdown["eager"]["optimizer"] > 0 else None),
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
        eager_bytes = n_params * state_bytes_per_param(nst, "eager")
        out["cpu_baseline"] = {"value": round(eager_bytes / dt / 1e9, 4), "unit": "GB/s",
                               "cores": cores, "kind": "oracle",
                               "ms_per_step": round(dt * 1e3, 2),
                               "sample": f"{n} eager float64 steps of {args.workload}"
                                         + (" (one of its blocks, time x blocks)"
                                            if cfg["kind"] == "tblock" else "")
                                         + f" (oracle, numpy, {cores} host threads)"}
    ceil = hbm_ceiling(torch)
    out["hbm_ceiling"] = ceil
    if roof["bound"] == "hbm":
        roof["frac_of_measured_copy_rate"] = round(roof["achieved"] / ceil["copy_GBps"], 4)
        roof["frac_of_measured_rmw_rate"] = round(roof["achieved"] / ceil["rmw_GBps"], 4)
        roof["frac_of_measured_rmw3_rate"] = round(roof["achieved"] / ceil["rmw3_GBps"], 4)
        if "rmw3_columns_GBps" in ceil:
            roof["frac_of_measured_rmw3_columns_rate"] = round(
                roof["achieved"] / ceil["rmw3_columns_GBps"], 4)
    for name in [w for w in args.extra_workloads.split(",") if w and w != args.workload]:
        out.setdefault("extra_workloads", {})[name] = extra_workload(torch, name, args.steps,
                                                                     args.warmup)
    if args.depthwise:
        out["depthwise_mbv2"] = depthwise_stack(torch, 32, args.steps, args.warmup)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
