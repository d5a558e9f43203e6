"""Whole training trajectories of the oracle pinned to an independent float64
implementation: the same models written with torch's autograd (gradients) and
torch.optim's single-tensor optimizers (updates), trained on the same seeded
initial parameters and batches (the shared generators in workloads/).

The oracle computes every gradient with its own hand-written backward and its
own optimizer code, so agreement over K steps pins both, and, through the
ordering invariant (eager == forward-fusion flushed == backward-fusion bit for
bit, tests/test_oracle_orderings.py), every ordering's trajectory.  Float64 on
both sides: the two differ only by summation order (~1e-15 relative per step).

Covered, on every model family: linear, ReLU, cross-entropy and MSE; 3x3
convolution, 2x2 max-pool, flatten; depthwise 3x3 convolution (stride 1 and
2), 1x1 convolutions over pixel rows, inverted-residual additions, global
average pooling; LayerNorm, GELU, the V third of a fused QKV projection,
pre-LN residual blocks with bf16 matmul operands; SGD-momentum and Adam with
coupled weight decay, AdamW; and a layer applied twice (mlp4tied: one update
from the sum of both uses' gradients).

bf16 operands (the transformer block's matmuls; the paper itself trains in
float32): both matmul operands, and the output gradient entering the two
backward products, rounded to the nearest bfloat16 (ties to even) while the
bias gradient sums the unrounded output gradient.  The rounding here works on
the float64 bit pattern (the oracle scales by a power of two and rounds), so
the two implementations share no code.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from workloads import (get_config, reduced_config, make_params, make_batch, mlp_ties,
                       mbv2_blocks)

TOL = 1e-9


def _optimizer(cfg, params):
    h = cfg["opt"]
    if h["kind"] == "sgd":
        return torch.optim.SGD(params, lr=h["lr"], momentum=h["momentum"],
                               weight_decay=h["weight_decay"], foreach=False)
    if h["kind"] == "adam":
        return torch.optim.Adam(params, lr=h["lr"], betas=(h["beta1"], h["beta2"]), eps=h["eps"],
                                weight_decay=h.get("weight_decay", 0.0), foreach=False)
    if h["kind"] == "adamw":
        return torch.optim.AdamW(params, lr=h["lr"], betas=(h["beta1"], h["beta2"]), eps=h["eps"],
                                 weight_decay=h["weight_decay"], foreach=False)
    raise ValueError(h["kind"])


def _mlp_forward(cfg, P, x):
    n_layers = len(cfg["dims"]) - 1
    tie = mlp_ties(cfg)
    h = x
    for i in range(1, n_layers + 1):
        j = tie.get(i, i)          # a tied layer applies another layer's parameters
        h = h @ P[f"fc{j}.weight"].T
        if cfg["bias"]:
            h = h + P[f"fc{j}.bias"]
        if i < n_layers and cfg["act"] == "relu":
            h = torch.relu(h)
    return h


_KEEP = 52 - 7                  # float64 mantissa bits below bfloat16's 7 stored ones


def _bf16_bits(t):
    """Nearest bfloat16 value of float64 `t` (ties to even), by integer
    arithmetic on the bit pattern: add just under half a unit of the last kept
    place plus that place's bit, then clear the dropped bits.  Normal bfloat16
    range only (asserted)."""
    t = t.detach().contiguous()
    a = t.abs()
    assert bool(torch.all(torch.isfinite(t))) and bool(torch.all((a == 0) | (a >= 2.0 ** -126)))
    i = t.view(torch.int64)
    lsb = (i >> _KEEP) & 1
    i = (i + ((1 << (_KEEP - 1)) - 1) + lsb) & ~((1 << _KEEP) - 1)
    out = i.view(torch.float64)
    assert bool(torch.all(out.abs() < 2.0 ** 128))
    return out


class _Bf16Linear(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w, b):
        xq, wq = _bf16_bits(x), _bf16_bits(w)
        ctx.save_for_backward(xq, wq)
        return xq @ wq.T + b

    @staticmethod
    def backward(ctx, dz):
        xq, wq = ctx.saved_tensors
        dzq = _bf16_bits(dz)
        return dzq @ wq, dzq.T @ xq, dz.sum(0)


def _tblock_forward(cfg, P, x):
    d = cfg["hidden"]
    assert cfg["dtype"] == "bf16"

    def lin(name, h):
        return _Bf16Linear.apply(h, P[name + ".weight"], P[name + ".bias"])

    def ln(name, h):
        return F.layer_norm(h, (d,), P[name + ".weight"], P[name + ".bias"], cfg["ln_eps"])

    for b in range(1, cfg["blocks"] + 1):
        p = f"blk{b}."
        v = lin(p + "qkv", ln(p + "ln1", x))[:, 2 * d:3 * d]
        h = x + lin(p + "proj", v)
        x = h + lin(p + "fc2", F.gelu(lin(p + "fc1", ln(p + "ln2", h))))
    return x


def _mbv2_forward(cfg, P, x):
    def pointwise(name, h):        # a 1x1 convolution, NCHW
        w = P[name + ".weight"]
        return F.conv2d(h, w[:, :, None, None], P[name + ".bias"])

    stem = P["stem.weight"].permute(0, 3, 1, 2)
    h = torch.relu(F.conv2d(x.permute(0, 3, 1, 2), stem, P["stem.bias"], padding=1))
    for b in mbv2_blocks(cfg):
        p, x_in = b["name"], h
        if b["t"] != 1:
            h = torch.relu(pointwise(p + "expand", h))
        dw = P[p + "dw.weight"].permute(2, 0, 1)[:, None]   # [3,3,C] -> [C,1,3,3]
        h = torch.relu(F.conv2d(h, dw, P[p + "dw.bias"], stride=b["stride"], padding=1,
                                groups=dw.shape[0]))
        h = pointwise(p + "project", h)
        if b["residual"]:
            h = h + x_in
    h = torch.relu(pointwise("head", h)).mean(dim=(2, 3))
    return h @ P["fc.weight"].T + P["fc.bias"]


def _vgg_forward(cfg, P, x):
    h = x.permute(0, 3, 1, 2)      # NHWC -> NCHW
    for i in range(1, len(cfg["channels"]) + 1):
        w = P[f"conv{i}.weight"].permute(0, 3, 1, 2)   # [Cout,3,3,Cin] -> [Cout,Cin,3,3]
        h = torch.relu(F.conv2d(h, w, P[f"conv{i}.bias"], padding=1))
        if i in cfg["pool_after"]:
            h = F.max_pool2d(h, 2)
    h = h.permute(0, 2, 3, 1).reshape(h.shape[0], -1)   # flatten in NHWC order
    return h @ P["fc.weight"].T + P["fc.bias"]


def _torch_run(cfg, forward, steps):
    P = {k: torch.tensor(np.asarray(v, np.float64), requires_grad=True)
         for k, v in make_params(cfg).items()}
    opt = _optimizer(cfg, list(P.values()))
    losses = []
    for t in range(1, steps + 1):
        x, y = make_batch(cfg, t)
        z = forward(cfg, P, torch.tensor(np.asarray(x, np.float64)))
        if cfg["loss"] == "xent":
            loss = F.cross_entropy(z, torch.tensor(y))
        else:
            loss = F.mse_loss(z, torch.tensor(np.asarray(y, np.float64)))
        opt.zero_grad(set_to_none=True)
        loss.backward()
        opt.step()
        losses.append(float(loss.detach()))
    return np.array(losses), {k: v.detach().numpy() for k, v in P.items()}


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(float(np.max(np.abs(b))), 1e-300))


@pytest.mark.parametrize("name,how,forward", [
    ("mlp3", "full", _mlp_forward),
    ("mlp4tied", "full", _mlp_forward),
    ("mlp8x1024", "reduced", _mlp_forward),
    ("vgg11", "reduced", _vgg_forward),
    ("linear4x8192", "reduced", _mlp_forward),
    ("mbv2", "reduced", _mbv2_forward),
    ("tblock12", "reduced", _tblock_forward),
])
def test_trajectory_matches_torch_autograd(name, how, forward):
    torch.set_num_threads(4)
    cfg = get_config(name) if how == "full" else reduced_config(name)
    steps = cfg["steps"]
    ref = oracle.run(cfg, "eager", steps=steps)
    losses, params = _torch_run(cfg, forward, steps)
    assert _rel(ref["losses"], losses) <= TOL, (ref["losses"], losses)
    assert set(params) == set(ref["params"])
    for k in params:
        r = _rel(ref["params"][k], params[k])
        assert r <= TOL, f"{name} {k}: rel {r:.2e}"
        # and the trajectory actually moved the tensor
        assert np.max(np.abs(params[k] - make_params(cfg)[k])) > 0.0
