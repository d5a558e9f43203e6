"""The synthetic training workloads, as data.

Each workload is a dict with:
  kind      "mlp" | "tblock" | "vgg" | "mbv2"  (model family)
  batch     rows per mini-batch (tokens for "tblock", images for "vgg")
  loss      "xent" (softmax cross-entropy, int64 labels) | "mse"
  opt       optimizer kind and hyperparameters
  steps     training steps K
  dtype     "f32" | "bf16" (the precision of every matmul operand)

Model families:
  mlp     dims [d0..dL]: L linear layers d_{i-1} -> d_i, activation `act` after
          every layer but the last, bias if `bias`.
  tblock  `blocks` pre-LayerNorm residual blocks of width `hidden`:
              h = x + OutProj(V(QKV(LN1(x))))     (attention replaced by identity,
                                                    so the context is the V third)
              y = h + FC2(GELU(FC1(LN2(h))))
  vgg     3x3 convolutions (stride 1, zero pad 1, bias, ReLU) with output
          channels `channels`; a 2x2 max-pool after the convolutions listed in
          `pool_after` (1-based); a final linear classifier on the 1x1 map.
  mbv2    MobileNetV2-like: a 3x3 stem convolution (stride 1, bias, ReLU) with
          `stem` output channels, then inverted-residual blocks from the rows
          (t, c, n, s) of `blocks` (n blocks of c output channels, the first
          with stride s, the rest stride 1; expansion t):
              1x1 expand to t * c_in channels (a linear over the N*H*W pixel
                  rows, bias, ReLU; absent when t == 1),
              3x3 depthwise convolution (stride s, zero pad 1, bias, ReLU),
              1x1 project to c channels (linear over pixel rows, bias, no
                  activation),
              + the block input when the stride is 1 and c_in == c;
          then a 1x1 convolution to `head` channels (bias, ReLU), the global
          average over the spatial positions and a linear classifier.  ReLU
          stands in for MobileNetV2's ReLU6 and there is no batch normalisation
          (as in vgg).

Layouts (shared by both sides): activations are row-major [rows, features];
images are NHWC; a linear weight is [out, in]; a conv filter is
[Cout, 3, 3, Cin].
"""
import copy

CONFIGS = {
    # 3-layer MLP, SGD with momentum: the small case every ordering is checked on.
    "mlp3": dict(
        kind="mlp", dims=[64, 128, 128, 10], act="relu", bias=True,
        batch=32, loss="xent", classes=10, dtype="f32", steps=5,
        opt=dict(kind="sgd", lr=0.01, momentum=0.9, weight_decay=1e-4),
    ),
    # 8-layer MLP of width 1024, Adam; bias updates take the elementwise path.
    "mlp8x1024": dict(
        kind="mlp", dims=[1024] * 8 + [10], act="relu", bias=True,
        batch=256, loss="xent", classes=10, dtype="f32", steps=20,
        opt=dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                 weight_decay=0.0),
    ),
    # 12 transformer-block linear stacks, bf16 matmul operands, fp32 AdamW state.
    "tblock12": dict(
        kind="tblock", blocks=12, hidden=1024, ffn=4096, batch=4096,
        loss="mse", dtype="bf16", steps=10,
        opt=dict(kind="adamw", lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8,
                 weight_decay=0.01),
        ln_eps=1e-5,
    ),
    # VGG-11-style convolution stack on 32x32x3 images, SGD with momentum.
    "vgg11": dict(
        kind="vgg", channels=[64, 128, 256, 256, 512, 512, 512, 512],
        pool_after=[1, 2, 4, 6, 8], image=32, in_channels=3, batch=128,
        loss="xent", classes=10, dtype="f32", steps=10,
        opt=dict(kind="sgd", lr=0.1, momentum=0.9, weight_decay=5e-4),
    ),
    # A parameter used twice in one step (Alg. 2's `updated` flag, Alg. 3's
    # `count`): layer 3 applies layer 2's weight and bias again.
    "mlp4tied": dict(
        kind="mlp", dims=[64, 128, 128, 128, 10], act="relu", bias=True, tie={3: 2},
        batch=32, loss="xent", classes=10, dtype="f32", steps=5,
        opt=dict(kind="sgd", lr=0.01, momentum=0.9, weight_decay=1e-4),
    ),
    # MobileNetV2-like network (the paper's Fig. 3 / Table 2 model) with its
    # ImageNet layer shapes: the rows of MobileNetV2's block table, a 112x112
    # input to a stride-1 stem standing in for its stride-2 stem on 224x224
    # images, batch 32 (as in Fig. 3), Adam with coupled weight decay
    # (PyTorch 1.6's Adam(weight_decay=...), the framework the paper's
    # implementation uses).
    "mbv2": dict(
        kind="mbv2", image=112, in_channels=3, stem=32,
        blocks=[[1, 16, 1, 1], [6, 24, 2, 2], [6, 32, 3, 2], [6, 64, 4, 2], [6, 96, 3, 1],
                [6, 160, 3, 2], [6, 320, 1, 1]],
        head=1280, batch=32, loss="xent", classes=10, dtype="f32", steps=10,
        opt=dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                 weight_decay=4e-5),
    ),
    # Parameter-bound stack: 4 linear layers 8192x8192, no bias, no activation.
    "linear4x8192": dict(
        kind="mlp", dims=[8192] * 5, act="none", bias=False,
        batch=64, loss="mse", dtype="f32", steps=10,
        opt=dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                 weight_decay=0.0),
    ),
}

# Reduced versions of the same families, for checks the CPU oracle finishes in
# seconds.  Sizes are chosen to span several GPU tiles and leave ragged tails.
_REDUCED = {
    "mlp3": {},
    "mlp4tied": {},
    "mlp8x1024": dict(dims=[200, 168, 168, 168, 10], batch=72, steps=4),
    "tblock12": dict(blocks=2, hidden=96, ffn=160, batch=136, steps=3),
    # The full learning rate (0.1, no normalisation layers) diverges within a few
    # steps at this size; the reduced run uses 0.01 so that K-step parity compares
    # a training trajectory rather than an overflow.
    "vgg11": dict(channels=[16, 24, 40, 40, 48, 48, 56, 56], batch=3, steps=4,
                  opt=dict(kind="sgd", lr=0.01, momentum=0.9, weight_decay=5e-4)),
    "linear4x8192": dict(dims=[520] * 5, batch=40, steps=3),
    # every kind of block: t = 1, stride 2, residual repeats; ragged widths
    "mbv2": dict(image=14, stem=8, blocks=[[1, 6, 1, 1], [6, 12, 2, 2], [6, 16, 2, 2],
                                           [4, 20, 1, 1]],
                 head=40, batch=3, steps=3),
}


def get_config(name):
    """Full-size workload `name` (a deep copy, safe to modify)."""
    cfg = copy.deepcopy(CONFIGS[name])
    cfg["name"] = name
    return cfg


def reduced_config(name, **overrides):
    """Small workload of the same family as `name`, with optional overrides."""
    cfg = get_config(name)
    cfg.update(copy.deepcopy(_REDUCED[name]))
    cfg.update(overrides)
    cfg["name"] = name + "-reduced"
    return cfg


def mlp_ties(cfg):
    """{layer: earlier layer whose weight and bias it applies again} (1-based) of
    an MLP workload; checked to be a same-shape, earlier, untied layer."""
    tie = {int(k): int(v) for k, v in cfg.get("tie", {}).items()}
    dims = cfg["dims"]
    for i, j in tie.items():
        if not (1 <= j < i <= len(dims) - 1) or j in tie:
            raise ValueError(f"layer {i} cannot apply layer {j}'s parameters")
        if (dims[i - 1], dims[i]) != (dims[j - 1], dims[j]):
            raise ValueError(f"layers {i} and {j} have different shapes")
    return tie


def mbv2_blocks(cfg):
    """The inverted-residual blocks of an mbv2 workload, in order: dicts with
    name (parameter prefix), t, cin, hidden (t * cin), cout, stride,
    residual, and the input and output spatial sizes h_in, h_out."""
    out = []
    cin, h = cfg["stem"], cfg["image"]
    k = 0
    for t, c, n, s in cfg["blocks"]:
        for r in range(n):
            k += 1
            stride = s if r == 0 else 1
            h_out = (h - 1) // stride + 1
            out.append(dict(name=f"blk{k}.", t=t, cin=cin, hidden=t * cin, cout=c, stride=stride,
                            residual=stride == 1 and cin == c, h_in=h, h_out=h_out))
            cin, h = c, h_out
    return out


def param_specs(cfg):
    """Trainable tensors in model order: list of (name, shape, init, fan_in).

    init is "kaiming" (uniform on +-sqrt(6/fan_in)), "zeros" or "ones".
    """
    specs = []
    kind = cfg["kind"]
    if kind == "mlp":
        dims = cfg["dims"]
        tie = mlp_ties(cfg)
        for i in range(len(dims) - 1):
            if i + 1 in tie:
                continue   # applies an earlier layer's parameters
            specs.append((f"fc{i + 1}.weight", (dims[i + 1], dims[i]), "kaiming", dims[i]))
            if cfg["bias"]:
                specs.append((f"fc{i + 1}.bias", (dims[i + 1],), "zeros", dims[i]))
    elif kind == "tblock":
        d, f = cfg["hidden"], cfg["ffn"]
        for b in range(cfg["blocks"]):
            p = f"blk{b + 1}."
            specs += [
                (p + "ln1.weight", (d,), "ones", d),
                (p + "ln1.bias", (d,), "zeros", d),
                (p + "qkv.weight", (3 * d, d), "kaiming", d),
                (p + "qkv.bias", (3 * d,), "zeros", d),
                (p + "proj.weight", (d, d), "kaiming", d),
                (p + "proj.bias", (d,), "zeros", d),
                (p + "ln2.weight", (d,), "ones", d),
                (p + "ln2.bias", (d,), "zeros", d),
                (p + "fc1.weight", (f, d), "kaiming", d),
                (p + "fc1.bias", (f,), "zeros", d),
                (p + "fc2.weight", (d, f), "kaiming", f),
                (p + "fc2.bias", (d,), "zeros", f),
            ]
    elif kind == "vgg":
        cin = cfg["in_channels"]
        for i, cout in enumerate(cfg["channels"]):
            specs.append((f"conv{i + 1}.weight", (cout, 3, 3, cin), "kaiming", 9 * cin))
            specs.append((f"conv{i + 1}.bias", (cout,), "zeros", 9 * cin))
            cin = cout
        specs.append(("fc.weight", (cfg["classes"], cin), "kaiming", cin))
        specs.append(("fc.bias", (cfg["classes"],), "zeros", cin))
    elif kind == "mbv2":
        cin = cfg["in_channels"]
        specs.append(("stem.weight", (cfg["stem"], 3, 3, cin), "kaiming", 9 * cin))
        specs.append(("stem.bias", (cfg["stem"],), "zeros", 9 * cin))
        for b in mbv2_blocks(cfg):
            p, ci, hd, co = b["name"], b["cin"], b["hidden"], b["cout"]
            if b["t"] != 1:
                specs.append((p + "expand.weight", (hd, ci), "kaiming", ci))
                specs.append((p + "expand.bias", (hd,), "zeros", ci))
            specs.append((p + "dw.weight", (3, 3, hd), "kaiming", 9))
            specs.append((p + "dw.bias", (hd,), "zeros", 9))
            specs.append((p + "project.weight", (co, hd), "kaiming", hd))
            specs.append((p + "project.bias", (co,), "zeros", hd))
        last = mbv2_blocks(cfg)[-1]["cout"]
        specs.append(("head.weight", (cfg["head"], last), "kaiming", last))
        specs.append(("head.bias", (cfg["head"],), "zeros", last))
        specs.append(("fc.weight", (cfg["classes"], cfg["head"]), "kaiming", cfg["head"]))
        specs.append(("fc.bias", (cfg["classes"],), "zeros", cfg["head"]))
    else:
        raise ValueError(f"unknown model kind {kind!r}")
    return specs


def input_shape(cfg):
    """Shape of one input batch."""
    if cfg["kind"] == "mlp":
        return (cfg["batch"], cfg["dims"][0])
    if cfg["kind"] == "tblock":
        return (cfg["batch"], cfg["hidden"])
    if cfg["kind"] in ("vgg", "mbv2"):
        s = cfg["image"]
        return (cfg["batch"], s, s, cfg["in_channels"])
    raise ValueError(cfg["kind"])


def output_shape(cfg):
    """Shape of the model output (logits or regression output)."""
    if cfg["kind"] == "mlp":
        return (cfg["batch"], cfg["dims"][-1])
    if cfg["kind"] == "tblock":
        return (cfg["batch"], cfg["hidden"])
    return (cfg["batch"], cfg["classes"])


def describe(cfg):
    """One-line human description of a workload."""
    k = cfg["kind"]
    if k == "mlp":
        s = "mlp " + "-".join(map(str, cfg["dims"]))
    elif k == "tblock":
        s = f"tblock x{cfg['blocks']} d{cfg['hidden']} ffn{cfg['ffn']}"
    elif k == "mbv2":
        s = f"mbv2 {len(mbv2_blocks(cfg))} blocks stem{cfg['stem']} head{cfg['head']} img{cfg['image']}"
    else:
        s = "vgg " + "-".join(map(str, cfg["channels"])) + f" img{cfg['image']}"
    return f"{s} batch{cfg['batch']} {cfg['dtype']} {cfg['opt']['kind']} {cfg['loss']}"
