"""Models and the three training orderings, float64.

A model is a topologically sorted array of nodes (operator, input names,
output name) -- the input of Alg. 2 and Alg. 3.  The orderings:

  eager  Section 1 / Fig. 1(b): forward of every node, backward of every node
         accumulating every gradient, then the optimizer of every parameter.
  ff     forward-fusion, Appendix B.1, Alg. 2: before a node executes, if its
         `updated` flag is False, the optimizer of each of its parameters runs
         (consuming the gradient pending from the previous iteration) and the
         flag is set; backward accumulates gradients and clears the flag.
  bf     backward-fusion, Appendix B.2, Alg. 3: forward counts the uses of each
         parameter; backward accumulates, decrements the count and runs the
         optimizer when it reaches 0 -- after the node's input gradient was
         computed with the old value (the dependency rule after Alg. 3).

Readings where the paper is silent:
  * FF, first iteration: nothing is pending, so every `updated` flag starts
    True (running the optimizer on an absent gradient would take a spurious
    step with weight decay or Adam).
  * FF, end of training: the last update stays pending until the next forward
    of the node; flush() applies it (an evaluation forward does the same).
  * The update applied during forward t+1 is eager's update t, counted when
    it is applied.
  * Global-norm clipping (optional `clip_norm` in the optimizer dict): eager
    and forward-fusion scale every gradient of the step right after the
    backward pass; backward-fusion refuses it (Table 1).

Returned by run(): per-step losses (loss t uses theta^(t-1)), the evaluation
loss at theta^(K), final values / histories / step counters of every
parameter, the flags and counts, and the max-pool argmax of step 1.

For Adam-family optimizers run() also reports, per parameter element, the
smallest positive bias-corrected second-moment root sqrt(v_t / (1 - beta2^t))
seen over the steps (inf if the gradient was exactly 0 at every step: such an
element never moves under Adam); this is instrumentation only.  Where it is
comparable to eps, the update
m_hat / (sqrt(v_hat) + eps) is ill-conditioned in the gradient (its derivative
reaches 1/eps), so any float32 rounding of the gradient moves that element by
up to a whole step; the GPU parity tests use this to tell such elements apart.

Pinned by: the ordering invariant eager == ff(flushed) == bf bit for bit, a
planted dependency violation that breaks it, a shared-parameter toy with
step == K (tests/test_oracle_orderings.py); whole K-step eager trajectories of
every model family against torch autograd + torch.optim in float64
(tests/test_oracle_vs_torch.py).  The paper prints no reference values for
trajectories, so these are independent-implementation pins.
"""
import itertools

import numpy as np

from workloads import make_params, make_batch, make_eval_batch, mlp_ties, mbv2_blocks
from . import layers as L
from .losses import LOSSES
from .optim import SLICE, apply as apply_optimizer, clip_scale


class Model:
    def __init__(self, nodes, params, loss, hyper):
        self.nodes = nodes            # [(op, [input names], output name)]
        self.params = params          # {name: Param} in model order
        self.loss = loss
        self.hyper = hyper
        self.last_argmax = {}
        self.last_clip = None         # (scale, norm) of the last clipped step

    # -- plain passes ---------------------------------------------------
    def forward(self, x, before_node=None):
        env = {"input": x}
        tape = []
        for i, (op, ins, out) in enumerate(self.nodes):
            if before_node is not None:
                before_node(op)
            y, ctx = op.forward(*[env[n] for n in ins])
            env[out] = y
            tape.append(ctx)
            if isinstance(op, L.MaxPool2x2):
                self.last_argmax[i] = op.last_argmax
        return env["output"], tape

    def backward(self, tape, dout, after_node=None, race_bug=False):
        genv = {"output": dout}
        for (op, ins, out), ctx in zip(reversed(self.nodes), reversed(tape)):
            dy = genv.pop(out)
            if race_bug:
                # Planted violation of the dependency rule (tests only): update
                # the parameters first, then back-propagate with the new values.
                _, grads = op.backward(ctx, dy)
                _accumulate(op, grads)
                after_node(op)
                dxs, _ = op.backward(ctx, dy)
            else:
                dxs, grads = op.backward(ctx, dy)
                _accumulate(op, grads)
                if after_node is not None:
                    after_node(op)
            for name, dx in zip(ins, dxs):
                genv[name] = genv[name] + dx if name in genv else dx

    def loss_and_grad(self, out, target):
        return LOSSES[self.loss](out, target)

    def eval_loss(self, x, target):
        out, _ = self.forward(x)
        return LOSSES[self.loss](out, target)[0]

    # -- orderings ------------------------------------------------------
    def clip(self):
        """Global-norm clipping of every accumulated gradient when the optimizer
        dict sets `clip_norm` (Appendix B.1): after the backward pass, before
        any of these gradients is consumed.  Records (scale, norm)."""
        max_norm = self.hyper.get("clip_norm")
        if max_norm is None:
            return
        ps = [p for p in self.params.values() if p.grad is not None]
        scale, norm = clip_scale([p.grad for p in ps], max_norm)
        self.last_clip = (scale, norm)
        for p in ps:
            p.grad = p.grad * scale

    def step_eager(self, x, target):
        out, tape = self.forward(x)
        loss, dout = self.loss_and_grad(out, target)
        self.backward(tape, dout)
        self.clip()
        for p in self.params.values():
            if p.grad is not None:
                apply_optimizer(p, self.hyper)
        return loss

    def step_ff(self, x, target):
        def before(op):
            if not op.updated:
                for p in op.params:
                    if p.grad is not None:
                        apply_optimizer(p, self.hyper)
                op.updated = True

        def after(op):
            op.updated = False

        out, tape = self.forward(x, before_node=before)
        loss, dout = self.loss_and_grad(out, target)
        self.backward(tape, dout, after_node=after)
        self.clip()   # the pending gradients, before the next forward consumes them
        return loss

    def flush(self):
        """Apply every update forward-fusion still holds (the next forward would)."""
        for op, _, _ in self.nodes:
            if not op.updated:
                for p in op.params:
                    if p.grad is not None:
                        apply_optimizer(p, self.hyper)
                op.updated = True

    def step_bf(self, x, target, race_bug=False):
        if self.hyper.get("clip_norm") is not None:
            raise ValueError("backward-fusion updates each tensor before the other gradients "
                             "exist, so it cannot clip by the global norm (Table 1)")

        def count(op):
            for p in op.params:
                p.count += 1

        def after(op):
            for p in op.params:
                p.count -= 1
                if p.count == 0:
                    apply_optimizer(p, self.hyper)

        out, tape = self.forward(x, before_node=count)
        loss, dout = self.loss_and_grad(out, target)
        self.backward(tape, dout, after_node=after, race_bug=race_bug)
        return loss


def ambiguous_relu_decisions(model, x, c=1.0):
    """Backward ReLU decisions a float32 run may take differently.

    A decision z > 0 is ambiguous when |z| < c * 2^-24 * S, with S the sum
    of |x w| over the contraction that produced z (+|b|): the rounding scale
    of the float32 sum (S = 0 means every term is exactly 0: not ambiguous).  ReLUs fed by a Linear (directly or through a PixelMap
    reshape of its rows), a Conv3x3 or a DepthwiseConv3x3 are examined.
    Returns [(node index, index of the element in the ReLU input ..., |z| /
    scale)] sorted from most to least ambiguous; for a [rows, cols] input the
    index is (row, column).
    """
    u = 2.0 ** -24
    env = {"input": x}
    producer = {}
    out = []
    for i, (op, ins, name) in enumerate(model.nodes):
        vals = [env[n] for n in ins]
        y, _ = op.forward(*vals)
        if isinstance(op, L.ReLU) and ins[0] in producer:
            src, src_in = producer[ins[0]]
            scale = (u * src.abs_bound(src_in)).reshape(vals[0].shape)
            ratio = np.abs(vals[0]) / np.maximum(scale, 1e-300)
            # S == 0: every term and the bias are exactly 0, so is z on any machine
            for idx in zip(*np.nonzero((ratio < c) & (scale > 0))):
                out.append((i,) + tuple(int(t) for t in idx) + (float(ratio[idx]),))
        if isinstance(op, (L.Linear, L.Conv3x3, L.DepthwiseConv3x3)):
            producer[name] = (op, vals[0])
        elif isinstance(op, L.PixelMap) and ins[0] in producer:
            producer[name] = producer[ins[0]]   # the same values, reshaped
        env[name] = y
    out.sort(key=lambda d: d[-1])
    return out


def candidate_steps(cfg, state, t, max_decisions=8, seed=0, c=1.0):
    """Every valid float32 outcome of eager step t from `state` (a snapshot).

    Enumerates the subsets of the ambiguous ReLU decisions of the step (at most
    `max_decisions`, the most ambiguous ones; the threshold c of
    ambiguous_relu_decisions allows for error carried in from earlier layers),
    fewest flips first, and yields
    (flipped decisions, loss, state after the step) for each; for Adam-family
    optimizers the state also holds min_sqrt_vhat, the positive bias-corrected
    sqrt(v_hat) after the step (inf where v is 0), as run() reports it.
    """
    x, y = make_batch(cfg, t, seed)
    x = np.asarray(x, np.float64)
    y = y if y.dtype == np.int64 else np.asarray(y, np.float64)
    probe = new_model(cfg, init=state["params"])
    dec = ambiguous_relu_decisions(probe, x, c)[:max_decisions]
    shapes = {}
    env = {"input": x}
    for i, (op, ins, name) in enumerate(probe.nodes):
        env[name] = op.forward(*[env[n] for n in ins])[0]
        if isinstance(op, L.ReLU):
            shapes[i] = env[ins[0]].shape
    for nflip in range(len(dec) + 1):
        for subset in itertools.combinations(dec, nflip):
            model = new_model(cfg, init=state["params"])
            for k, p in model.params.items():
                p.m, p.v, p.step = state["m"][k].copy(), state["v"][k].copy(), state["step"][k]
            for d in subset:
                i, idx = d[0], d[1:-1]
                op = model.nodes[i][0]
                if op.flip is None:
                    op.flip = np.zeros(shapes[i], bool)
                op.flip[idx] = True
            loss = model.step_eager(x, y)
            ps = model.params
            vh = {}
            if cfg["opt"]["kind"] in ("adam", "adamw"):
                for k, p in ps.items():
                    r = np.sqrt(p.v / (1.0 - cfg["opt"]["beta2"] ** p.step))
                    vh[k] = np.where(r > 0.0, r, np.inf)
            yield subset, loss, dict(params={k: p.value for k, p in ps.items()},
                                     m={k: p.m for k, p in ps.items()},
                                     v={k: p.v for k, p in ps.items()},
                                     step={k: p.step for k, p in ps.items()},
                                     min_sqrt_vhat=vh)


def _accumulate(op, grads):
    for p, g in zip(op.params, grads):
        p.grad = g.copy() if p.grad is None else p.grad + g


def new_model(cfg, init=None, seed=0):
    """Build the model of workload `cfg` from its seeded initial parameters."""
    init = make_params(cfg, seed) if init is None else init
    params = {k: L.Param(k, v) for k, v in init.items()}
    P = params.get
    nodes = []
    kind = cfg["kind"]
    if kind == "mlp":
        n_layers = len(cfg["dims"]) - 1
        tie = mlp_ties(cfg)
        lin = {}
        cur = "input"
        for i in range(1, n_layers + 1):
            z = f"z{i}"
            # a tied layer is the same operator applied again (one `updated` flag,
            # its parameters counted once per use)
            lin[i] = lin[tie[i]] if i in tie else L.Linear(P(f"fc{i}.weight"), P(f"fc{i}.bias"))
            nodes.append((lin[i], [cur], z))
            cur = z
            if i < n_layers and cfg["act"] == "relu":
                nodes.append((L.ReLU(), [z], f"a{i}"))
                cur = f"a{i}"
        nodes[-1] = (nodes[-1][0], nodes[-1][1], "output")
    elif kind == "tblock":
        d = cfg["hidden"]
        bf16 = cfg["dtype"] == "bf16"
        cur = "input"
        for b in range(1, cfg["blocks"] + 1):
            p = f"blk{b}."
            nodes += [
                (L.LayerNorm(P(p + "ln1.weight"), P(p + "ln1.bias"), cfg["ln_eps"]), [cur], p + "a"),
                (L.Linear(P(p + "qkv.weight"), P(p + "qkv.bias"), bf16), [p + "a"], p + "qkv"),
                (L.SliceCols(2 * d, 3 * d), [p + "qkv"], p + "v"),
                (L.Linear(P(p + "proj.weight"), P(p + "proj.bias"), bf16), [p + "v"], p + "o"),
                (L.Add(), [cur, p + "o"], p + "h"),
                (L.LayerNorm(P(p + "ln2.weight"), P(p + "ln2.bias"), cfg["ln_eps"]), [p + "h"], p + "c"),
                (L.Linear(P(p + "fc1.weight"), P(p + "fc1.bias"), bf16), [p + "c"], p + "u"),
                (L.GELU(), [p + "u"], p + "g"),
                (L.Linear(P(p + "fc2.weight"), P(p + "fc2.bias"), bf16), [p + "g"], p + "w"),
                (L.Add(), [p + "h", p + "w"], p + "y"),
            ]
            cur = p + "y"
        nodes[-1] = (nodes[-1][0], nodes[-1][1], "output")
    elif kind == "vgg":
        cur = "input"
        for i in range(1, len(cfg["channels"]) + 1):
            nodes.append((L.Conv3x3(P(f"conv{i}.weight"), P(f"conv{i}.bias")), [cur], f"c{i}"))
            nodes.append((L.ReLU(), [f"c{i}"], f"r{i}"))
            cur = f"r{i}"
            if i in cfg["pool_after"]:
                nodes.append((L.MaxPool2x2(), [cur], f"p{i}"))
                cur = f"p{i}"
        nodes.append((L.Flatten(), [cur], "flat"))
        nodes.append((L.Linear(P("fc.weight"), P("fc.bias")), ["flat"], "output"))
    elif kind == "mbv2":
        n = cfg["batch"]

        def pointwise(prefix, src, h, tag):
            """A 1x1 convolution: a linear over the pixel rows of an [n,h,h,c] map."""
            nodes.extend([(L.PixelRows(), [src], tag + "r"),
                          (L.Linear(P(prefix + ".weight"), P(prefix + ".bias")), [tag + "r"], tag + "z"),
                          (L.PixelMap(n, h, h), [tag + "z"], tag + "m")])
            return tag + "m"

        nodes.append((L.Conv3x3(P("stem.weight"), P("stem.bias")), ["input"], "s"))
        nodes.append((L.ReLU(), ["s"], "sa"))
        cur = "sa"
        for b in mbv2_blocks(cfg):
            p = b["name"]
            x_in = cur
            if b["t"] != 1:
                z = pointwise(p + "expand", cur, b["h_in"], p + "e")
                nodes.append((L.ReLU(), [z], p + "ea"))
                cur = p + "ea"
            nodes.append((L.DepthwiseConv3x3(P(p + "dw.weight"), P(p + "dw.bias"), b["stride"]),
                          [cur], p + "d"))
            nodes.append((L.ReLU(), [p + "d"], p + "da"))
            cur = pointwise(p + "project", p + "da", b["h_out"], p + "p")
            if b["residual"]:
                nodes.append((L.Add(), [x_in, cur], p + "y"))
                cur = p + "y"
        z = pointwise("head", cur, mbv2_blocks(cfg)[-1]["h_out"], "h")
        nodes.append((L.ReLU(), [z], "ha"))
        nodes.append((L.GlobalAvgPool(), ["ha"], "pool"))
        nodes.append((L.Linear(P("fc.weight"), P("fc.bias")), ["pool"], "output"))
    else:
        raise ValueError(kind)
    return Model(nodes, params, cfg["loss"], cfg["opt"])


def _min_sqrt_vhat(prev, v, bc2):
    """Element-wise running minimum over steps of sqrt(v / bc2), zeros read as
    infinite (test bookkeeping for the tolerance of Adam's update; no part of
    the training arithmetic), taken in slices of the optimizer's slice size."""
    out = np.empty_like(v)
    fv, fo = v.reshape(-1), out.reshape(-1)
    fp = prev.reshape(-1) if prev is not None else None
    for s in range(0, v.size, SLICE):
        sl = slice(s, s + SLICE)
        r = np.sqrt(fv[sl] / bc2)
        r = np.where(r > 0.0, r, np.inf)
        fo[sl] = np.minimum(fp[sl], r) if fp is not None else r
    return out


def run(cfg, ordering, steps=None, seed=0, race_bug=False, init=None, batches=None,
        snapshots=(), on_step=None):
    """Train workload `cfg` for `steps` steps under `ordering` in float64.

    Returns a dict: losses, eval_loss, params / m / v (float64 arrays by name),
    step (int by name), updated (per node, after the run), count (by name),
    argmax (max-pool window positions of step 1, by node index),
    clips ((scale, norm) of each step's global-norm clipping, or None),
    snapshots {t: state after step t (t = 0: the initial state)} for t in
    `snapshots` -- params / m / v copies, step counters, the gradient the
    update of step t consumed and min_sqrt_vhat up to step t (eager ordering).
    on_step: optional callable given each finished step's index (progress
    reports of long runs; it sees nothing of the arithmetic).
    """
    steps = cfg["steps"] if steps is None else steps
    model = new_model(cfg, init, seed)
    losses = []
    argmax = {}
    hyper = cfg["opt"]
    min_vhat = {}
    snaps = {}
    clips = []

    def snap():
        ps = model.params
        return dict(params={k: p.value.copy() for k, p in ps.items()},
                    m={k: p.m.copy() for k, p in ps.items()},
                    v={k: p.v.copy() for k, p in ps.items()},
                    step={k: p.step for k, p in ps.items()},
                    grad={k: getattr(p, "last_grad", None) for k, p in ps.items()},
                    min_sqrt_vhat={k: v.copy() for k, v in min_vhat.items()})

    if 0 in snapshots:
        snaps[0] = snap()
    for t in range(1, steps + 1):
        x, y = batches[t - 1] if batches is not None else make_batch(cfg, t, seed)
        x = np.asarray(x, np.float64)
        y = y if y.dtype == np.int64 else np.asarray(y, np.float64)
        if ordering == "eager":
            losses.append(model.step_eager(x, y))
        elif ordering == "ff":
            losses.append(model.step_ff(x, y))
        elif ordering == "bf":
            losses.append(model.step_bf(x, y, race_bug=race_bug))
        else:
            raise ValueError(ordering)
        clips.append(model.last_clip)
        if t == 1:
            argmax = dict(model.last_argmax)
        if hyper["kind"] in ("adam", "adamw"):
            for k, p in model.params.items():
                if p.step > 0:
                    min_vhat[k] = _min_sqrt_vhat(min_vhat.get(k), p.v,
                                                 1.0 - hyper["beta2"] ** p.step)
        if t in snapshots:
            snaps[t] = snap()
        if on_step is not None:
            on_step(t)
    updated_before_flush = [op.updated for op, _, _ in model.nodes]
    if ordering == "ff":
        model.flush()
    xe, ye = make_eval_batch(cfg, seed)
    ye = ye if ye.dtype == np.int64 else np.asarray(ye, np.float64)
    eval_loss = model.eval_loss(np.asarray(xe, np.float64), ye)
    ps = model.params
    return dict(
        losses=np.array(losses),
        eval_loss=eval_loss,
        params={k: p.value for k, p in ps.items()},
        m={k: p.m for k, p in ps.items()},
        v={k: p.v for k, p in ps.items()},
        step={k: p.step for k, p in ps.items()},
        count={k: p.count for k, p in ps.items()},
        updated_before_flush=updated_before_flush,
        updated=[op.updated for op, _, _ in model.nodes],
        argmax=argmax,
        clips=clips,
        min_sqrt_vhat=min_vhat,
        snapshots=snaps,
    )


class DecisionSearch:
    """Eager step t from a snapshot on a chain model, with the backward pass's
    rounding-sensitive decisions left open and settled node by node.

    A float32 run takes each ReLU mask (z > 0) and each max-pool window choice
    from values whose rounding error is of the order of u * S, with u = 2^-24
    and S = sum |x||w| + |b| over the contraction that produced them.  With a
    factor c for error carried in from earlier layers, a decision is ambiguous
    when
      ReLU      |z| < c u S(z);
      max-pool  an entry q of the window lies within c u (S_p + S_q) of the
                window's first maximum p and one of the two is positive; the
                flipped decision routes the gradient to q.
    Any set of flipped ambiguous decisions is a valid float32 outcome of the
    step.  At full size there are far too many sets to enumerate, but in a
    chain the gradient of a parametrised node depends only on the decisions
    above it.  So the search visits the parametrised nodes from the output
    down: candidates() yields, for each subset of the open decisions between
    the node and the one above it (the most ambiguous `max_decisions`, at most
    `max_flips` flipped, fewest flips first), the node's parameters after the
    update; accept() settles one subset and moves down; finish() returns the
    whole state after the step.  The forward pass takes the oracle's own
    decisions (a flipped one changes a forward value only at rounding level).
    """

    def __init__(self, cfg, state, t, c=8.0, max_decisions=6, seed=0):
        x, y = make_batch(cfg, t, seed)
        x = np.asarray(x, np.float64)
        y = y if y.dtype == np.int64 else np.asarray(y, np.float64)
        self.model = model = new_model(cfg, init=state["params"])
        for k, p in model.params.items():
            p.m, p.v, p.step = state["m"][k].copy(), state["v"][k].copy(), state["step"][k]
        self.hyper = cfg["opt"]
        self.max_decisions = max_decisions
        nodes = model.nodes
        prev = "input"
        for op, ins, out in nodes:
            if ins != [prev]:
                raise ValueError("the decision search needs a chain model")
            prev = out
        u = 2.0 ** -24
        self.tape, self.decisions = [], {}
        h, scale = x, None
        for i, (op, _, _) in enumerate(nodes):
            out, ctx = op.forward(h)
            self.tape.append(ctx)
            dec = []
            next_scale = None
            if isinstance(op, (L.Linear, L.Conv3x3)):
                next_scale = op.abs_bound(h)
            elif isinstance(op, L.ReLU) and scale is not None:
                ratio = np.abs(h) / np.maximum(c * u * scale, 1e-300)
                for idx in zip(*np.nonzero(ratio < 1.0)):
                    dec.append((float(ratio[idx]), ("relu", i, tuple(int(a) for a in idx), None)))
                next_scale = scale
            elif isinstance(op, L.MaxPool2x2) and scale is not None:
                arg = ctx[1]
                win = [h[:, a::2, b::2, :] for a in (0, 1) for b in (0, 1)]
                sc = [scale[:, a::2, b::2, :] for a in (0, 1) for b in (0, 1)]
                best = np.choose(arg, win)
                sbest = np.choose(arg, sc)
                for q in range(4):
                    den = np.maximum(c * u * (sbest + sc[q]), 1e-300)
                    ratio = np.abs(best - win[q]) / den
                    amb = (ratio < 1.0) & (arg != q) & (np.maximum(best, win[q]) > 0.0)
                    for idx in zip(*np.nonzero(amb)):
                        dec.append((float(ratio[idx]),
                                    ("pool", i, tuple(int(a) for a in idx), q)))
            if dec:
                self.decisions[i] = dec
            h, scale = out, next_scale
        self.loss, self.g = model.loss_and_grad(h, y)
        self.pos = len(nodes) - 1      # next node to back-propagate
        self.grads = {}
        self.flipped = []
        self._cache = None
        self._advance_to_param()

    # -- walking ----------------------------------------------------------
    def _advance_to_param(self):
        """Find the next parametrised node at or below self.pos."""
        k = self.pos
        while k >= 0 and not self.model.nodes[k][0].params:
            k -= 1
        self.node = k if k >= 0 else None

    @property
    def done(self):
        return self.node is None

    def current(self):
        """(node index, parameter names) of the node being settled."""
        op = self.model.nodes[self.node][0]
        return self.node, [p.name for p in op.params]

    def open_decisions(self):
        """The ambiguous decisions between the current node and the one above,
        most ambiguous first, at most max_decisions of them."""
        dec = []
        for j in range(self.node + 1, self.pos + 1):
            dec += self.decisions.get(j, [])
        dec.sort(key=lambda d: d[0])
        return [d[1] for d in dec[: self.max_decisions]]

    def _through(self, subset):
        """Gradient w.r.t. the current node's output with `subset` flipped, then
        the node's own backward: (dxs, grads)."""
        g = self.g
        for j in range(self.pos, self.node, -1):
            op = self.model.nodes[j][0]
            ctx = self.tape[j]
            mine = [d for d in subset if d[1] == j]
            if mine and isinstance(op, L.ReLU):
                op.flip = np.zeros(ctx.shape, bool)
                for d in mine:
                    op.flip[d[2]] = True
                try:
                    (g,), _ = op.backward(ctx, g)
                finally:
                    op.flip = None
            elif mine:
                shape, arg = ctx
                arg = arg.copy()
                for d in mine:
                    arg[d[2]] = d[3]
                (g,), _ = op.backward((shape, arg), g)
            else:
                (g,), _ = op.backward(ctx, g)
        return self.model.nodes[self.node][0].backward(self.tape[self.node], g)

    def candidates(self, max_flips=2):
        """Yield (flipped decisions, {name: (value, m, v)} after the update) for
        the current node, fewest flips first."""
        op = self.model.nodes[self.node][0]
        dec = self.open_decisions()
        for n in range(min(max_flips, len(dec)) + 1):
            for subset in itertools.combinations(dec, n):
                dxs, grads = self._through(subset)
                self._cache = (subset, dxs, grads)
                upd = {}
                for p, g in zip(op.params, grads):
                    q = L.Param(p.name, p.value)
                    q.m, q.v, q.step, q.grad = p.m.copy(), p.v.copy(), p.step, g
                    apply_optimizer(q, self.hyper)
                    upd[p.name] = (q.value, q.m, q.v)
                yield subset, upd

    def accept(self, subset):
        """Settle the current node's decisions to `subset` and move down."""
        subset = tuple(subset)
        if self._cache is not None and self._cache[0] == subset:
            _, dxs, grads = self._cache
        else:
            dxs, grads = self._through(subset)
        op = self.model.nodes[self.node][0]
        for p, g in zip(op.params, grads):
            self.grads[p.name] = g
        self.flipped += list(subset)
        self.g = dxs[0]
        self.pos = self.node - 1
        self._cache = None
        self._advance_to_param()

    def finish(self):
        """State after the step (every node settled): params, m, v, step by name."""
        if not self.done:
            raise RuntimeError("nodes left to settle")
        ps = self.model.params
        for k, p in ps.items():
            p.grad = self.grads[k]
            apply_optimizer(p, self.hyper)
        return dict(params={k: p.value for k, p in ps.items()},
                    m={k: p.m for k, p in ps.items()},
                    v={k: p.v for k, p in ps.items()},
                    step={k: p.step for k, p in ps.items()})
