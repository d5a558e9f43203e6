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

Returned by run(): per-step losses (loss t uses theta^(t-1)), the evaluation
loss at theta^(K), final values / histories / step counters of every
parameter, the flags and counts, and the max-pool argmax of step 1.

Pinned by: the ordering invariant eager == ff(flushed) == bf bit for bit, a
planted dependency violation that breaks it, a shared-parameter toy with
step == K (tests/test_oracle_orderings.py).  Whole K-step trajectories have no
printed reference values in the paper: beyond the component pins and the
invariant they are parity unpinned.
"""
import numpy as np

from workloads import make_params, make_batch, make_eval_batch
from . import layers as L
from .losses import LOSSES
from .optim import apply as apply_optimizer


class Model:
    def __init__(self, nodes, params, loss, hyper):
        self.nodes = nodes            # [(op, [input names], output name)]
        self.params = params          # {name: Param} in model order
        self.loss = loss
        self.hyper = hyper
        self.last_argmax = {}

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
    def step_eager(self, x, target):
        out, tape = self.forward(x)
        loss, dout = self.loss_and_grad(out, target)
        self.backward(tape, dout)
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
        cur = "input"
        for i in range(1, n_layers + 1):
            z = f"z{i}"
            nodes.append((L.Linear(P(f"fc{i}.weight"), P(f"fc{i}.bias")), [cur], z))
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
    else:
        raise ValueError(kind)
    return Model(nodes, params, cfg["loss"], cfg["opt"])


def run(cfg, ordering, steps=None, seed=0, race_bug=False, init=None, batches=None):
    """Train workload `cfg` for `steps` steps under `ordering` in float64.

    Returns a dict: losses, eval_loss, params / m / v (float64 arrays by name),
    step (int by name), updated (per node, after the run), count (by name),
    argmax (max-pool window positions of step 1, by node index).
    """
    steps = cfg["steps"] if steps is None else steps
    model = new_model(cfg, init, seed)
    losses = []
    argmax = {}
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
        if t == 1:
            argmax = dict(model.last_argmax)
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
    )
