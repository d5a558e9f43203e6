"""Host scheduler: the three training orderings over the opfuse C ABI.

The model is a topologically sorted array of operators (the input of Alg. 2
and Alg. 3): linear or 3x3-convolution layers, each followed by its
activation (fused into the kernel's epilogue) and optionally by a 2x2
max-pool.  Every kernel runs in libopfuse.so; this module only decides which
entry point runs where and keeps the per-parameter state the paper's
algorithms need:

  step[theta]   1-based index of the update applied last (mirrored on the device)
  updated[f]    Alg. 2 flag: False while f holds a pending update
  count[theta]  Alg. 3 counter: forward uses not yet back-propagated

Orderings (Section 3, Fig. 1(b)-(d)):
  eager  forward; backward writing every gradient; one multi-tensor optimizer
         launch over every parameter.
  ff     forward-fusion: a layer whose `updated` flag is False applies its
         pending update in its forward (linear layers: of_linear_fwd_fused,
         while the W tiles load; convolutions: an element-wise pass right
         before the forward); backward writes the gradients, which stay
         pending; flush() applies what is still pending.
  bf     backward-fusion: each layer's data gradient runs with the old weights
         on the main stream, then its weight-gradient kernel with the
         optimizer in the epilogue runs on a second stream, so the update of
         layer i overlaps the back-propagation of layer i-1 (Section 3,
         "parallelism"); the next step's forward waits for it.

Torch is used for device memory, streams and events only.
"""
import numpy as np
import torch

from . import _lib as L


class ParamBuf:
    """A trainable tensor on the device with its history and host counters."""

    def __init__(self, name, value, kind, device, with_grad=True):
        self.name = name
        self.w = torch.as_tensor(np.ascontiguousarray(value, dtype=np.float32)).to(device)
        self.m = torch.zeros_like(self.w)
        self.v = torch.zeros_like(self.w) if kind != "sgd" else None
        self.g = torch.zeros_like(self.w) if with_grad else None
        self.p = L.param_of(self.w, self.m, self.v)
        self.step = 0
        self.count = 0

    @property
    def numel(self):
        return self.w.numel()


def _ptr(t):
    return t.data_ptr() if t is not None else None


class LinearOp:
    """f = act(X W^T + b) on a [M, K] input."""

    kind = "linear"

    def __init__(self, name, W, b, M, act):
        N, K = W.w.shape
        self.name, self.W, self.b = name, W, b
        self.M, self.N, self.K = M, N, K
        self.act = act
        self.desc = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.ACTS[act], int(b is not None))
        self.updated = True
        self.params = [W] if b is None else [W, b]
        self.out_shape = (M, N)

    def ws(self, which):
        return L.of_linear_workspace_size(self.desc, which)

    def fwd(self, tr, x, y):
        L.of_linear_fwd(self.desc, x, self.W.p, _ptr(self.b.w) if self.b else None, None, y,
                        *tr.ws_main_args(), tr._s())

    def fwd_ff(self, tr, x, y):
        b = self.b
        L.of_linear_fwd_fused(self.desc, x, self.W.p, self.W.g.data_ptr(),
                              b.p if b else None, b.g.data_ptr() if b else None, tr.opt, None, y,
                              *tr.ws_main_args(), tr._s())

    def dgrad(self, tr, g, prev, act_prev, dx):
        L.of_linear_bwd_data(self.desc, g, self.W.p, prev, act_prev, dx, *tr.ws_main_args(),
                             tr._s())

    def wgrad(self, tr, g, x):
        L.of_linear_bwd_weight(self.desc, g, x, self.W.g.data_ptr(),
                               self.b.g.data_ptr() if self.b else None, 0, *tr.ws_main_args(),
                               tr._s())

    def wgrad_fused(self, tr, g, x, stream):
        b = self.b
        L.of_linear_bwd_fused(self.desc, g, x, self.W.p, b.p if b else None, None, None, tr.opt,
                              None, 0, None, None, 0, *tr.ws_side_args(), stream, None)

    def bwd_fused(self, tr, g, x, prev, act_prev, dx):
        """Data gradient on the main stream, fused update on the side stream (one call)."""
        b = self.b
        L.of_linear_bwd_fused(self.desc, g, x, self.W.p, b.p if b else None, None, None, tr.opt,
                              prev, act_prev, dx, *tr.ws_main_args(), *tr.ws_side_args(),
                              tr._s(), tr.side.cuda_stream)


class ConvOp:
    """f = act(conv3x3(X, W) + b), padding 1, stride 1, on an NHWC [N, H, W, C] input."""

    kind = "conv"

    def __init__(self, name, W, b, N, H, Wd, act):
        Cout, _, _, C = W.w.shape
        self.name, self.W, self.b = name, W, b
        self.act = act
        self.desc = L.OfConvDesc(N, H, Wd, C, Cout, L.ACTS[act], int(b is not None))
        self.updated = True
        self.params = [W] if b is None else [W, b]
        self.out_shape = (N, H, Wd, Cout)
        # the implicit-GEMM view: [N*H*W, 9*C] x [9*C, Cout]
        self.M, self.N, self.K = N * H * Wd, Cout, 9 * C

    def ws(self, which):
        return L.of_conv_workspace_size(self.desc, which)

    def fwd(self, tr, x, y):
        L.of_conv_fwd(self.desc, x, self.W.p, _ptr(self.b.w) if self.b else None, y,
                      *tr.ws_main_args(), tr._s())

    def fwd_ff(self, tr, x, y):
        # The pending update runs element-wise right before the forward; the
        # filter-tile prologue of the convolution is not fused.
        for p in self.params:
            L.of_elementwise_fused_update(p.p, p.g.data_ptr(), 1, 0, tr.opt, tr._s())
        self.fwd(tr, x, y)

    def dgrad(self, tr, g, prev, act_prev, dx):
        L.of_conv_bwd_data(self.desc, g, self.W.p, prev, act_prev, dx, *tr.ws_main_args(),
                           tr._s())

    def wgrad(self, tr, g, x):
        L.of_conv_bwd_weight(self.desc, g, x, self.W.g.data_ptr(),
                             self.b.g.data_ptr() if self.b else None, 0, *tr.ws_main_args(),
                             tr._s())

    def wgrad_fused(self, tr, g, x, stream):
        b = self.b
        L.of_conv_wgrad_fused(self.desc, g, x, self.W.p, b.p if b else None, None, None, tr.opt,
                              *tr.ws_side_args(), stream)


class Trainer:
    """Trains one workload on one GPU under a chosen ordering."""

    def __init__(self, cfg, init, device="cuda:0"):
        if cfg["dtype"] != "f32":
            raise NotImplementedError("only fp32 operands in this build")
        L.load()
        self.cfg, self.hyper = cfg, cfg["opt"]
        self.device = torch.device(device)
        kind = self.hyper["kind"]
        self.params = {}
        self.ops, self.pool = [], []

        def pb(name):
            p = ParamBuf(name, init[name], kind, self.device)
            self.params[name] = p
            return p

        if cfg["kind"] == "mlp":
            M, dims = cfg["batch"], cfg["dims"]
            nl = len(dims) - 1
            for i in range(1, nl + 1):
                W = pb(f"fc{i}.weight")
                b = pb(f"fc{i}.bias") if cfg["bias"] else None
                self.ops.append(LinearOp(f"fc{i}", W, b, M, cfg["act"] if i < nl else "none"))
                self.pool.append(False)
        elif cfg["kind"] == "vgg":
            N, s, c = cfg["batch"], cfg["image"], cfg["in_channels"]
            for i, cout in enumerate(cfg["channels"], start=1):
                W, b = pb(f"conv{i}.weight"), pb(f"conv{i}.bias")
                self.ops.append(ConvOp(f"conv{i}", W, b, N, s, s, "relu"))
                pool = i in cfg["pool_after"]
                self.pool.append(pool)
                if pool:
                    s //= 2
                c = cout
            if s != 1:
                raise NotImplementedError("the classifier expects a 1x1 feature map")
            self.ops.append(LinearOp("fc", pb("fc.weight"), pb("fc.bias"), N, "none"))
            self.pool.append(False)
        else:
            raise NotImplementedError(f"model kind {cfg['kind']!r} has no GPU path in this build")

        f32 = dict(dtype=torch.float32, device=self.device)
        n = len(self.ops)
        # y[i]: layer i's output after its activation; gz[i]: gradient w.r.t. its
        # pre-activation; p/arg/gp: pooled output, position of each window's
        # maximum, gradient w.r.t. the pooled output.
        self.y = [torch.empty(op.out_shape, **f32) for op in self.ops]
        self.gz = [torch.empty(op.out_shape, **f32) for op in self.ops]
        self.p, self.arg, self.gp = [None] * n, [None] * n, [None] * n
        for i, op in enumerate(self.ops):
            if self.pool[i]:
                N_, H_, W_, C_ = op.out_shape
                ps = (N_, H_ // 2, W_ // 2, C_)
                self.p[i] = torch.empty(ps, **f32)
                self.arg[i] = torch.empty(ps, dtype=torch.uint8, device=self.device)
                self.gp[i] = torch.empty(ps, **f32)
        wsm = max([op.ws(w) for op in self.ops for w in (0, 1, 2)] + [16])
        wss = max([op.ws(2) for op in self.ops] + [16])
        if cfg["loss"] == "mse":
            wsm = max(wsm, L.of_mse_workspace_size(*self.ops[-1].out_shape))
        self.ws_main = torch.empty((wsm + 15) // 16 * 4, **f32)
        self.ws_side = torch.empty((wss + 15) // 16 * 4, **f32)
        self.losses = torch.zeros(4096, **f32)
        self.t = 0
        # Device copy of the 1-based index of the update being applied: advanced in
        # stream order right before each step's updates, read by the kernels when
        # they run, so one launch sequence (or a captured graph) serves every step.
        self.step_dev = torch.zeros(1, dtype=torch.int64, device=self.device)
        self.opt = L.make_opt(self.hyper, 0, self.step_dev.data_ptr())
        self.stream = torch.cuda.current_stream(self.device)
        self.side = torch.cuda.Stream(self.device)
        self.side_done = torch.cuda.Event()
        self.pending_ordering = None
        self.timer = None   # optional KernelTimer: HIP events around chosen launch classes

    # ------------------------------------------------------------ helpers
    def ws_main_args(self):
        return self.ws_main.data_ptr(), self.ws_main.numel() * 4

    def ws_side_args(self):
        return self.ws_side.data_ptr(), self.ws_side.numel() * 4

    def _s(self):
        return self.stream.cuda_stream

    def _advance(self, ps):
        """Next update index for parameters ps (host mirror + device counter)."""
        step = ps[0].step + 1
        if any(p.step + 1 != step for p in ps):
            raise RuntimeError("parameters out of step: this trainer keeps one update counter")
        L.of_step_advance(self.step_dev.data_ptr(), 1, self._s())
        return step

    def _t0(self, cls, stream, op=None):
        if self.timer is not None:
            self.timer.start(cls, stream, op)

    def _t1(self, cls, stream):
        if self.timer is not None:
            self.timer.stop(cls, stream)

    def _in(self, i, x):
        """Device pointer of layer i's input."""
        if i == 0:
            return x.data_ptr()
        return (self.p[i - 1] if self.pool[i - 1] else self.y[i - 1]).data_ptr()

    def _loss(self, y):
        self._t0("loss", self.stream)
        out = self.y[-1]
        M, C = out.shape
        loss_ptr = self.losses.data_ptr() + 4 * (self.t % self.losses.numel())
        if self.cfg["loss"] == "xent":
            L.of_xent_fwd_bwd(out.data_ptr(), y.data_ptr(), M, C, 0, loss_ptr,
                              self.gz[-1].data_ptr(), self._s())
        else:
            L.of_mse_fwd_bwd(out.data_ptr(), y.data_ptr(), M, C, 0, loss_ptr,
                             self.gz[-1].data_ptr(), *self.ws_main_args(), self._s())
        self._t1("loss", self.stream)

    def _forward(self, x, fused):
        for i, op in enumerate(self.ops):
            if fused and not op.updated:
                self._t0("fwd_ff", self.stream, op)
                op.fwd_ff(self, self._in(i, x), self.y[i].data_ptr())
                self._t1("fwd_ff", self.stream)
                op.updated = True
            else:
                self._t0("fwd", self.stream, op)
                op.fwd(self, self._in(i, x), self.y[i].data_ptr())
                self._t1("fwd", self.stream)
            if self.pool[i]:
                N, H, W, C = op.out_shape
                L.of_maxpool2x2_fwd(self.y[i].data_ptr(), N, H, W, C, self.p[i].data_ptr(),
                                    self.arg[i].data_ptr(), self._s())

    def _dgrad_target(self, i):
        """Where layer i's data gradient goes: (dx, prev, act_prev).  Through a
        max-pool the ReLU mask is applied by the pool's backward instead."""
        if self.pool[i - 1]:
            return self.gp[i - 1].data_ptr(), None, L.OF_ACT_NONE
        prev_act = self.ops[i - 1].act
        prev = self.y[i - 1].data_ptr() if prev_act != "none" else None
        return self.gz[i - 1].data_ptr(), prev, L.ACTS[prev_act]

    def _pool_bwd(self, i):
        """After layer i's data gradient: back through layer i-1's max-pool and ReLU."""
        if i > 0 and self.pool[i - 1]:
            N, H, W, C = self.ops[i - 1].out_shape
            L.of_maxpool2x2_bwd(self.gp[i - 1].data_ptr(), self.arg[i - 1].data_ptr(),
                                self.y[i - 1].data_ptr(), N, H, W, C,
                                self.gz[i - 1].data_ptr(), self._s())

    def _dgrad(self, i, op):
        dx, prev, act_prev = self._dgrad_target(i)
        self._t0("dgrad", self.stream, op)
        op.dgrad(self, self.gz[i].data_ptr(), prev, act_prev, dx)
        self._t1("dgrad", self.stream)

    def _backward_plain(self, x):
        for i in reversed(range(len(self.ops))):
            op = self.ops[i]
            if i > 0:
                self._dgrad(i, op)
            self._t0("wgrad", self.stream, op)
            op.wgrad(self, self.gz[i].data_ptr(), self._in(i, x))
            self._t1("wgrad", self.stream)
            self._pool_bwd(i)

    # ---------------------------------------------------------- orderings
    def step(self, x, y, ordering):
        """One training step on batch (x, y); the loss stays on the device."""
        if self.pending_ordering == "ff" and ordering != "ff":
            self.flush()
        if ordering == "eager":
            self._step_eager(x, y)
        elif ordering == "ff":
            self._step_ff(x, y)
        elif ordering == "bf":
            self._step_bf(x, y)
        else:
            raise ValueError(ordering)
        self.pending_ordering = ordering
        self.t += 1

    def _step_eager(self, x, y):
        self._forward(x, fused=False)
        self._loss(y)
        self._backward_plain(x)
        ps = list(self.params.values())
        step = self._advance(ps)
        arr = (L.OfParam * len(ps))(*[p.p for p in ps])
        grads = (L.c_void_p * len(ps))(*[p.g.data_ptr() for p in ps])
        self._t0("opt", self.stream)
        L.of_optimizer_step(len(ps), arr, grads, self.opt, self._s())
        self._t1("opt", self.stream)
        for p in ps:
            p.step = step

    def _step_ff(self, x, y):
        pending = [p for op in self.ops if not op.updated for p in op.params]
        if pending:
            step = self._advance(pending)
            for p in pending:
                p.step = step
        self._forward(x, fused=True)
        self._loss(y)
        self._backward_plain(x)
        for op in self.ops:
            op.updated = False

    def flush(self):
        """Apply every update forward-fusion still holds (what the next forward would do)."""
        pending = [p for op in self.ops if not op.updated for p in op.params]
        if pending:
            step = self._advance(pending)
            for p in pending:
                L.of_elementwise_fused_update(p.p, p.g.data_ptr(), 1, 0, self.opt, self._s())
                p.step = step
            for op in self.ops:
                op.updated = True
        self.pending_ordering = None

    def _step_bf(self, x, y):
        # The forward of layer i at this step needs its update from the last step:
        # the previous step ended with the main stream joining the update stream.
        for op in self.ops:
            for p in op.params:
                p.count += 1
        self._forward(x, fused=False)
        self._loss(y)
        step = self._advance(list(self.params.values()))
        timed = self.timer is not None and self.timer.wants("wgrad_bf")
        for i in reversed(range(len(self.ops))):
            op = self.ops[i]
            for p in op.params:
                p.count -= 1
            if any(p.count != 0 for p in op.params):
                raise NotImplementedError("shared parameters are not supported on the GPU path")
            if op.kind == "linear" and not timed:
                # one library call: dgrad with the old W on the main stream, then
                # the fused update on the side stream behind an event
                dx, prev, act_prev = self._dgrad_target(i) if i > 0 else (None, None, 0)
                op.bwd_fused(self, self.gz[i].data_ptr(), self._in(i, x), prev, act_prev, dx)
            else:
                # the same order by hand (events can then bracket the fused kernel):
                # dgrad on the main stream, event, fused wgrad + update on the side
                if i > 0:
                    self._dgrad(i, op)
                ev = torch.cuda.Event()
                ev.record(self.stream)
                self.side.wait_event(ev)
                self._t0("wgrad_bf", self.side, op)
                op.wgrad_fused(self, self.gz[i].data_ptr(), self._in(i, x), self.side.cuda_stream)
                self._t1("wgrad_bf", self.side)
            self._pool_bwd(i)
            for p in op.params:
                p.step = step
        self.side_done.record(self.side)
        self.stream.wait_event(self.side_done)

    # ------------------------------------------------------------- graphs
    def capture(self, x, y, ordering):
        """Capture one steady-state training step on (x, y) as a HIP graph.

        Returns a callable that replays it and advances the host counters as
        step() would.  The step-dependent optimizer constants come from the
        device step counter, so every replay is the next step.  Forward-fusion
        is captured with its pending updates in place (call after one ff step).
        """
        if ordering == "ff" and all(op.updated for op in self.ops):
            raise RuntimeError("capture forward-fusion after one ff step (steady state)")
        if self.pending_ordering == "ff" and ordering != "ff":
            self.flush()
        saved = ([(p.step, p.count) for p in self.params.values()],
                 [op.updated for op in self.ops], self.t, self.pending_ordering)
        g = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream(self.device)
        cap.wait_stream(self.stream)
        main = self.stream
        torch.cuda.synchronize(self.device)
        try:
            self.stream = cap
            with torch.cuda.graph(g, stream=cap):
                self.step(x, y, ordering)
        finally:
            self.stream = main
        flags = [op.updated for op in self.ops]
        for p, (st, cn) in zip(self.params.values(), saved[0]):
            p.step, p.count = st, cn
        for op, u in zip(self.ops, saved[1]):
            op.updated = u
        self.t, self.pending_ordering = saved[2], saved[3]

        def replay():
            g.replay()
            for p in self.params.values():
                p.step += 1
            for op, u in zip(self.ops, flags):
                op.updated = u
            self.pending_ordering = ordering
            self.t += 1

        replay.graph = g
        return replay

    # --------------------------------------------------------------- state
    def load_state(self, params, m, v, step, pending=None):
        """Set parameters, histories (host arrays by name) and step counters.
        pending: optional gradients by name held as forward-fusion's pending
        update (their layers' `updated` flags become False)."""
        torch.cuda.synchronize(self.device)
        for k, p in self.params.items():
            p.w.copy_(torch.as_tensor(np.asarray(params[k], np.float32)))
            p.m.copy_(torch.as_tensor(np.asarray(m[k], np.float32)))
            if p.v is not None:
                p.v.copy_(torch.as_tensor(np.asarray(v[k], np.float32)))
            p.step = int(step[k])
            p.count = 0
        steps = {p.step for p in self.params.values()}
        if len(steps) != 1:
            raise RuntimeError("parameters out of step: this trainer keeps one update counter")
        self.step_dev.fill_(steps.pop())
        for op in self.ops:
            op.updated = True
        self.pending_ordering = None
        if pending:
            for op in self.ops:
                if all(p.name in pending for p in op.params):
                    for p in op.params:
                        p.g.copy_(torch.as_tensor(np.asarray(pending[p.name], np.float32)))
                    op.updated = False
            self.pending_ordering = "ff"
        torch.cuda.synchronize(self.device)

    def loss_history(self):
        torch.cuda.synchronize(self.device)
        return self.losses[: self.t].cpu().numpy().astype(np.float64)

    def argmax(self):
        """Max-pool window positions of the last forward by layer index (synchronises)."""
        torch.cuda.synchronize(self.device)
        return {i: a.cpu().numpy().astype(np.int32) for i, a in enumerate(self.arg)
                if a is not None}

    def state(self):
        """Parameters, histories and counters as host arrays (synchronises)."""
        torch.cuda.synchronize(self.device)
        out = dict(params={}, m={}, v={}, step={}, count={})
        for k, p in self.params.items():
            out["params"][k] = p.w.cpu().numpy()
            out["m"][k] = p.m.cpu().numpy()
            out["v"][k] = p.v.cpu().numpy() if p.v is not None else np.zeros_like(out["m"][k])
            out["step"][k] = p.step
            out["count"][k] = p.count
        out["updated"] = [op.updated for op in self.ops]
        return out

    def eval_loss(self, x, y):
        """Loss of a forward pass at the current (flushed) parameters."""
        if self.pending_ordering == "ff":
            self.flush()
        self.stream.wait_event(self.side_done)
        self._forward(x, fused=False)
        saved = self.t
        self._loss(y)
        torch.cuda.synchronize(self.device)
        return float(self.losses[saved % self.losses.numel()].item())


class KernelTimer:
    """HIP events around chosen launch classes, recorded on the launch's stream."""

    def __init__(self, classes):
        self.classes = set(classes)
        self.records = {c: [] for c in self.classes}
        self._open = {}

    def wants(self, cls):
        return cls in self.classes

    def start(self, cls, stream, op=None):
        if cls in self.classes:
            e = torch.cuda.Event(enable_timing=True)
            e.record(stream)
            self._open[cls] = (e, op)

    def stop(self, cls, stream):
        if cls in self.classes:
            e0, op = self._open.pop(cls)
            e1 = torch.cuda.Event(enable_timing=True)
            e1.record(stream)
            self.records[cls].append((e0, e1, op))

    def clear(self):
        self.records = {c: [] for c in self.classes}

    def durations(self, cls):
        """[(milliseconds, op)] of every recorded launch of `cls` (synchronises)."""
        torch.cuda.synchronize()
        return [(e0.elapsed_time(e1), op) for e0, e1, op in self.records[cls]]

    @staticmethod
    def marker_overhead_ms(stream, samples=50):
        """Mean elapsed time of an event pair with nothing between it on `stream`:
        the cost of the markers themselves, which bracketing a kernel adds."""
        pairs = []
        for _ in range(samples):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            e1.record(stream)
            pairs.append((e0, e1))
        torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in pairs]))
