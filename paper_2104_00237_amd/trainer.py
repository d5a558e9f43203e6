"""Host scheduler: the three training orderings over the opfuse C ABI.

The model is a topologically sorted array of operators (the input of Alg. 2
and Alg. 3); every kernel runs in libopfuse.so, this module only decides
which entry point runs where and keeps the per-parameter state the paper's
algorithms need:

  step[theta]   1-based index of the next update (the optimizer's t)
  updated[f]    Alg. 2 flag: False while f holds a pending update
  count[theta]  Alg. 3 counter: forward uses not yet back-propagated

Orderings (Section 3, Fig. 1(b)-(d)):
  eager  forward; backward writing every gradient; one multi-tensor optimizer
         launch over every parameter.
  ff     forward-fusion: a layer whose `updated` flag is False runs
         of_linear_fwd_fused (the pending update applied while W is loaded);
         backward writes the gradients, which stay pending; flush() applies
         what is still pending.
  bf     backward-fusion: each layer's backward is of_linear_bwd_fused: the
         data gradient with the old W on the main stream, then the weight
         gradient with the optimizer in its epilogue on a second stream, so
         the update of layer i overlaps the back-propagation of layer i-1
         (Section 3, "parallelism"); the next step's forward waits for it.

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


class LinearOp:
    """f_i = act(X W^T + b) on a [M, K] input."""

    def __init__(self, name, W, b, M, act, act_prev):
        N, K = W.w.shape
        self.name, self.W, self.b = name, W, b
        self.M, self.N, self.K = M, N, K
        self.act, self.act_prev = act, act_prev
        self.desc = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.ACTS[act], int(b is not None))
        self.updated = True
        self.params = [W] if b is None else [W, b]

    def ws_bytes(self, op):
        return L.of_linear_workspace_size(self.desc, op)


class Trainer:
    """Trains one workload on one GPU under a chosen ordering."""

    def __init__(self, cfg, init, device="cuda:0"):
        if cfg["kind"] != "mlp":
            raise NotImplementedError(f"model kind {cfg['kind']!r} has no GPU path in this build")
        if cfg["dtype"] != "f32":
            raise NotImplementedError("only fp32 operands in this build")
        L.load()
        self.cfg, self.hyper = cfg, cfg["opt"]
        self.device = torch.device(device)
        kind = self.hyper["kind"]
        M = cfg["batch"]
        dims = cfg["dims"]
        nl = len(dims) - 1
        self.params = {}
        self.ops = []
        for i in range(1, nl + 1):
            W = ParamBuf(f"fc{i}.weight", init[f"fc{i}.weight"], kind, self.device)
            b = ParamBuf(f"fc{i}.bias", init[f"fc{i}.bias"], kind, self.device) if cfg["bias"] else None
            for p in (W, b):
                if p is not None:
                    self.params[p.name] = p
            act = cfg["act"] if i < nl else "none"
            act_prev = cfg["act"] if i > 1 else "none"
            self.ops.append(LinearOp(f"fc{i}", W, b, M, act, act_prev))
        f32 = dict(dtype=torch.float32, device=self.device)
        # a[i]: output of layer i (post-activation); d[i]: gradient w.r.t. Z_i.
        self.a = [None] + [torch.empty(M, op.N, **f32) for op in self.ops]
        self.d = [None] + [torch.empty(M, op.N, **f32) for op in self.ops]
        ws_main = max([op.ws_bytes(L.OF_LINEAR_FWD) for op in self.ops] +
                      [op.ws_bytes(L.OF_LINEAR_BWD_DATA) for op in self.ops] +
                      [op.ws_bytes(L.OF_LINEAR_BWD_WEIGHT) for op in self.ops] + [16])
        ws_side = max([op.ws_bytes(L.OF_LINEAR_BWD_WEIGHT) for op in self.ops] + [16])
        if cfg["loss"] == "mse":
            ws_main = max(ws_main, L.of_mse_workspace_size(M, dims[-1]))
        self.ws_main = torch.empty((ws_main + 15) // 16 * 4, **f32)
        self.ws_side = torch.empty((ws_side + 15) // 16 * 4, **f32)
        self.ws_main_bytes = self.ws_main.numel() * 4
        self.ws_side_bytes = self.ws_side.numel() * 4
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
    def _advance(self, ps):
        """Next update index for parameters ps (host mirror + device counter)."""
        step = ps[0].step + 1
        if any(p.step + 1 != step for p in ps):
            raise RuntimeError("parameters out of step: this trainer keeps one update counter")
        L.of_step_advance(self.step_dev.data_ptr(), 1, self._s())
        return step

    def _s(self):
        return self.stream.cuda_stream

    def _loss(self, y):
        self._t0("loss", self.stream)
        self._loss_launch(y)
        self._t1("loss", self.stream)

    def _loss_launch(self, y):
        out = self.a[-1]
        M, C = out.shape
        loss_ptr = self.losses.data_ptr() + 4 * (self.t % self.losses.numel())
        if self.cfg["loss"] == "xent":
            L.of_xent_fwd_bwd(out.data_ptr(), y.data_ptr(), M, C, 0, loss_ptr,
                              self.d[-1].data_ptr(), self._s())
        else:
            L.of_mse_fwd_bwd(out.data_ptr(), y.data_ptr(), M, C, 0, loss_ptr,
                             self.d[-1].data_ptr(), self.ws_main.data_ptr(), self.ws_main_bytes,
                             self._s())

    def _x(self, i, x):
        return x.data_ptr() if i == 0 else self.a[i].data_ptr()

    def _bias_ptr(self, op):
        return op.b.w.data_ptr() if op.b is not None else None

    def _t0(self, cls, stream, op=None):
        if self.timer is not None:
            self.timer.start(cls, stream, op)

    def _t1(self, cls, stream):
        if self.timer is not None:
            self.timer.stop(cls, stream)

    def _fwd_plain(self, i, op, x):
        self._t0("fwd", self.stream, op)
        L.of_linear_fwd(op.desc, self._x(i, x), op.W.p, self._bias_ptr(op), None,
                        self.a[i + 1].data_ptr(), self.ws_main.data_ptr(), self.ws_main_bytes,
                        self._s())
        self._t1("fwd", self.stream)

    def _bwd_data(self, i, op):
        prev = self.a[i].data_ptr() if op.act_prev != "none" else None
        self._t0("dgrad", self.stream, op)
        L.of_linear_bwd_data(op.desc, self.d[i + 1].data_ptr(), op.W.p, prev,
                             L.ACTS[op.act_prev], self.d[i].data_ptr(), self.ws_main.data_ptr(),
                             self.ws_main_bytes, self._s())
        self._t1("dgrad", self.stream)

    def _bwd_weight(self, i, op, x):
        self._t0("wgrad", self.stream, op)
        L.of_linear_bwd_weight(op.desc, self.d[i + 1].data_ptr(), self._x(i, x),
                               op.W.g.data_ptr(), op.b.g.data_ptr() if op.b is not None else None,
                               0, self.ws_main.data_ptr(), self.ws_main_bytes, self._s())
        self._t1("wgrad", self.stream)

    # ---------------------------------------------------------- orderings
    def step(self, x, y, ordering):
        """One training step on batch (x, y); returns nothing (loss stays on the device)."""
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
        for i, op in enumerate(self.ops):
            self._fwd_plain(i, op, x)
        self._loss(y)
        for i in reversed(range(len(self.ops))):
            op = self.ops[i]
            if i > 0:
                self._bwd_data(i, op)
            self._bwd_weight(i, op, x)
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
        for i, op in enumerate(self.ops):
            if not op.updated:
                b = op.b
                self._t0("fwd_ff", self.stream, op)
                L.of_linear_fwd_fused(op.desc, self._x(i, x), op.W.p, op.W.g.data_ptr(),
                                      b.p if b is not None else None,
                                      b.g.data_ptr() if b is not None else None,
                                      self.opt, None, self.a[i + 1].data_ptr(),
                                      self.ws_main.data_ptr(), self.ws_main_bytes, self._s())
                self._t1("fwd_ff", self.stream)
                for p in op.params:
                    p.step = step
                op.updated = True
            else:
                self._fwd_plain(i, op, x)
        self._loss(y)
        for i in reversed(range(len(self.ops))):
            op = self.ops[i]
            if i > 0:
                self._bwd_data(i, op)
            self._bwd_weight(i, op, x)
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
        for i, op in enumerate(self.ops):
            self._fwd_plain(i, op, x)
            for p in op.params:
                p.count += 1
        self._loss(y)
        side = self.side.cuda_stream
        step = self._advance(list(self.params.values()))
        for i in reversed(range(len(self.ops))):
            op = self.ops[i]
            for p in op.params:
                p.count -= 1
            if any(p.count != 0 for p in op.params):
                raise NotImplementedError("shared parameters are not supported on the GPU path")
            b = op.b
            dx = self.d[i].data_ptr() if i > 0 else None
            prev = self.a[i].data_ptr() if (i > 0 and op.act_prev != "none") else None
            if self.timer is not None and self.timer.wants("wgrad_bf"):
                # Same launches, split so that events can bracket the fused kernel on
                # the update stream: dgrad on S, event, wait, fused wgrad on U.
                if i > 0:
                    self._bwd_data(i, op)
                ev = torch.cuda.Event()
                ev.record(self.stream)
                self.side.wait_event(ev)
                self._t0("wgrad_bf", self.side, op)
                L.of_linear_bwd_fused(op.desc, self.d[i + 1].data_ptr(), self._x(i, x), op.W.p,
                                      b.p if b is not None else None, None, None,
                                      self.opt, None, 0, None, None, 0,
                                      self.ws_side.data_ptr(), self.ws_side_bytes, side, None)
                self._t1("wgrad_bf", self.side)
            else:
                L.of_linear_bwd_fused(op.desc, self.d[i + 1].data_ptr(), self._x(i, x), op.W.p,
                                      b.p if b is not None else None, None, None,
                                      self.opt, prev, L.ACTS[op.act_prev] if i > 0 else 0,
                                      dx, self.ws_main.data_ptr(), self.ws_main_bytes,
                                      self.ws_side.data_ptr(), self.ws_side_bytes, self._s(),
                                      side)
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
        for i, op in enumerate(self.ops):
            self._fwd_plain(i, op, x)
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
