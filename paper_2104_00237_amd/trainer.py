"""Host scheduler: the three training orderings over the opfuse C ABI.

The model is a topologically sorted array of operators (the input of Alg. 2
and Alg. 3): a chain of linear or 3x3-convolution layers, each followed by
its activation (fused into the kernel's epilogue) and optionally by a 2x2
max-pool, or pre-LN residual blocks of LayerNorm and bf16-operand linears.
Every kernel runs in libopfuse.so; this module only decides which entry point
runs where and keeps the per-parameter state the paper's algorithms need:

  step[theta]   1-based index of the update applied last (mirrored on the device)
  updated[f]    Alg. 2 flag: False while f holds a pending update
  count[theta]  Alg. 3 counter: forward uses not yet back-propagated

Orderings (Section 3, Fig. 1(b)-(d)):
  eager  forward; backward writing every gradient; one multi-tensor optimizer
         launch over every parameter.
  ff     forward-fusion: a layer whose `updated` flag is False applies its
         pending update in its forward (fp32 linear layers: of_linear_fwd_fused,
         while the W tiles load; convolutions, LayerNorms and bf16 linears: an
         element-wise pass right before the forward); backward writes the
         gradients, which stay pending; flush() applies what is still pending.
  bf     backward-fusion: each layer's data gradient runs with the old weights
         on the main stream, then its weight-gradient kernel with the
         optimizer in the epilogue runs on a second stream, so the update of
         layer i overlaps the back-propagation of layer i-1 (Section 3,
         "parallelism"); the next step's forward waits for it.

Torch is used for device memory, streams and events only.
"""
import ctypes

import numpy as np
import torch

from . import _lib as L


def _bf16_bits(a):
    """bf16 bits (round to nearest even) of fp32 values, as int16 for torch."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(np.asarray(a, np.float32))
    r[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return r.view(np.int16)


class ParamBuf:
    """A trainable tensor on the device with its history and host counters.

    g holds the gradient as one vector (eager, and forward-fusion's pending
    gradient); a LayerNorm parameter also has `rows`, its gradient as row-group
    partials [G, numel] (summed by the fused update, or reduced into g).
    A bf16-operand weight also keeps its bf16 shadow `wb`.
    """

    def __init__(self, name, value, kind, device, shadow=False, rows=0):
        self.name = name
        self.w = torch.as_tensor(np.ascontiguousarray(value, dtype=np.float32)).to(device)
        self.m = torch.zeros_like(self.w)
        self.v = torch.zeros_like(self.w) if kind != "sgd" else None
        self.g = torch.zeros_like(self.w)
        self.wb = torch.as_tensor(_bf16_bits(value)).to(device) if shadow else None
        self.rows = (torch.zeros((rows,) + tuple(self.w.shape), dtype=torch.float32, device=device)
                     if rows else None)
        self.p = L.param_of(self.w, self.m, self.v, self.wb)
        self.step = 0
        self.count = 0

    @property
    def numel(self):
        return self.w.numel()

    def pending(self):
        """(device pointer, rows, row stride) of the gradient an update consumes."""
        if self.rows is not None:
            return self.rows.data_ptr(), self.rows.shape[0], self.numel
        return self.g.data_ptr(), 1, 0

    def swap_generation(self):
        """Make the second buffer set (written by a fused convolution forward)
        the current one; the old set becomes the next step's output.  Allocated
        on first use."""
        if getattr(self, "_alt", None) is None:
            w2 = torch.empty_like(self.w)
            m2 = torch.empty_like(self.m)
            v2 = torch.empty_like(self.v) if self.v is not None else None
            p2 = L.param_of(w2, m2, v2)
            if self.p.m is None:      # an optimizer without m keeps none
                p2.m = None
            self._alt = (w2, m2, v2, p2)
        w2, m2, v2, p2 = self._alt
        self._alt = (self.w, self.m, self.v, self.p)
        self.w, self.m, self.v, self.p = w2, m2, v2, p2

    def alt_param(self):
        """of_param of the buffer set the next fused convolution forward writes."""
        if getattr(self, "_alt", None) is None:
            self.swap_generation()
            self.swap_generation()   # allocate, keep the current set current
        return self._alt[3]

    def set(self, value):
        self.w.copy_(torch.as_tensor(np.asarray(value, np.float32)))
        if self.wb is not None:
            self.wb.copy_(torch.as_tensor(_bf16_bits(np.asarray(value, np.float32))))

    def set_pending(self, g):
        g = torch.as_tensor(np.asarray(g, np.float32))
        if self.rows is not None:
            self.rows.zero_()
            self.rows[0].copy_(g)
        else:
            self.g.copy_(g)


def _unique(ps):
    """Parameters in first-use order, each once (a shared operator is listed once
    per use)."""
    seen, out = set(), []
    for p in ps:
        if id(p) not in seen:
            seen.add(id(p))
            out.append(p)
    return out


def _ptr(t):
    return t.data_ptr() if t is not None else None


def _update(tr, p, stream):
    """Element-wise fused update of p from its pending gradient (a7)."""
    ptr, rows, ld = p.pending()
    L.of_elementwise_fused_update(p.p, ptr, rows, ld, tr.opt, stream)


def _self_update(tr, params):
    """Forward-fusion of an operator no earlier launch carried: its pending
    update as its own pass right before its forward (one launch for vector
    gradients, a7 per row-partial gradient)."""
    vec = [p for p in params if p.rows is None]
    if vec:
        arr = (L.OfParam * len(vec))(*[p.p for p in vec])
        gp = (ctypes.c_void_p * len(vec))(*[p.g.data_ptr() for p in vec])
        L.of_optimizer_step(len(vec), arr, gp, tr.opt, tr._s())
    for p in params:
        if p.rows is not None:
            _update(tr, p, tr._s())


def _carry_of(tr, params):
    """of_carry of parameters (at most OF_CARRY_MAX) with their pending gradients."""
    return L.make_carry(tr.opt, [(p.p, p.pending()[0], p.pending()[1]) for p in params])


class LinearOp:
    """f = act(X W^T + b) on a [M, K] input (row stride ldx)."""

    kind = "linear"

    def __init__(self, name, W, b, M, act, dtype=L.OF_F32, ldx=0, io=0):
        N, K = W.w.shape
        self.name, self.W, self.b = name, W, b
        self.M, self.N, self.K = M, N, K
        self.act = act
        self.desc = L.OfLinearDesc(M, N, K, ldx, 0, dtype, L.ACTS[act], int(b is not None), io)
        self.updated = True
        self.params = [W] if b is None else [W, b]
        self.out_shape = (M, N)
        # Forward-fusion: an fp32 layer with M <= 64 rows applies its pending
        # update while its own W tiles load (one row tile covers M); any other
        # layer has it carried by the previous operator's forward launch.
        self.fp32 = dtype == L.OF_F32
        self.prologue_ff = self.fp32 and M <= 64
        # Backward-fusion overlaps the fused update with the next data gradient
        # on a second stream when the update is heavy enough (>= 4M parameters or
        # >= 4 GFLOP) to repay the event pair that orders it; a lighter update runs
        # in stream order right after its layer's data gradient (measured on
        # MI355X: with 1024x1024 layers the two-stream step is bound by its host
        # calls, and the overlap gains less than they cost).
        self.overlap_update = N * K >= (1 << 22) or 2.0 * M * N * K >= 4e9
        # Backward-fusion with the data gradient merged into the update's read
        # of W (of_linear_bwd_merged): fp32 layers with M <= 64 rows, when the
        # trainer asks for it.
        self.merge_ok = dtype == L.OF_F32 and M <= 64
        self.merge_dgrad = False

    def ws(self, which):
        if which == L.OF_LINEAR_BWD_MERGED and not self.merge_ok:
            return 0
        return L.of_linear_workspace_size(self.desc, which)

    def fwd(self, tr, x, y, z=None, carry=None, res=None):
        """y = act(x W^T + b) (+ res, a residual connection added in the epilogue)."""
        b = _ptr(self.b.w) if self.b else None
        if res is not None:
            L.of_linear_fwd_res(self.desc, x, self.W.p, b, res, z, y, carry, *tr.ws_main_args(),
                                tr._s())
        elif carry is None:
            L.of_linear_fwd(self.desc, x, self.W.p, b, z, y, *tr.ws_main_args(), tr._s())
        else:
            L.of_linear_fwd_carry(self.desc, x, self.W.p, b, z, y, carry, *tr.ws_main_args(),
                                  tr._s())

    def two_sets(self):
        """Whether this operator's prologue alternates two parameter buffer sets."""
        return self.prologue_ff and self.M > 64

    def fwd_ff(self, tr, x, y, z=None):
        """Forward-fusion in the W-tile prologue: in place when the M rows fit one
        row tile, else into the second buffer set, which then becomes current."""
        b = self.b
        two_sets = self.M > 64
        L.of_linear_fwd_fused(self.desc, x, self.W.p, self.W.alt_param() if two_sets else None,
                              self.W.g.data_ptr(), b.p if b else None,
                              b.alt_param() if (b and two_sets) else None,
                              b.g.data_ptr() if b else None, tr.opt, z, y,
                              *tr.ws_main_args(), tr._s())
        if two_sets:
            for p in self.params:
                p.swap_generation()

    def dgrad(self, tr, g, prev, act_prev, dx, res=None):
        """dx = (g W) * act_prev'(prev) (+ res, a skip connection's gradient)."""
        if res is None:
            L.of_linear_bwd_data(self.desc, g, self.W.p, prev, act_prev, dx, *tr.ws_main_args(),
                                 tr._s())
        else:
            L.of_linear_bwd_data_res(self.desc, g, self.W.p, prev, act_prev, res, dx,
                                     *tr.ws_main_args(), tr._s())

    def wgrad(self, tr, g, x, accumulate=0, side=False):
        """Plain weight gradient into W.g (and b.g); accumulate=1 adds to what an
        earlier use of a shared parameter left there.  side: on the second
        stream, with its workspace."""
        L.of_linear_bwd_weight(self.desc, g, x, self.W.g.data_ptr(),
                               self.b.g.data_ptr() if self.b else None, accumulate,
                               *_ws_args(tr, side), _stream(tr, side))

    def _partials(self, partial):
        """(gW, gb) of earlier uses of a shared parameter for the fused update."""
        if not partial:
            return None, None
        return self.W.g.data_ptr(), (self.b.g.data_ptr() if self.b else None)

    def wgrad_fused(self, tr, g, x, stream, partial=False):
        b = self.b
        L.of_linear_bwd_fused(self.desc, g, x, self.W.p, b.p if b else None,
                              *self._partials(partial), tr.opt, None, 0, None, None, 0,
                              *tr.ws_side_args(), stream, None)

    def bwd_merged(self, tr, g, x, prev, act_prev, dx, partial=False):
        """Data gradient (old W) and fused update in one pass over W, m, v."""
        b = self.b
        L.of_linear_bwd_merged(self.desc, g, x, self.W.p, b.p if b else None,
                               *self._partials(partial), tr.opt, prev, act_prev, dx,
                               *tr.ws_main_args(), tr._s())

    def bwd_fused(self, tr, g, x, prev, act_prev, dx, partial=False, res=None):
        """Data gradient on the main stream, then the fused update: on the side
        stream (behind an event) or in stream order (one call).  res: a skip
        connection's gradient added to dx (then the data gradient is its own
        call, and the fused call only updates)."""
        b = self.b
        if res is not None:
            self.dgrad(tr, g, prev, act_prev, dx, res=res)
            prev, act_prev, dx = None, 0, None
        L.of_linear_bwd_fused(self.desc, g, x, self.W.p, b.p if b else None,
                              *self._partials(partial), tr.opt, prev, act_prev, dx,
                              *tr.ws_main_args(), *tr.ws_side_args(), tr._s(),
                              tr.side.cuda_stream if self.overlap_update else None)


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

    # Forward-fusion in the filter-tile prologue (of_conv_fwd_fused, when the
    # trainer asks for it): every workgroup updates its filter tile in
    # registers from the current buffers, the first pixel-row tile writes it to
    # the other buffer set, which becomes current.  Every pixel-row tile re-reads
    # the filter's gradient and history, so by default the update is carried by
    # the previous launch instead (measured faster on VGG-11); a captured step
    # keeps the buffers fixed and always carries it.  Same values either way.
    prologue_ff = False
    overlap_update = True  # a convolution's fused wgrad + update is heavy: second stream

    def two_sets(self):
        """The filter-tile prologue always alternates two buffer sets."""
        return self.prologue_ff

    def fwd(self, tr, x, y, carry=None):
        if carry is None:
            L.of_conv_fwd(self.desc, x, self.W.p, _ptr(self.b.w) if self.b else None, y,
                          *tr.ws_main_args(), tr._s())
        else:
            L.of_conv_fwd_carry(self.desc, x, self.W.p, _ptr(self.b.w) if self.b else None, y,
                                carry, *tr.ws_main_args(), tr._s())

    def fwd_ff(self, tr, x, y):
        b = self.b
        L.of_conv_fwd_fused(self.desc, x, self.W.p, self.W.alt_param(), self.W.g.data_ptr(),
                            b.p if b else None, b.alt_param() if b else None,
                            b.g.data_ptr() if b else None, tr.opt, y, *tr.ws_main_args(),
                            tr._s())
        for p in self.params:
            p.swap_generation()

    def dgrad(self, tr, g, prev, act_prev, dx):
        L.of_conv_bwd_data(self.desc, g, self.W.p, prev, act_prev, dx, *tr.ws_main_args(),
                           tr._s())

    def wgrad(self, tr, g, x, accumulate=0, side=False):
        L.of_conv_bwd_weight(self.desc, g, x, self.W.g.data_ptr(),
                             self.b.g.data_ptr() if self.b else None, accumulate,
                             *_ws_args(tr, side), _stream(tr, side))

    def wgrad_fused(self, tr, g, x, stream, partial=False):
        """Fused weight gradient + update; partial: add the gradient earlier uses
        of a shared filter left in W.g / b.g."""
        b = self.b
        gw = self.W.g.data_ptr() if partial else None
        gb = b.g.data_ptr() if (partial and b) else None
        L.of_conv_wgrad_fused(self.desc, g, x, self.W.p, b.p if b else None, gw, gb, tr.opt,
                              *tr.ws_side_args(), stream)


class DwOp:
    """f = act(dwconv3x3(X, W, stride) + b) on an NHWC [N, H, W, C] input: one 3x3
    filter per channel (MobileNetV2's depthwise layers)."""

    kind = "dw"
    prologue_ff = False      # its update is carried by the previous launch
    overlap_update = False   # a few thousand parameters: updated in stream order

    def __init__(self, name, W, b, N, H, Wd, C, stride, act):
        self.name, self.W, self.b = name, W, b
        self.act = act
        self.desc = L.OfConvDesc(N, H, Wd, C, C, L.ACTS[act], int(b is not None), stride)
        self.updated = True
        self.params = [W] if b is None else [W, b]
        Ho, Wo = (H - 1) // stride + 1, (Wd - 1) // stride + 1
        self.out_shape = (N, Ho, Wo, C)
        self.M, self.N, self.K = N * Ho * Wo, C, 9

    def two_sets(self):
        return False

    def ws(self, which):
        return L.of_dwconv_workspace_size(self.desc) if which == L.OF_LINEAR_BWD_WEIGHT else 0

    def fwd(self, tr, x, y):
        L.of_dwconv_fwd(self.desc, x, self.W.w.data_ptr(), _ptr(self.b.w) if self.b else None, y,
                        tr._s())

    def dgrad(self, tr, g, prev, act_prev, dx):
        L.of_dwconv_bwd_data(self.desc, g, self.W.w.data_ptr(), prev, act_prev, dx, tr._s())

    def wgrad(self, tr, g, x, accumulate=0, side=False):
        L.of_dwconv_bwd_weight(self.desc, g, x, self.W.g.data_ptr(),
                               self.b.g.data_ptr() if self.b else None, accumulate,
                               *_ws_args(tr, side), _stream(tr, side))

    def wgrad_fused(self, tr, g, x, stream, partial=False):
        b = self.b
        side = stream == tr.side.cuda_stream
        L.of_dwconv_wgrad_fused(self.desc, g, x, self.W.p, b.p if b else None,
                                self.W.g.data_ptr() if partial else None,
                                (b.g.data_ptr() if (b and partial) else None), tr.opt,
                                *_ws_args(tr, side), stream)


class LayerNormOp:
    """f = LayerNorm(X) * gamma + beta over the last dimension of [M, D]."""

    kind = "ln"

    def __init__(self, name, g, b, M, D, eps, y_bf16=False):
        self.name, self.g, self.b = name, g, b
        self.M, self.D, self.eps = M, D, eps
        self.N, self.K = D, 0
        self.updated = True
        self.params = [g, b]
        self.y_bf16 = y_bf16    # the output is stored as bf16 (only bf16 operands read it)

    def ws(self, which):
        return 0

    def fwd(self, tr, x, y, mu, rs):
        fn = L.of_layernorm_fwd_bf16 if self.y_bf16 else L.of_layernorm_fwd
        fn(x, self.M, self.D, self.g.w.data_ptr(), self.b.w.data_ptr(), self.eps, y, mu, rs,
           tr._s())

    prologue_ff = False   # gamma and beta are carried by the previous launch, or updated first

    def two_sets(self):
        return False

    def bwd(self, tr, dy, x, mu, rs, dres, dx, side=None, params=True):
        """dx (+ dres) on the main stream and, unless params is False, the
        parameter-gradient row partials: on the stream `side` when given (already
        ordered after dy; both launches only read dy and x), else in the same
        call as dx."""
        if side is None and params:
            L.of_layernorm_bwd(dy, x, mu, rs, self.g.w.data_ptr(), dres, self.M, self.D, dx,
                               self.g.rows.data_ptr(), self.b.rows.data_ptr(), tr._s())
            return
        if params:
            self.bwd_params(dy, x, mu, rs, side)
        L.of_layernorm_bwd(dy, x, mu, rs, self.g.w.data_ptr(), dres, self.M, self.D, dx, None,
                           None, tr._s())

    def bwd_params(self, dy, x, mu, rs, stream):
        """The parameter-gradient row partials alone, on `stream`."""
        L.of_layernorm_bwd(dy, x, mu, rs, None, None, self.M, self.D, None,
                           self.g.rows.data_ptr(), self.b.rows.data_ptr(), stream)

    def reduce(self, tr, stream=None):
        """Eager: materialise the gradient vectors from the row partials."""
        for p in self.params:
            L.of_reduce_rows(p.rows.data_ptr(), p.rows.shape[0], 0, p.numel, p.g.data_ptr(),
                             stream if stream is not None else tr._s())


def _ff_prologue(tr, op):
    """Whether forward-fusion applies op's pending update in its forward's W-tile
    loads (else a previous launch carries it, or a pass of its own runs)."""
    return op.prologue_ff and not (op.two_sets() and tr.capturing)


# One side stream and one capture stream per device, made once.  HIP maps each
# new stream onto one of a few hardware queues; a side stream made per trainer
# can land on the main stream's queue, and its work then no longer overlaps
# (measured: steps alternating between 4.0 and 4.9 ms on the MobileNetV2-like
# network from one trainer to the next).  Streams keep the default priority.
_STREAMS = {}


def device_stream(device, role):
    key = (str(device), role)
    if key not in _STREAMS:
        _STREAMS[key] = torch.cuda.Stream(device)
    return _STREAMS[key]


def _ws_args(tr, side):
    return tr.ws_side_args() if side else tr.ws_main_args()


def _stream(tr, side):
    return tr.side.cuda_stream if side else tr._s()


def _side_after_main(tr):
    """Order the side stream after everything enqueued so far on the main stream;
    returns the event it waits for."""
    ev = torch.cuda.Event(enable_timing=tr.timer is not None)
    ev.record(tr.stream)
    tr.side.wait_event(ev)
    return ev


class ChainNet:
    """Linear / conv layers in a chain, each with its activation and an
    optional 2x2 max-pool after it (the MLP and VGG workloads)."""

    side_updates = False   # only layers with overlap_update use the side stream

    def __init__(self, tr, cfg, pb):
        self.tr = tr
        self.ops, self.pool = [], []
        if cfg["kind"] == "mlp":
            M, dims = cfg["batch"], cfg["dims"]
            nl = len(dims) - 1
            tie = {int(k): int(v) for k, v in cfg.get("tie", {}).items()}
            for i in range(1, nl + 1):
                act = cfg["act"] if i < nl else "none"
                if i in tie:
                    # the same operator applied again (Alg. 2 / Alg. 3 shared parameters)
                    if not 1 <= tie[i] < i or (dims[i - 1], dims[i]) != (dims[tie[i] - 1], dims[tie[i]]):
                        raise ValueError(f"layer {i} cannot apply layer {tie[i]}'s parameters")
                    src = self.ops[tie[i] - 1]
                    if src.act != act:
                        raise NotImplementedError("a tied layer must have its source's activation")
                    self.ops.append(src)
                else:
                    W = pb(f"fc{i}.weight")
                    b = pb(f"fc{i}.bias") if cfg["bias"] else None
                    self.ops.append(LinearOp(f"fc{i}", W, b, M, act))
                self.pool.append(False)
        else:
            N, s = cfg["batch"], cfg["image"]
            for i, cout in enumerate(cfg["channels"], start=1):
                W, b = pb(f"conv{i}.weight"), pb(f"conv{i}.bias")
                self.ops.append(ConvOp(f"conv{i}", W, b, N, s, s, "relu"))
                pool = i in cfg["pool_after"]
                self.pool.append(pool)
                if pool:
                    s //= 2
            if s != 1:
                raise NotImplementedError("the classifier expects a 1x1 feature map")
            self.ops.append(LinearOp("fc", pb("fc.weight"), pb("fc.bias"), N, "none"))
            self.pool.append(False)
        dev = tr.device
        f32 = dict(dtype=torch.float32, device=dev)
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
                self.arg[i] = torch.empty(ps, dtype=torch.uint8, device=dev)
                self.gp[i] = torch.empty(ps, **f32)
        self.out, self.gout = self.y[-1], self.gz[-1]

    def _in(self, i, x):
        """Device pointer of layer i's input."""
        if i == 0:
            return x.data_ptr()
        return (self.p[i - 1] if self.pool[i - 1] else self.y[i - 1]).data_ptr()

    def forward(self, x, fused):
        tr = self.tr
        n = len(self.ops)
        for i, op in enumerate(self.ops):
            if fused and not op.updated and _ff_prologue(tr, op):
                tr._t0("fwd_ff", tr.stream, op)
                op.fwd_ff(tr, self._in(i, x), self.y[i].data_ptr())
                tr._t1("fwd_ff", tr.stream)
                op.updated = True
            else:
                if fused and not op.updated:
                    _self_update(tr, op.params)   # no earlier launch carried it
                    op.updated = True
                nxt = self.ops[i + 1] if i + 1 < n else None
                carry = None
                if fused and nxt is not None and not nxt.updated and not _ff_prologue(tr, nxt):
                    carry = _carry_of(tr, nxt.params)
                tr._t0("fwd", tr.stream, op)
                op.fwd(tr, self._in(i, x), self.y[i].data_ptr(), carry=carry)
                tr._t1("fwd", tr.stream)
                if carry is not None:
                    nxt.updated = True   # its update is enqueued with this launch
            if self.pool[i]:
                N, H, W, C = op.out_shape
                L.of_maxpool2x2_fwd(self.y[i].data_ptr(), N, H, W, C, self.p[i].data_ptr(),
                                    self.arg[i].data_ptr(), tr._s())

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
                                self.gz[i - 1].data_ptr(), self.tr._s())

    def _dgrad(self, i, op):
        tr = self.tr
        dx, prev, act_prev = self._dgrad_target(i)
        tr._t0("dgrad", tr.stream, op)
        op.dgrad(tr, self.gz[i].data_ptr(), prev, act_prev, dx)
        tr._t1("dgrad", tr.stream)

    def backward_plain(self, x):
        tr = self.tr
        seen = set()   # operators whose gradient this backward pass has started
        for i in reversed(range(len(self.ops))):
            op = self.ops[i]
            if i > 0:
                self._dgrad(i, op)
            tr._t0("wgrad", tr.stream, op)
            op.wgrad(tr, self.gz[i].data_ptr(), self._in(i, x), int(id(op) in seen))
            tr._t1("wgrad", tr.stream)
            seen.add(id(op))
            self._pool_bwd(i)

    def backward_fused(self, x, done):
        """Backward-fusion: `done(op)` is called after each layer's update is enqueued."""
        tr = self.tr
        timed = tr.timer is not None and (tr.timer.wants("wgrad_bf") or tr.timer.wants("dgrad"))
        seen = set()
        for i in reversed(range(len(self.ops))):
            op = self.ops[i]
            partial = id(op) in seen          # earlier uses' gradient is in W.g / b.g
            seen.add(id(op))
            if any(p.count > 1 for p in op.params):
                # A shared parameter with backward uses still to come (Alg. 3:
                # count > 0 after this one): its data gradient with the old W and
                # its weight gradient into the gradient buffer; the last use
                # updates.
                if i > 0:
                    self._dgrad(i, op)
                tr._t0("wgrad", tr.stream, op)
                op.wgrad(tr, self.gz[i].data_ptr(), self._in(i, x), int(partial))
                tr._t1("wgrad", tr.stream)
            elif op.kind == "linear" and op.merge_dgrad:
                # one kernel reads W once for the data gradient and the update
                dx, prev, act_prev = self._dgrad_target(i) if i > 0 else (None, None, 0)
                tr._t0("wgrad_bf", tr.stream, op)
                op.bwd_merged(tr, self.gz[i].data_ptr(), self._in(i, x), prev, act_prev, dx,
                              partial)
                tr._t1("wgrad_bf", tr.stream)
            elif op.kind == "linear" and not timed:
                # one library call: dgrad with the old W on the main stream, then
                # the fused update on the side stream behind an event
                dx, prev, act_prev = self._dgrad_target(i) if i > 0 else (None, None, 0)
                op.bwd_fused(tr, self.gz[i].data_ptr(), self._in(i, x), prev, act_prev, dx,
                             partial)
            else:
                # the same order by hand (events can then bracket the fused kernel):
                # dgrad on the main stream, then the fused wgrad + update, behind
                # an event on the side stream or in order on the main one
                if i > 0:
                    self._dgrad(i, op)
                if op.overlap_update:
                    gate = _side_after_main(tr)
                    tr._t0_after("wgrad_bf", tr.side, op, gate)
                    op.wgrad_fused(tr, self.gz[i].data_ptr(), self._in(i, x), tr.side.cuda_stream,
                                   partial)
                    tr._t1("wgrad_bf", tr.side)
                else:
                    tr._t0("wgrad_bf", tr.stream, op)
                    op.wgrad_fused(tr, self.gz[i].data_ptr(), self._in(i, x), tr._s(), partial)
                    tr._t1("wgrad_bf", tr.stream)
            self._pool_bwd(i)
            done(op)

    def argmax(self):
        return {i: a for i, a in enumerate(self.arg) if a is not None}


class TBlockNet:
    """Pre-LN residual blocks with bf16-operand linears (the tblock workload):

        a = LN1(x); qkv = a Wqkv^T + b; v = qkv[:, 2d:3d]   (identity attention)
        h = x + v Wproj^T + b
        c = LN2(h); u = c W1^T + b; g = GELU(u); y = h + g W2^T + b

    Every tensor a later kernel reads is kept per block, and so is every
    gradient buffer, so the side stream's fused updates of block b never race
    with the main stream's back-propagation through the blocks below.  With
    bf16 operands, a, qkv, c and g are read by the bf16 contractions alone
    (forward and weight gradient; GELU's derivative reads u), so their
    producers store them as bf16 (`bf16_acts`): the rounding each contraction
    would apply, so results are bit-identical, in half the bytes.  In the
    plain backward (eager and forward-fusion) the LayerNorm parameter-gradient
    partials run on the side stream, so those steps join it before their
    optimizer step, clipping norm or next forward; backward-fusion computes
    them, and updates gamma and beta, on a second side stream.
    """

    eager_side = True

    def __init__(self, tr, cfg, pb, bf16_acts=True):
        self.tr = tr
        M, d, f, nb = cfg["batch"], cfg["hidden"], cfg["ffn"], cfg["blocks"]
        self.M, self.d, self.f = M, d, f
        dt = L.OF_BF16 if cfg["dtype"] == "bf16" else L.OF_F32
        eps = cfg["ln_eps"]
        G = L.of_layernorm_partial_rows(M)
        shadow = dt == L.OF_BF16
        acts = shadow and bf16_acts
        xb = L.OF_IO_X_BF16 if acts else 0
        yb = L.OF_IO_Y_BF16 if acts else 0
        self.blocks = []
        self.ops = []
        for b in range(1, nb + 1):
            p = f"blk{b}."
            blk = dict(
                ln1=LayerNormOp(p + "ln1", pb(p + "ln1.weight", rows=G), pb(p + "ln1.bias", rows=G),
                                M, d, eps, y_bf16=acts),
                qkv=LinearOp(p + "qkv", pb(p + "qkv.weight", shadow), pb(p + "qkv.bias"), M, "none",
                             dt, io=xb | yb),
                proj=LinearOp(p + "proj", pb(p + "proj.weight", shadow), pb(p + "proj.bias"), M,
                              "none", dt, ldx=3 * d, io=xb),
                ln2=LayerNormOp(p + "ln2", pb(p + "ln2.weight", rows=G), pb(p + "ln2.bias", rows=G),
                                M, d, eps, y_bf16=acts),
                fc1=LinearOp(p + "fc1", pb(p + "fc1.weight", shadow), pb(p + "fc1.bias"), M, "gelu",
                             dt, io=xb | yb),
                fc2=LinearOp(p + "fc2", pb(p + "fc2.weight", shadow), pb(p + "fc2.bias"), M, "none",
                             dt, io=xb),
            )
            self.ops += [blk[k] for k in ("ln1", "qkv", "proj", "ln2", "fc1", "fc2")]
            self.blocks.append(blk)
        f32 = dict(dtype=torch.float32, device=tr.device)
        act = dict(dtype=torch.bfloat16 if acts else torch.float32, device=tr.device)

        def t(*shape):
            return torch.empty(shape, **f32)

        def ta(*shape):   # read only as a bf16 matmul operand
            return torch.empty(shape, **act)

        for blk in self.blocks:
            blk.update(a=ta(M, d), mu1=t(M), rs1=t(M), qkv_out=ta(M, 3 * d), h=t(M, d),
                       c=ta(M, d), mu2=t(M), rs2=t(M), u=t(M, f), g=ta(M, f), y=t(M, d),
                       gy=t(M, d), gu=t(M, f), gc=t(M, d), gh=t(M, d), ga=t(M, d),
                       # the Q and K thirds of the QKV gradient stay zero
                       gqkv=torch.zeros((M, 3 * d), **f32))
        self.gx = t(M, d)   # gradient w.r.t. the network input (not used further)
        self.out = self.blocks[-1]["y"]
        self.gout = self.blocks[-1]["gy"]

    def _v(self, blk):
        """Address of the V third of the block's QKV output."""
        q = blk["qkv_out"]
        return q.data_ptr() + 2 * self.d * q.element_size()

    def forward(self, x, fused):
        tr = self.tr
        xin = x.data_ptr()
        order = [(b, name) for b in range(len(self.blocks))
                 for name in ("ln1", "qkv", "proj", "ln2", "fc1", "fc2")]
        for k, (bi, name) in enumerate(order):
            blk = self.blocks[bi]
            op = blk[name]
            if fused and not op.updated:
                _self_update(tr, op.params)   # no earlier launch carried it
                op.updated = True
            # A linear's launch carries the next operators' pending updates: the
            # next one, and through a LayerNorm (whose kernel carries nothing)
            # the one after it too.
            carry, carried = None, []
            if fused and name not in ("ln1", "ln2"):
                k2 = k + 1
                while k2 < len(order) and len(carried) < 2:
                    nb, nn = order[k2]
                    nxt = self.blocks[nb][nn]
                    if nxt.updated:
                        break
                    carried.append(nxt)
                    if nn not in ("ln1", "ln2"):
                        break
                    k2 += 1
                if carried:
                    carry = _carry_of(tr, [p for o in carried for p in o.params])
            tr._t0("fwd", tr.stream, op)
            if name == "ln1":
                op.fwd(tr, xin, blk["a"].data_ptr(), blk["mu1"].data_ptr(), blk["rs1"].data_ptr())
            elif name == "qkv":
                op.fwd(tr, blk["a"].data_ptr(), blk["qkv_out"].data_ptr(), carry=carry)
            elif name == "proj":     # h = x + attention output (residual in the epilogue)
                op.fwd(tr, self._v(blk), blk["h"].data_ptr(), carry=carry, res=xin)
            elif name == "ln2":
                op.fwd(tr, blk["h"].data_ptr(), blk["c"].data_ptr(), blk["mu2"].data_ptr(),
                       blk["rs2"].data_ptr())
            elif name == "fc1":
                op.fwd(tr, blk["c"].data_ptr(), blk["g"].data_ptr(), blk["u"].data_ptr(),
                       carry=carry)
            else:                    # y = h + MLP output, the next block's input
                op.fwd(tr, blk["g"].data_ptr(), blk["y"].data_ptr(), carry=carry,
                       res=blk["h"].data_ptr())
            tr._t1("fwd", tr.stream)
            for o in carried:
                o.updated = True     # their updates are enqueued with this launch
            if name == "fc2":
                xin = blk["y"].data_ptr()

    def _block_in(self, k, x):
        return x.data_ptr() if k == 0 else self.blocks[k - 1]["y"].data_ptr()

    def _gx_of(self, k):
        return self.gx.data_ptr() if k == 0 else self.blocks[k - 1]["gy"].data_ptr()

    def _linear_bwd(self, op, dz, x, prev, act_prev, dx, fused, done):
        tr = self.tr
        if not fused:
            tr._t0("dgrad", tr.stream, op)
            op.dgrad(tr, dz, prev, act_prev, dx)
            tr._t1("dgrad", tr.stream)
            tr._t0("wgrad", tr.stream, op)
            op.wgrad(tr, dz, x)
            tr._t1("wgrad", tr.stream)
        elif tr.timer is not None and (tr.timer.wants("wgrad_bf") or tr.timer.wants("dgrad")):
            tr._t0("dgrad", tr.stream, op)
            op.dgrad(tr, dz, prev, act_prev, dx)
            tr._t1("dgrad", tr.stream)
            if op.overlap_update:
                gate = _side_after_main(tr)
                tr._t0_after("wgrad_bf", tr.side, op, gate)
                op.wgrad_fused(tr, dz, x, tr.side.cuda_stream)
                tr._t1("wgrad_bf", tr.side)
            else:
                tr._t0("wgrad_bf", tr.stream, op)
                op.wgrad_fused(tr, dz, x, tr._s())
                tr._t1("wgrad_bf", tr.stream)
            done(op)
        else:
            op.bwd_fused(tr, dz, x, prev, act_prev, dx)
            done(op)

    def _ln_bwd(self, op, dy, x, mu, rs, dres, dx, fused, done):
        tr = self.tr
        if fused:
            # Backward-fusion's side stream already carries the fused weight
            # gradients of the linears, so the partials and the update of gamma
            # and beta take a second one: the partials once dy exists, the
            # update once dx has read the old gamma (the dependency rule of
            # Alg. 3).  The step's end joins it (measured on tblock12:
            # 10.67 -> 10.53 ms per step against the partials on the main
            # stream after dx).
            side2 = tr.side2()
            ev = torch.cuda.Event()
            ev.record(tr.stream)
            side2.wait_event(ev)
            op.bwd_params(dy, x, mu, rs, side2.cuda_stream)
            tr._t0("ln_bwd", tr.stream, op)
            op.bwd(tr, dy, x, mu, rs, dres, dx, side=None, params=False)
            tr._t1("ln_bwd", tr.stream)
            ev = torch.cuda.Event()
            ev.record(tr.stream)
            side2.wait_event(ev)
            for p in op.params:
                _update(tr, p, side2.cuda_stream)
            done(op)
            return
        # Plain backward: the partials, and after them the eager reduce, run on
        # the side stream beside the data gradient; the step joins it before
        # the optimizer step (eager) or the next forward (forward-fusion), and
        # no later kernel of the step writes dy, x or the row statistics.
        _side_after_main(tr)
        tr._t0("ln_bwd", tr.stream, op)
        op.bwd(tr, dy, x, mu, rs, dres, dx, side=tr.side.cuda_stream)
        tr._t1("ln_bwd", tr.stream)
        if tr.eager_reduce:
            op.reduce(tr, tr.side.cuda_stream)

    def _backward(self, x, fused, done):
        d = self.d
        for k in reversed(range(len(self.blocks))):
            blk = self.blocks[k]
            P = {n: blk[n].data_ptr() for n in blk if isinstance(blk[n], torch.Tensor)}
            self._linear_bwd(blk["fc2"], P["gy"], P["g"], P["u"], L.OF_ACT_GELU, P["gu"], fused,
                             done)
            self._linear_bwd(blk["fc1"], P["gu"], P["c"], None, L.OF_ACT_NONE, P["gc"], fused,
                             done)
            self._ln_bwd(blk["ln2"], P["gc"], P["h"], P["mu2"], P["rs2"], P["gy"], P["gh"], fused,
                         done)
            self._linear_bwd(blk["proj"], P["gh"], self._v(blk), None, L.OF_ACT_NONE,
                             P["gqkv"] + 8 * d, fused, done)
            self._linear_bwd(blk["qkv"], P["gqkv"], P["a"], None, L.OF_ACT_NONE, P["ga"], fused,
                             done)
            self._ln_bwd(blk["ln1"], P["ga"], self._block_in(k, x), P["mu1"], P["rs1"], P["gh"],
                         self._gx_of(k), fused, done)

    def backward_plain(self, x):
        self._backward(x, False, None)

    def backward_fused(self, x, done):
        self._backward(x, True, done)

    def argmax(self):
        return {}


class MBNet:
    """MobileNetV2-like network (the mbv2 workload): a 3x3 stem convolution, then
    inverted-residual blocks

        e = ReLU(x W_e^T + b_e)        1x1 expand: a linear over the N*H*W pixel rows
        d = ReLU(dwconv3x3(e, s) + b)  depthwise, stride s
        p = d W_p^T + b_p              1x1 project
        y = x + p                      when s == 1 and the widths match, else y = p

    then a 1x1 head convolution with ReLU, the global average pool and a linear
    classifier.  Every activation and gradient has its own buffer, so nothing a
    later kernel reads is overwritten within a step.  Forward-fusion carries each
    operator's pending update in the previous operator's linear or convolution
    launch (a depthwise launch carries nothing, so the launch before it also
    carries the next linear's update); backward-fusion applies each operator's
    update right after its gradient.

    Both the eager and the backward-fusion orderings run a layer's weight
    gradient (eager: into its gradient buffer; backward-fusion: with the
    update) on the second stream, behind an event recorded after the layer's
    data gradient, so that it overlaps the data gradients further down; each
    reads only buffers that no later kernel of the step writes, the data
    gradient needs the old weights only (Alg. 3), and the main stream joins
    the second one before the eager optimizer step or the next forward.  The
    1x1 layers' split weight gradients are latency-bound kernels of a few
    microseconds that fill the chip poorly on their own (measured on MI355X,
    graph replay: every ordering about 0.2 ms faster per step); the depthwise
    filter gradients gain nothing there and stay in stream order.
    """

    side_updates = False
    side_linear = True   # 1x1 (linear) weight gradients on the second stream
    side_dw = False      # depthwise filter gradients in stream order (measured: no gain)
    eager_side = True    # the eager step joins the second stream before its optimizer

    def __init__(self, tr, cfg, pb):
        self.tr = tr
        N, H = cfg["batch"], cfg["image"]
        f32 = dict(dtype=torch.float32, device=tr.device)
        self.N = N
        self.stem = ConvOp("stem", pb("stem.weight"), pb("stem.bias"), N, H, H, "relu")
        self.ops = [self.stem]
        self.stem_y = torch.empty(self.stem.out_shape, **f32)
        self.stem_g = torch.empty(self.stem.out_shape, **f32)   # grad of the stem's pre-activation
        self.blocks = []
        cin, h, k = cfg["stem"], H, 0
        for t, c, n, s in cfg["blocks"]:
            for r in range(n):
                k += 1
                stride = s if r == 0 else 1
                ho = (h - 1) // stride + 1
                p = f"blk{k}."
                hid = t * cin
                blk = dict(t=t, cin=cin, cout=c, hid=hid, h=h, ho=ho,
                           residual=stride == 1 and cin == c)
                if t != 1:
                    blk["expand"] = LinearOp(p + "expand", pb(p + "expand.weight"),
                                             pb(p + "expand.bias"), N * h * h, "relu")
                    blk["e"] = torch.empty((N * h * h, hid), **f32)
                    blk["ge"] = torch.empty((N * h * h, hid), **f32)
                    self.ops.append(blk["expand"])
                blk["dw"] = DwOp(p + "dw", pb(p + "dw.weight"), pb(p + "dw.bias"), N, h, h, hid,
                                 stride, "relu")
                blk["project"] = LinearOp(p + "project", pb(p + "project.weight"),
                                          pb(p + "project.bias"), N * ho * ho, "none")
                self.ops += [blk["dw"], blk["project"]]
                blk["d"] = torch.empty((N, ho, ho, hid), **f32)
                blk["gd"] = torch.empty((N, ho, ho, hid), **f32)
                # the block output; with a residual connection the projection's
                # epilogue adds the block input to it
                blk["y"] = torch.empty((N * ho * ho, c), **f32)
                blk["gy"] = torch.empty((N * ho * ho, c), **f32)   # grad of the block output
                self.blocks.append(blk)
                cin, h = c, ho
        head, classes = cfg["head"], cfg["classes"]
        self.hf = h
        self.head = LinearOp("head", pb("head.weight"), pb("head.bias"), N * h * h, "relu")
        self.fc = LinearOp("fc", pb("fc.weight"), pb("fc.bias"), N, "none")
        self.ops += [self.head, self.fc]
        self.set_side(self.side_linear, self.side_dw)
        self.hh = torch.empty((N * h * h, head), **f32)
        self.ghh = torch.empty((N * h * h, head), **f32)
        self.pool = torch.empty((N, head), **f32)
        self.gpool = torch.empty((N, head), **f32)
        self.out = torch.empty((N, classes), **f32)
        self.gout = torch.empty((N, classes), **f32)
        # each operator's (input, output) buffers
        self.io = {}
        cur = self.stem_y
        for blk in self.blocks:
            blk["x"] = cur
            if blk["t"] != 1:
                self.io[id(blk["expand"])] = (cur, blk["e"])
                self.io[id(blk["dw"])] = (blk["e"], blk["d"])
            else:
                self.io[id(blk["dw"])] = (cur, blk["d"])
            self.io[id(blk["project"])] = (blk["d"], blk["y"])
            cur = blk["y"]
        self.io[id(self.head)] = (cur, self.hh)
        self.io[id(self.fc)] = (self.pool, self.out)
        # the blocks whose projection adds the block input (residual connection)
        self.residual_of = {id(b["project"]): b for b in self.blocks if b["residual"]}

    def _carry(self, i, fused):
        """Pending updates the forward launch of operator i carries: the next
        operators', through depthwise ones, up to the next linear (at most
        four tensors)."""
        tr = self.tr
        if not fused:
            return None, []
        carried, n = [], 0
        for nxt in self.ops[i + 1:]:
            if nxt.updated or n + len(nxt.params) > L.OF_CARRY_MAX:
                break
            carried.append(nxt)
            n += len(nxt.params)
            if nxt.kind != "dw":
                break
        if not carried:
            return None, []
        return _carry_of(tr, [p for o in carried for p in o.params]), carried

    def forward(self, x, fused):
        tr = self.tr
        s = tr._s()
        for i, op in enumerate(self.ops):
            if fused and not op.updated:
                _self_update(tr, op.params)   # no earlier launch carried it
                op.updated = True
            carry, carried = (None, []) if op.kind == "dw" else self._carry(i, fused)
            tr._t0("fwd", tr.stream, op)
            if op is self.stem:
                op.fwd(tr, x.data_ptr(), self.stem_y.data_ptr(), carry=carry)
            elif op.kind == "dw":
                src, dst = self.io[id(op)]
                op.fwd(tr, src.data_ptr(), dst.data_ptr())
            else:
                src, dst = self.io[id(op)]
                blk = self.residual_of.get(id(op))
                op.fwd(tr, src.data_ptr(), dst.data_ptr(), carry=carry,
                       res=blk["x"].data_ptr() if blk is not None else None)
            tr._t1("fwd", tr.stream)
            for o in carried:
                o.updated = True     # their updates are enqueued with this launch
            if op is self.head:
                tr._t0("fwd", tr.stream)
                L.of_avgpool_fwd(self.hh.data_ptr(), self.N, self.hf * self.hf,
                                 self.hh.shape[1], self.pool.data_ptr(), s)
                tr._t1("fwd", tr.stream)

    def set_side(self, linear, dw):
        """Which weight gradients run on the second stream (both orderings)."""
        self.side_linear, self.side_dw = linear, dw
        for op in self.ops:
            if isinstance(op, LinearOp):
                op.overlap_update = linear

    def _wgrad_plain(self, op, dz, x, side):
        tr = self.tr
        if side:
            gate = _side_after_main(tr)
            tr._t0_after("wgrad", tr.side, op, gate)
            op.wgrad(tr, dz, x, side=True)
            tr._t1("wgrad", tr.side)
        else:
            tr._t0("wgrad", tr.stream, op)
            op.wgrad(tr, dz, x)
            tr._t1("wgrad", tr.stream)

    def _lin_bwd(self, op, dz, x, prev, act_prev, dx, fused, done, dres=None):
        """dres: the gradient of a skip connection from the layer's input, added
        to dx in the data gradient's epilogue."""
        tr = self.tr
        if not fused:
            if dx is not None:
                tr._t0("dgrad", tr.stream, op)
                op.dgrad(tr, dz, prev, act_prev, dx, res=dres)
                tr._t1("dgrad", tr.stream)
            self._wgrad_plain(op, dz, x, op.overlap_update)
        elif tr.timer is not None and (tr.timer.wants("wgrad_bf") or tr.timer.wants("dgrad")):
            if dx is not None:
                tr._t0("dgrad", tr.stream, op)
                op.dgrad(tr, dz, prev, act_prev, dx, res=dres)
                tr._t1("dgrad", tr.stream)
            if op.overlap_update:
                gate = _side_after_main(tr)
                tr._t0_after("wgrad_bf", tr.side, op, gate)
                op.wgrad_fused(tr, dz, x, tr.side.cuda_stream)
                tr._t1("wgrad_bf", tr.side)
            else:
                tr._t0("wgrad_bf", tr.stream, op)
                op.wgrad_fused(tr, dz, x, tr._s())
                tr._t1("wgrad_bf", tr.stream)
            done(op)
        else:
            op.bwd_fused(tr, dz, x, prev, act_prev, dx, res=dres)
            done(op)

    def _dw_bwd(self, op, dy, x, prev, act_prev, dx, fused, done):
        tr = self.tr
        tr._t0("dgrad", tr.stream, op)
        op.dgrad(tr, dy, prev, act_prev, dx)
        tr._t1("dgrad", tr.stream)
        if fused:
            if self.side_dw:
                gate = _side_after_main(tr)
                tr._t0_after("wgrad_bf", tr.side, op, gate)
                op.wgrad_fused(tr, dy, x, tr.side.cuda_stream)
                tr._t1("wgrad_bf", tr.side)
            else:
                tr._t0("wgrad_bf", tr.stream, op)
                op.wgrad_fused(tr, dy, x, tr._s())
                tr._t1("wgrad_bf", tr.stream)
            done(op)
        else:
            self._wgrad_plain(op, dy, x, self.side_dw)

    def _backward(self, x, fused, done):
        tr = self.tr
        s = tr._s()
        P = lambda t: t.data_ptr()  # noqa: E731
        relu, none = L.OF_ACT_RELU, L.OF_ACT_NONE
        # classifier, pool and head
        self._lin_bwd(self.fc, P(self.gout), P(self.pool), None, none, P(self.gpool), fused, done)
        tr._t0("dgrad", tr.stream)
        L.of_avgpool_bwd(P(self.gpool), P(self.hh), self.N, self.hf * self.hf, self.hh.shape[1],
                         P(self.ghh), s)
        tr._t1("dgrad", tr.stream)
        last = self.blocks[-1]
        self._lin_bwd(self.head, P(self.ghh), P(last["y"]), None, none, P(last["gy"]), fused, done)
        for bi in reversed(range(len(self.blocks))):
            blk = self.blocks[bi]
            # the block input's gradient: the previous block's output gradient,
            # or the stem's pre-activation gradient (through the stem's ReLU)
            if bi > 0:
                gin, in_act = self.blocks[bi - 1]["gy"], none
            else:
                gin, in_act = self.stem_g, relu
            xin = blk["x"]
            self._lin_bwd(blk["project"], P(blk["gy"]), P(blk["d"]), P(blk["d"]), relu,
                          P(blk["gd"]), fused, done)
            # the skip connection: the block input also gets the output's gradient,
            # added in the expand layer's data-gradient epilogue
            skip = P(blk["gy"]) if blk["residual"] else None
            if blk["t"] != 1:
                self._dw_bwd(blk["dw"], P(blk["gd"]), P(blk["e"]), P(blk["e"]), relu,
                             P(blk["ge"]), fused, done)
                self._lin_bwd(blk["expand"], P(blk["ge"]), P(xin), P(xin) if in_act else None,
                              in_act, P(gin), fused, done, dres=skip)
            else:
                self._dw_bwd(blk["dw"], P(blk["gd"]), P(xin), P(xin) if in_act else None, in_act,
                             P(gin), fused, done)
                if skip is not None:   # a depthwise data gradient takes no residual
                    tr._t0("add", tr.stream)
                    L.of_add(P(gin), skip, gin.numel(), P(gin), s)
                    tr._t1("add", tr.stream)
        # the stem is the first layer: no data gradient
        stem = self.stem
        if fused:
            gate = _side_after_main(tr) if stem.overlap_update else None
            if gate is not None:
                tr._t0_after("wgrad_bf", tr.side, stem, gate)
                stem.wgrad_fused(tr, P(self.stem_g), P(x), tr.side.cuda_stream)
                tr._t1("wgrad_bf", tr.side)
            else:
                tr._t0("wgrad_bf", tr.stream, stem)
                stem.wgrad_fused(tr, P(self.stem_g), P(x), tr._s())
                tr._t1("wgrad_bf", tr.stream)
            done(stem)
        else:
            self._wgrad_plain(stem, P(self.stem_g), P(x), stem.overlap_update)

    def backward_plain(self, x):
        self._backward(x, False, None)

    def backward_fused(self, x, done):
        self._backward(x, True, done)

    def argmax(self):
        return {}


class Trainer:
    """Trains one workload on one GPU under a chosen ordering."""

    def __init__(self, cfg, init, device="cuda:0", merge_dgrad=False, conv_prologue=False,
                 linear_prologue=False, bf16_acts=True):
        """merge_dgrad: backward-fusion runs each fp32 linear layer with at most
        64 rows as one merged data-gradient + update pass (of_linear_bwd_merged).
        conv_prologue: forward-fusion applies a convolution's pending update in
        its forward's filter-tile loads (of_conv_fwd_fused) instead of carrying
        it in the previous launch.
        linear_prologue: the same for fp32 linear layers of more than 64 rows
        (of_linear_fwd_fused with a second buffer set); layers of at most 64
        rows always take the prologue (in place)."""
        L.load()
        self.cfg, self.hyper = cfg, cfg["opt"]
        self.device = torch.device(device)
        kind = self.hyper["kind"]
        self.params = {}

        def pb(name, shadow=False, rows=0):
            p = ParamBuf(name, init[name], kind, self.device, shadow, rows)
            self.params[name] = p
            return p

        if cfg["kind"] in ("mlp", "vgg"):
            if cfg["dtype"] != "f32":
                raise NotImplementedError("linear / conv chains run with fp32 operands")
            self.net = ChainNet(self, cfg, pb)
        elif cfg["kind"] == "tblock":
            self.net = TBlockNet(self, cfg, pb, bf16_acts=bf16_acts)
        elif cfg["kind"] == "mbv2":
            if cfg["dtype"] != "f32":
                raise NotImplementedError("the MobileNetV2-like network runs with fp32 operands")
            self.net = MBNet(self, cfg, pb)
        else:
            raise NotImplementedError(f"model kind {cfg['kind']!r} has no GPU path in this build")
        self.ops = self.net.ops
        # Adagrad and RMSprop without momentum keep no m: the kernels get a NULL m
        # and neither read nor write it (m stays zero on the host side too).
        if kind == "adagrad" or (kind == "rmsprop" and not self.hyper.get("momentum", 0.0)):
            for p in self.params.values():
                p.p.m = None
        self.eager_reduce = True
        for op in self.ops:
            if op.kind == "linear" and merge_dgrad and op.merge_ok:
                op.merge_dgrad = True
            if op.kind == "conv":
                op.prologue_ff = bool(conv_prologue)
            if op.kind == "linear" and op.fp32 and op.M > 64:
                op.prologue_ff = bool(linear_prologue)
        f32 = dict(dtype=torch.float32, device=self.device)
        wsm = max([op.ws(w) for op in self.ops for w in (0, 1, 2)] + [16])
        wsm = max([wsm] + [op.ws(L.OF_LINEAR_BWD_MERGED) for op in self.ops if op.kind == "linear"
                           and op.merge_dgrad])
        wss = max([op.ws(2) for op in self.ops] + [16])
        if cfg["loss"] == "mse":
            wsm = max(wsm, L.of_mse_workspace_size(*self.net.out.shape))
        self.ws_main = torch.empty((wsm + 15) // 16 * 4, **f32)
        self.ws_side = torch.empty((wss + 15) // 16 * 4, **f32)
        self.losses = torch.zeros(4096, **f32)
        self.t = 0
        # The 1-based index of the update being applied travels by value in
        # launched steps.  A captured step instead reads it from this device
        # counter, advanced in stream order right before the step's updates, so
        # one captured launch sequence serves every later step.
        self.step_dev = torch.zeros(1, dtype=torch.int64, device=self.device)
        # Global-norm clipping (optimizer dict `clip_norm`): the factor and the
        # norm live on the device, written after each backward pass and read by
        # the updates that consume those gradients.
        self.clip_norm = self.hyper.get("clip_norm")
        self.grad_scale = None
        if self.clip_norm is not None:
            self.clip_out = torch.ones(2, **f32)           # (scale, norm)
            self.clip_ws = torch.empty(L.OF_CLIP_WS_BYTES // 4, **f32)
            self.grad_scale = self.clip_out.data_ptr()
        self.opt_dev = L.make_opt(self.hyper, 0, self.step_dev.data_ptr(), self.grad_scale)
        self.opt = self.opt_dev
        self.capturing = False
        self.stream = torch.cuda.current_stream(self.device)
        self.side = device_stream(self.device, "side")
        self._side2 = None   # a second side stream, made on first use
        self.side2_done = torch.cuda.Event()
        self.side_done = torch.cuda.Event()
        # Whether backward-fusion puts any update on the side stream: a chain of
        # light layers updates in stream order and needs no join at the step's
        # end (two runtime calls fewer per step); the Transformer blocks update
        # their LayerNorm parameters there.
        self.uses_side = (getattr(self.net, "side_updates", True) or
                          any(op.overlap_update and not getattr(op, "merge_dgrad", False)
                              for op in self.ops))
        self.pending_ordering = None
        self.timer = None   # optional KernelTimer: HIP events around chosen launch classes

    # ------------------------------------------------------------ helpers
    def ws_main_args(self):
        return self.ws_main.data_ptr(), self.ws_main.numel() * 4

    def ws_side_args(self):
        return self.ws_side.data_ptr(), self.ws_side.numel() * 4

    def _s(self):
        return self.stream.cuda_stream

    def side2(self):
        """A second side stream (backward-fusion's LayerNorm updates), one per
        device like the first; a step that used it joins it at its end."""
        if self._side2 is None:
            self._side2 = device_stream(self.device, "side2")
        return self._side2

    def _advance(self, ps):
        """Next update index for parameters ps; sets the optimizer argument the
        step's updating launches take (by value, or the advanced device counter)."""
        step = ps[0].step + 1
        if any(p.step + 1 != step for p in ps):
            raise RuntimeError("parameters out of step: this trainer keeps one update counter")
        if self.capturing:
            L.of_step_advance(self.step_dev.data_ptr(), 1, self._s())
            self.opt = self.opt_dev
        else:
            self.opt = L.make_opt(self.hyper, step, None, self.grad_scale)
        return step

    def _clip(self, vector):
        """Global-norm clipping factor of the gradients just computed (Appendix
        B.1): `vector` -- every gradient is in p.g (eager); else the pending ones
        (forward-fusion: LayerNorm gradients as row partials)."""
        if self.clip_norm is None:
            return
        items = []
        for p in self.params.values():
            if vector or p.rows is None:
                items.append((p.g.data_ptr(), p.numel, 1, 0))
            else:
                ptr, rows, ld = p.pending()
                items.append((ptr, p.numel, rows, ld))
        self._t0("clip", self.stream)
        L.of_grad_clip_scale(len(items), L.grad_refs(items), self.clip_norm,
                             self.clip_out.data_ptr(), self.clip_out.data_ptr() + 4,
                             self.clip_ws.data_ptr(), L.OF_CLIP_WS_BYTES, self._s())
        self._t1("clip", self.stream)

    def _t0(self, cls, stream, op=None):
        if self.timer is not None:
            self.timer.start(cls, stream, op)

    def _t0_after(self, cls, stream, op, gate):
        if self.timer is not None:
            self.timer.start_after(cls, stream, op, gate)

    def _t1(self, cls, stream):
        if self.timer is not None:
            self.timer.stop(cls, stream)

    def _loss(self, y):
        self._t0("loss", self.stream)
        out, gout = self.net.out, self.net.gout
        M, C = out.shape
        loss_ptr = self.losses.data_ptr() + 4 * (self.t % self.losses.numel())
        if self.cfg["loss"] == "xent":
            L.of_xent_fwd_bwd(out.data_ptr(), y.data_ptr(), M, C, 0, loss_ptr, gout.data_ptr(),
                              self._s())
        else:
            L.of_mse_fwd_bwd(out.data_ptr(), y.data_ptr(), M, C, 0, loss_ptr, gout.data_ptr(),
                             *self.ws_main_args(), self._s())
        self._t1("loss", self.stream)

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
        self.net.forward(x, fused=False)
        self._loss(y)
        self.eager_reduce = True
        self.net.backward_plain(x)
        self._join_plain_side()
        self._clip(vector=True)
        ps = list(self.params.values())
        step = self._advance(ps)
        arr = (L.OfParam * len(ps))(*[p.p for p in ps])
        grads = (L.c_void_p * len(ps))(*[p.g.data_ptr() for p in ps])
        self._t0("opt", self.stream)
        L.of_optimizer_step(len(ps), arr, grads, self.opt, self._s())
        self._t1("opt", self.stream)
        for p in ps:
            p.step = step

    def _join_plain_side(self):
        """After a plain backward that computed weight gradients on the second
        stream: the main stream waits for them (the eager optimizer step, the
        clipping norm and the next forward's pending updates read them)."""
        if self.uses_side and getattr(self.net, "eager_side", False):
            self.side_done.record(self.side)
            self.stream.wait_event(self.side_done)

    def _step_ff(self, x, y):
        pending = _unique([p for op in self.ops if not op.updated for p in op.params])
        if pending:
            step = self._advance(pending)
            for p in pending:
                p.step = step
        self.net.forward(x, fused=True)
        self._loss(y)
        # gradients stay pending (LayerNorm's as row partials)
        self.eager_reduce = False
        self.net.backward_plain(x)
        self._join_plain_side()
        self._clip(vector=False)
        for op in self.ops:
            op.updated = False

    def flush(self):
        """Apply every update forward-fusion still holds (what the next forward would do)."""
        pending = _unique([p for op in self.ops if not op.updated for p in op.params])
        if pending:
            step = self._advance(pending)
            for p in pending:
                _update(self, p, self._s())
                p.step = step
            for op in self.ops:
                op.updated = True
        self.pending_ordering = None

    def _step_bf(self, x, y):
        if self.clip_norm is not None:
            raise ValueError("backward-fusion updates each tensor before the other gradients "
                             "exist, so it cannot clip by the global norm (Table 1)")
        # The forward of each layer at this step needs its update from the last
        # step: the previous step ended with the main stream joining the side one
        # (when any update ran there).
        for op in self.ops:
            for p in op.params:
                p.count += 1
        self.net.forward(x, fused=False)
        self._loss(y)
        step = self._advance(list(self.params.values()))

        def done(op):
            # Alg. 3: a use's gradient is complete; the last use (count 0) updated
            for p in op.params:
                p.count -= 1
                if p.count == 0:
                    p.step = step

        self.net.backward_fused(x, done)
        if self.uses_side:
            # the next forward reads parameters the side stream updated
            self.side_done.record(self.side)
            self.stream.wait_event(self.side_done)
        if self._side2 is not None:
            self.side2_done.record(self._side2)
            self.stream.wait_event(self.side2_done)

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
        # A graph holds the parameter buffers current now; the convolutions'
        # filter-tile prologue would alternate them, so from here on their
        # updates are carried by the previous launch (the same values) in
        # launched steps too.
        for op in self.ops:
            if op.two_sets():
                op.prologue_ff = False
        saved = ([(p.step, p.count) for p in self.params.values()],
                 [op.updated for op in self.ops], self.t, self.pending_ordering)
        g = torch.cuda.CUDAGraph()
        cap = device_stream(self.device, "capture")
        # the device counter holds the index of the last applied update
        self.step_dev.fill_(next(iter(self.params.values())).step)
        cap.wait_stream(self.stream)
        main = self.stream
        torch.cuda.synchronize(self.device)
        try:
            self.stream = cap
            self.capturing = True
            with torch.cuda.graph(g, stream=cap):
                self.step(x, y, ordering)
        finally:
            self.stream = main
            self.capturing = False
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
            p.set(params[k])
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
                        p.set_pending(pending[p.name])
                    op.updated = False
            self.pending_ordering = "ff"
        torch.cuda.synchronize(self.device)

    def loss_history(self):
        torch.cuda.synchronize(self.device)
        return self.losses[: self.t].cpu().numpy().astype(np.float64)

    def argmax(self):
        """Max-pool window positions of the last forward by layer index (synchronises)."""
        torch.cuda.synchronize(self.device)
        return {i: a.cpu().numpy().astype(np.int32) for i, a in self.net.argmax().items()}

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
        self.net.forward(x, fused=False)
        saved = self.t
        self._loss(y)
        torch.cuda.synchronize(self.device)
        return float(self.losses[saved % self.losses.numel()].item())


class KernelTimer:
    """HIP events around chosen launch classes, recorded on the launch's stream.

    A launch on a stream that first waits for another stream's event is timed
    from the later of that event and a start event recorded on its own stream:
    an event recorded on a stream that is idle when the wait is enqueued can
    take its timestamp before the wait is satisfied, which would add the wait
    to the kernel's time."""

    def __init__(self, classes, pool=0):
        """pool: events created (and recorded once, which creates the HIP
        event) up front, so that timed steps do not create events: a host
        stall inside the timed region lets the GPU drain its queue, and the
        wait would be counted inside the bracket being timed."""
        self.classes = set(classes)
        self.records = {c: [] for c in self.classes}
        self._open = {}
        self._pool = [torch.cuda.Event(enable_timing=True) for _ in range(pool)]
        for e in self._pool:
            e.record()
        if pool:
            torch.cuda.synchronize()

    def _event(self):
        return self._pool.pop() if self._pool else torch.cuda.Event(enable_timing=True)

    def wants(self, cls):
        return cls in self.classes

    def start(self, cls, stream, op=None):
        if cls in self.classes:
            e = self._event()
            e.record(stream)
            self._open[cls] = (e, op)

    def start_after(self, cls, stream, op, gate):
        """Start a launch on `stream` that waits for `gate` (a timing event)."""
        if cls in self.classes:
            e = self._event()
            e.record(stream)
            self._open[cls] = ((gate, e), op)

    def stop(self, cls, stream):
        if cls in self.classes:
            e0, op = self._open.pop(cls)
            e1 = self._event()
            e1.record(stream)
            self.records[cls].append((e0, e1, op))

    def clear(self):
        self.records = {c: [] for c in self.classes}

    def durations(self, cls):
        """[(milliseconds, op)] of every recorded launch of `cls` (synchronises)."""
        torch.cuda.synchronize()
        out = []
        for e0, e1, op in self.records[cls]:
            if isinstance(e0, tuple):
                gate, start = e0
                out.append((min(gate.elapsed_time(e1), start.elapsed_time(e1)), op))
            else:
                out.append((e0.elapsed_time(e1), op))
        return out

    @staticmethod
    def marker_overhead_ms(stream, samples=40):
        """What an event pair adds to the time it brackets on `stream`, taken as a
        bracketed launch sees it: pairs queued behind work around one and around
        two back-to-back launches of the same copy kernel (medians B1, B2).
        B1 = c + k and B2 = c + 2k + g give 2*B1 - B2 = c - g, so a bracketed
        time minus this is the kernel's duration plus one back-to-back gap (an
        empty pair on an idle stream costs more than a pair around a launch)."""
        a = torch.empty(1 << 22, device=torch.cuda.current_device())
        b = torch.empty_like(a)

        def bracket(nk):
            pairs = []
            with torch.cuda.stream(stream):
                for _ in range(samples):
                    b.copy_(a)   # the pair is queued behind work, as in a step
                    e0 = torch.cuda.Event(enable_timing=True)
                    e1 = torch.cuda.Event(enable_timing=True)
                    e0.record(stream)
                    for _ in range(nk):
                        b.copy_(a)
                    e1.record(stream)
                    pairs.append((e0, e1))
            torch.cuda.synchronize()
            return float(np.median([x.elapsed_time(y) for x, y in pairs]))

        bracket(1)   # warm
        return max(0.0, 2.0 * bracket(1) - bracket(2))
