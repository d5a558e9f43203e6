"""Operators f_i of the training graph, float64, forward and backward.

Fig. 1(a) of the paper views training as a dependency graph of tensor
operators; each operator here is one node f_i.  An operator holds references
to its trainable parameters (objects of class Param) so that one operator may
appear several times in the topologically sorted array (the case the
`updated` flag of Alg. 2 and the `count` of Alg. 3 exist for).

backward(ctx, dy) reads the CURRENT value of the operator's parameters; the
orderings call it before any update of those parameters, which is the
dependency rule stated after Alg. 3 (the input gradient of f(theta, x) =
theta x needs the old theta).

Definitions (the readings where the paper is silent):
  linear      z = x W^T + b           W is [out, in]
  relu        y = max(z, 0); dz = dy where z > 0 (strictly), else 0
  gelu        y = z * Phi(z) (exact erf form); dz = dy (Phi(z) + z phi(z))
  layernorm   over the last axis, biased variance, eps inside the sqrt
  conv3x3     cross-correlation, stride 1, zero padding 1, NHWC / [Cout,3,3,Cin]
  dwconv3x3   the same per channel (depthwise, multiplier 1), filter [3,3,C],
              stride 1 or 2
  avgpool     mean over the spatial positions of each channel
  maxpool2x2  stride 2; the argmax is the first maximum of the window in
              row-major order (strict >), reported as its window position 0..3
  bf16        matmul operands rounded to bfloat16 just before the product

Pinned by: finite differences in float64, direct loop references for conv and
max-pool, closed values (tests/test_oracle_layers.py).
"""
import numpy as np
from scipy.special import erf

from .bf16 import round_bf16


class Param:
    """A trainable tensor theta with its optimizer history (Fig. 2, "History")."""

    def __init__(self, name, value):
        self.name = name
        self.value = np.array(value, dtype=np.float64)
        self.m = np.zeros_like(self.value)   # momentum buffer / Adam first moment
        self.v = np.zeros_like(self.value)   # Adam second moment
        self.grad = None                      # accumulated gradient (None = nothing pending)
        self.step = 0                         # number of updates applied so far
        self.count = 0                        # Alg. 3: forward uses not yet back-propagated


class Op:
    """Base operator: parameters plus the Alg. 2 `updated` flag."""

    params = ()

    def __init__(self):
        # Nothing is pending before the first iteration (see the FF reading in
        # the oracle's train module), so the flag starts True.
        self.updated = True


def _maybe_bf16(a, bf16):
    return round_bf16(a) if bf16 else a


class Linear(Op):
    def __init__(self, w, b=None, bf16=False):
        super().__init__()
        self.w, self.b, self.bf16 = w, b, bf16
        self.params = (w,) if b is None else (w, b)

    def forward(self, x):
        z = _maybe_bf16(x, self.bf16) @ _maybe_bf16(self.w.value, self.bf16).T
        if self.b is not None:
            z = z + self.b.value
        return z, x

    def abs_bound(self, x):
        """sum_k |x_mk w_nk| + |b_n|: the scale of the rounding error of z."""
        s = np.abs(_maybe_bf16(x, self.bf16)) @ np.abs(_maybe_bf16(self.w.value, self.bf16)).T
        return s + np.abs(self.b.value) if self.b is not None else s

    def backward(self, x, dz):
        dzq = _maybe_bf16(dz, self.bf16)
        dx = dzq @ _maybe_bf16(self.w.value, self.bf16)
        dw = dzq.T @ _maybe_bf16(x, self.bf16)
        grads = (dw,) if self.b is None else (dw, dz.sum(axis=0))
        return (dx,), grads


class ReLU(Op):
    """flip: optional boolean array; where True the backward mask decision is
    inverted (used to enumerate the decisions float32 rounding can change)."""

    flip = None

    def forward(self, z):
        return np.maximum(z, 0.0), z

    def backward(self, z, dy):
        mask = z > 0.0
        if self.flip is not None:
            mask = mask ^ self.flip
        return (np.where(mask, dy, 0.0),), ()


def gelu_cdf(z):
    return 0.5 * (1.0 + erf(z / np.sqrt(2.0)))


def gelu_pdf(z):
    return np.exp(-0.5 * z * z) / np.sqrt(2.0 * np.pi)


class GELU(Op):
    def forward(self, z):
        return z * gelu_cdf(z), z

    def backward(self, z, dy):
        return (dy * (gelu_cdf(z) + z * gelu_pdf(z)),), ()


class LayerNorm(Op):
    def __init__(self, gamma, beta, eps=1e-5):
        super().__init__()
        self.gamma, self.beta, self.eps = gamma, beta, eps
        self.params = (gamma, beta)

    def forward(self, x):
        mu = x.mean(axis=-1, keepdims=True)
        var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
        rstd = 1.0 / np.sqrt(var + self.eps)
        xhat = (x - mu) * rstd
        return xhat * self.gamma.value + self.beta.value, (xhat, rstd)

    def backward(self, ctx, dy):
        xhat, rstd = ctx
        dxhat = dy * self.gamma.value
        dx = rstd * (dxhat - dxhat.mean(axis=-1, keepdims=True)
                     - xhat * (dxhat * xhat).mean(axis=-1, keepdims=True))
        return (dx,), ((dy * xhat).sum(axis=0), dy.sum(axis=0))


class Add(Op):
    def forward(self, a, b):
        return a + b, None

    def backward(self, _, dy):
        return (dy, dy), ()


class SliceCols(Op):
    """Columns [lo, hi) of a [rows, cols] tensor (the V third of a fused QKV output)."""

    def __init__(self, lo, hi):
        super().__init__()
        self.lo, self.hi = lo, hi

    def forward(self, x):
        return x[:, self.lo:self.hi], x.shape

    def backward(self, shape, dy):
        dx = np.zeros(shape)
        dx[:, self.lo:self.hi] = dy
        return (dx,), ()


class Conv3x3(Op):
    """3x3 cross-correlation, stride 1, zero pad 1, NHWC input, [Cout,3,3,Cin] filter."""

    def __init__(self, w, b=None):
        super().__init__()
        self.w, self.b = w, b
        self.params = (w,) if b is None else (w, b)

    def forward(self, x):
        n, h, wd, _ = x.shape
        xp = np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)))
        w = self.w.value
        y = np.zeros((n, h, wd, w.shape[0]))
        for r in range(3):
            for s in range(3):
                y += xp[:, r:r + h, s:s + wd, :] @ w[:, r, s, :].T
        if self.b is not None:
            y += self.b.value
        return y, xp

    def abs_bound(self, x):
        """sum over taps and channels of |x||w| + |b|: the scale of the rounding error of y."""
        n, h, wd, _ = x.shape
        xp = np.pad(np.abs(x), ((0, 0), (1, 1), (1, 1), (0, 0)))
        w = np.abs(self.w.value)
        s = np.zeros((n, h, wd, w.shape[0]))
        for r in range(3):
            for c in range(3):
                s += xp[:, r:r + h, c:c + wd, :] @ w[:, r, c, :].T
        return s + np.abs(self.b.value) if self.b is not None else s

    def backward(self, xp, dy):
        n, h, wd, cout = dy.shape
        w = self.w.value
        dxp = np.zeros_like(xp)
        dw = np.zeros_like(w)
        for r in range(3):
            for s in range(3):
                dxp[:, r:r + h, s:s + wd, :] += dy @ w[:, r, s, :]
                dw[:, r, s, :] = np.tensordot(dy, xp[:, r:r + h, s:s + wd, :],
                                              axes=([0, 1, 2], [0, 1, 2]))
        grads = (dw,) if self.b is None else (dw, dy.sum(axis=(0, 1, 2)))
        return (dxp[:, 1:-1, 1:-1, :],), grads


class DepthwiseConv3x3(Op):
    """Depthwise 3x3 cross-correlation (one filter per channel), zero pad 1,
    stride 1 or 2, NHWC input, [3,3,C] filter:
    y[n,ho,wo,c] = b[c] + sum over taps of x[n, S ho + ky - 1, S wo + kx - 1, c] w[ky,kx,c],
    output [N, (H-1)//S + 1, (W-1)//S + 1, C].  The small-parameter layers of
    MobileNetV2, the network of the paper's Fig. 3 and Table 2."""

    def __init__(self, w, b=None, stride=1):
        super().__init__()
        self.w, self.b, self.stride = w, b, stride
        self.params = (w,) if b is None else (w, b)

    def _taps(self, xp, ho, wo):
        """The padded input seen by each tap: xp[:, S ho + r, S wo + s, :] for r, s < 3."""
        S = self.stride
        for r in range(3):
            for s in range(3):
                yield r, s, (slice(None), slice(r, r + S * (ho - 1) + 1, S),
                             slice(s, s + S * (wo - 1) + 1, S), slice(None))

    def _out_hw(self, x):
        return (x.shape[1] - 1) // self.stride + 1, (x.shape[2] - 1) // self.stride + 1

    def forward(self, x):
        ho, wo = self._out_hw(x)
        xp = np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)))
        w = self.w.value
        y = np.zeros((x.shape[0], ho, wo, x.shape[3]))
        for r, s, sl in self._taps(xp, ho, wo):
            y += xp[sl] * w[r, s, :]
        if self.b is not None:
            y += self.b.value
        return y, xp

    def abs_bound(self, x):
        """sum over taps of |x||w| + |b|: the scale of the rounding error of y."""
        ho, wo = self._out_hw(x)
        xp = np.pad(np.abs(x), ((0, 0), (1, 1), (1, 1), (0, 0)))
        w = np.abs(self.w.value)
        out = np.zeros((x.shape[0], ho, wo, x.shape[3]))
        for r, c, sl in self._taps(xp, ho, wo):
            out += xp[sl] * w[r, c, :]
        return out + np.abs(self.b.value) if self.b is not None else out

    def backward(self, xp, dy):
        ho, wo = dy.shape[1], dy.shape[2]
        w = self.w.value
        dxp = np.zeros_like(xp)
        dw = np.zeros_like(w)
        for r, s, sl in self._taps(xp, ho, wo):
            dxp[sl] += dy * w[r, s, :]
            dw[r, s, :] = (dy * xp[sl]).sum(axis=(0, 1, 2))
        grads = (dw,) if self.b is None else (dw, dy.sum(axis=(0, 1, 2)))
        return (dxp[:, 1:-1, 1:-1, :],), grads


class GlobalAvgPool(Op):
    """Mean over the spatial positions: [N,H,W,C] -> [N,C] (MobileNetV2's head)."""

    def forward(self, x):
        return x.mean(axis=(1, 2)), x.shape

    def backward(self, shape, dy):
        n, h, w, c = shape
        return (np.broadcast_to(dy[:, None, None, :] / (h * w), shape).copy(),), ()


class PixelRows(Op):
    """[N,H,W,C] feature map -> [N*H*W, C] rows: a 1x1 convolution is a linear
    layer over the pixels."""

    def forward(self, x):
        return x.reshape(-1, x.shape[-1]), x.shape

    def backward(self, shape, dy):
        return (dy.reshape(shape),), ()


class PixelMap(Op):
    """[N*H*W, C] rows -> [N,H,W,C] (the spatial shape of the map `like`)."""

    def __init__(self, n, h, w):
        super().__init__()
        self.shape = (n, h, w)

    def forward(self, x):
        return x.reshape(self.shape + (x.shape[-1],)), x.shape

    def backward(self, shape, dy):
        return (dy.reshape(shape),), ()


class MaxPool2x2(Op):
    """2x2 max-pool, stride 2, NHWC; records the window position of the first maximum."""

    def forward(self, x):
        n, h, w, c = x.shape
        win = np.stack([x[:, 0::2, 0::2, :], x[:, 0::2, 1::2, :],
                        x[:, 1::2, 0::2, :], x[:, 1::2, 1::2, :]])
        arg = np.zeros(win.shape[1:], dtype=np.int32)
        best = win[0].copy()
        for p in range(1, 4):
            take = win[p] > best            # strict: the earlier position wins ties
            best = np.where(take, win[p], best)
            arg = np.where(take, p, arg)
        self.last_argmax = arg
        return best, (x.shape, arg)

    def backward(self, ctx, dy):
        shape, arg = ctx
        dx = np.zeros(shape)
        for p, (di, dj) in enumerate(((0, 0), (0, 1), (1, 0), (1, 1))):
            dx[:, di::2, dj::2, :] = np.where(arg == p, dy, 0.0)
        return (dx,), ()


class Flatten(Op):
    """[N, 1, 1, C] feature map -> [N, C] rows for the classifier."""

    def forward(self, x):
        return x.reshape(x.shape[0], -1), x.shape

    def backward(self, shape, dy):
        return (dy.reshape(shape),), ()
