"""Pins for the oracle's operators and losses: finite differences, direct loops, closed values."""
import math

import numpy as np
import pytest

from oracle import layers as L
from oracle.losses import xent, mse


def _fd_check(f, arrays, h=1e-6, rtol=1e-6, atol=1e-9):
    """Central finite differences of scalar f() w.r.t. every entry of each array in `arrays`.

    Returns the numeric gradients, one per array (arrays are perturbed in place).
    """
    out = []
    for a in arrays:
        g = np.zeros_like(a)
        it = np.nditer(a, flags=["multi_index"])
        for _ in it:
            i = it.multi_index
            old = a[i]
            a[i] = old + h
            fp = f()
            a[i] = old - h
            fm = f()
            a[i] = old
            g[i] = (fp - fm) / (2 * h)
        out.append(g)
    return out


def _check_op(op, inputs, seed=0):
    """Compare op.backward against finite differences of sum(forward * R)."""
    rng = np.random.default_rng(seed)
    y, _ = op.forward(*inputs)
    R = rng.standard_normal(y.shape)

    def f():
        return float(np.sum(op.forward(*inputs)[0] * R))

    y, ctx = op.forward(*inputs)
    dxs, dps = op.backward(ctx, R)
    num = _fd_check(f, list(inputs) + [p.value for p in op.params])
    for a, n in zip(list(dxs) + list(dps), num):
        np.testing.assert_allclose(a, n, rtol=1e-6, atol=1e-8)


def _P(rng, shape, scale=1.0):
    return L.Param("p", rng.standard_normal(shape) * scale)


def test_linear_grads_and_matmul():
    rng = np.random.default_rng(0)
    w, b = _P(rng, (5, 4)), _P(rng, (5,))
    x = rng.standard_normal((3, 4))
    op = L.Linear(w, b)
    z, _ = op.forward(x)
    loops = np.array([[sum(x[i, k] * w.value[j, k] for k in range(4)) + b.value[j]
                       for j in range(5)] for i in range(3)])
    np.testing.assert_allclose(z, loops, rtol=1e-14, atol=1e-14)
    _check_op(op, [x])


def test_linear_bf16_rounds_operands_only():
    # Operands exactly on the bf16 grid: the product is the float64 product.
    rng = np.random.default_rng(1)
    xw = (rng.integers(-64, 64, (6, 8)) / 16.0)
    ww = (rng.integers(-64, 64, (3, 8)) / 32.0)
    w = L.Param("w", ww)
    z, _ = L.Linear(w, None, bf16=True).forward(xw)
    np.testing.assert_array_equal(z, xw @ ww.T)
    # Off-grid operand: the result differs from the float64 product.
    x2 = xw + 1e-3
    z2, _ = L.Linear(w, None, bf16=True).forward(x2)
    z3, _ = L.Linear(w, None, bf16=False).forward(x2)
    assert np.max(np.abs(z2 - z3)) > 1e-4


def test_relu_grad_and_strict_mask():
    rng = np.random.default_rng(2)
    z = rng.standard_normal((4, 6))
    z[np.abs(z) < 1e-2] = 0.5
    _check_op(L.ReLU(), [z])
    dz = L.ReLU().backward(np.array([0.0, -1.0, 2.0]), np.ones(3))[0][0]
    np.testing.assert_array_equal(dz, [0.0, 0.0, 1.0])


def test_gelu_values_and_grad():
    y, _ = L.GELU().forward(np.array([0.0, 1.0, -1.0, 8.0, -8.0]))
    # Phi(1) = 0.841344746068543 (standard normal CDF).
    np.testing.assert_allclose(y[:3], [0.0, 0.841344746068543, -(1 - 0.841344746068543)],
                               rtol=1e-14, atol=1e-15)
    assert y[3] == pytest.approx(8.0, rel=1e-12) and abs(y[4]) < 1e-12
    _check_op(L.GELU(), [np.random.default_rng(3).standard_normal((3, 5))])


def test_layernorm_values_and_grads():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((4, 7)) * 3 + 1
    op = L.LayerNorm(L.Param("g", np.ones(7)), L.Param("b", np.zeros(7)), eps=0.0)
    y, _ = op.forward(x)
    np.testing.assert_allclose(y.mean(axis=1), 0.0, atol=1e-14)
    np.testing.assert_allclose((y ** 2).mean(axis=1), 1.0, rtol=1e-13)
    op = L.LayerNorm(_P(rng, (7,)), _P(rng, (7,)), eps=1e-5)
    _check_op(op, [x])


def test_add_slice_flatten_grads():
    rng = np.random.default_rng(5)
    _check_op(L.Add(), [rng.standard_normal((3, 4)), rng.standard_normal((3, 4))])
    _check_op(L.SliceCols(2, 5), [rng.standard_normal((3, 6))])
    _check_op(L.Flatten(), [rng.standard_normal((2, 1, 1, 5))])


def _conv_loops(x, w, b):
    n, h, wd, cin = x.shape
    cout = w.shape[0]
    y = np.zeros((n, h, wd, cout))
    for a in range(n):
        for i in range(h):
            for j in range(wd):
                for o in range(cout):
                    s = b[o]
                    for r in range(3):
                        for q in range(3):
                            ii, jj = i + r - 1, j + q - 1
                            if 0 <= ii < h and 0 <= jj < wd:
                                s += float(np.dot(x[a, ii, jj, :], w[o, r, q, :]))
                    y[a, i, j, o] = s
    return y


def test_conv3x3_matches_direct_loops_and_grads():
    rng = np.random.default_rng(6)
    x = rng.standard_normal((2, 5, 4, 3))
    w, b = _P(rng, (4, 3, 3, 3)), _P(rng, (4,))
    op = L.Conv3x3(w, b)
    y, _ = op.forward(x)
    np.testing.assert_allclose(y, _conv_loops(x, w.value, b.value), rtol=1e-13, atol=1e-13)
    _check_op(op, [x])


def test_dwconv3x3_is_block_diagonal_conv_loops_and_grads():
    """Depthwise = the full 3x3 conv with a channel-diagonal filter (checked by direct
    loops); its gradients pass finite differences."""
    rng = np.random.default_rng(16)
    x = rng.standard_normal((2, 5, 4, 3))
    w, b = _P(rng, (3, 3, 3)), _P(rng, (3,))
    full = np.zeros((3, 3, 3, 3))
    for c in range(3):
        full[c, :, :, c] = w.value[:, :, c]
    op = L.DepthwiseConv3x3(w, b)
    y, _ = op.forward(x)
    np.testing.assert_allclose(y, _conv_loops(x, full, b.value), rtol=1e-13, atol=1e-13)
    # a one-hot input picks single filter taps out, transposed through the padding
    e = np.zeros((1, 3, 3, 3))
    e[0, 1, 1, 2] = 1.0
    ye, _ = L.DepthwiseConv3x3(L.Param("w", w.value), None).forward(e)
    np.testing.assert_array_equal(ye[0, :, :, 2], w.value[::-1, ::-1, 2])
    np.testing.assert_array_equal(ye[0, :, :, :2], 0.0)
    _check_op(op, [x])


def test_dwconv3x3_stride2_is_the_subsampled_stride1_output_and_grads():
    """Stride 2 (zero pad 1) keeps every second output of the stride-1 result,
    rows and columns 0, 2, 4, ... (odd and even sizes); gradients pass finite
    differences."""
    rng = np.random.default_rng(17)
    for h, wd in ((6, 4), (5, 7), (1, 1), (2, 3)):
        x = rng.standard_normal((2, h, wd, 3))
        w, b = _P(rng, (3, 3, 3)), _P(rng, (3,))
        y1, _ = L.DepthwiseConv3x3(w, b).forward(x)
        op = L.DepthwiseConv3x3(w, b, stride=2)
        y2, _ = op.forward(x)
        assert y2.shape == (2, (h - 1) // 2 + 1, (wd - 1) // 2 + 1, 3)
        np.testing.assert_allclose(y2, y1[:, ::2, ::2, :], rtol=1e-13, atol=1e-13)
        _check_op(op, [x])
    # the rounding scale with stride 2 is the stride-1 scale subsampled
    np.testing.assert_allclose(op.abs_bound(x),
                               L.DepthwiseConv3x3(w, b).abs_bound(x)[:, ::2, ::2, :], rtol=1e-13)


def test_global_avgpool_and_pixel_reshapes():
    rng = np.random.default_rng(18)
    x = rng.standard_normal((2, 3, 4, 5))
    y, _ = L.GlobalAvgPool().forward(x)
    np.testing.assert_allclose(y[1, 2], sum(x[1, i, j, 2] for i in range(3) for j in range(4)) / 12,
                               rtol=1e-14)
    c = np.full((1, 2, 2, 3), 7.5)
    np.testing.assert_array_equal(L.GlobalAvgPool().forward(c)[0], np.full((1, 3), 7.5))
    _check_op(L.GlobalAvgPool(), [x])
    rows, _ = L.PixelRows().forward(x)
    assert rows.shape == (24, 5)
    np.testing.assert_array_equal(rows[1 * 12 + 2 * 4 + 3], x[1, 2, 3])   # row (n, h, w)
    np.testing.assert_array_equal(L.PixelMap(2, 3, 4).forward(rows)[0], x)
    _check_op(L.PixelRows(), [x])
    _check_op(L.PixelMap(2, 3, 4), [rows])


def test_maxpool_first_max_and_grad():
    x = np.zeros((1, 2, 4, 1))
    x[0, :, :, 0] = [[1, 3, 2, 2], [3, 0, 2, 2]]   # window 1: tie 3/3, window 2: all equal
    y, (_, arg) = L.MaxPool2x2().forward(x)
    np.testing.assert_array_equal(y[0, 0, :, 0], [3, 2])
    np.testing.assert_array_equal(arg[0, 0, :, 0], [1, 0])  # first maximum in row-major order
    rng = np.random.default_rng(7)
    _check_op(L.MaxPool2x2(), [rng.permutation(64).reshape(2, 4, 4, 2).astype(float)])


def test_losses_closed_values_and_grads():
    loss, dz = xent(np.zeros((4, 10)), np.array([0, 3, 9, 3]))
    assert loss == pytest.approx(math.log(10), rel=1e-15)
    np.testing.assert_allclose(dz.sum(axis=1), 0.0, atol=1e-16)
    y = np.random.default_rng(8).standard_normal((3, 5))
    assert mse(y, y)[0] == 0.0
    rng = np.random.default_rng(9)
    z = rng.standard_normal((5, 10)) * 3
    lab = rng.integers(0, 10, 5)
    t = rng.standard_normal((5, 10))
    for fn, other in ((xent, lab), (mse, t)):
        _, g = fn(z, other)
        num, = _fd_check(lambda: fn(z, other)[0], [z])
        np.testing.assert_allclose(g, num, rtol=1e-6, atol=1e-9)


def test_xent_stable_for_large_logits():
    z = np.array([[1000.0, 0.0], [0.0, -1000.0]])
    loss, _ = xent(z, np.array([0, 0]))
    assert loss == pytest.approx(0.0, abs=1e-12)


def _brute_abs_conv(x, w, b, depthwise):
    """sum over taps (and input channels) of |x||w|, plus |b|, by direct loops
    over every output element; zero padding 1, stride 1."""
    n, h, wd, c = x.shape
    cout = w.shape[-1] if depthwise else w.shape[0]
    s = np.zeros((n, h, wd, cout))
    for i in range(n):
        for y in range(h):
            for xx in range(wd):
                for o in range(cout):
                    acc = abs(b[o])
                    for r in range(3):
                        for q in range(3):
                            yy, xq = y + r - 1, xx + q - 1
                            if not (0 <= yy < h and 0 <= xq < wd):
                                continue
                            if depthwise:
                                acc += abs(x[i, yy, xq, o]) * abs(w[r, q, o])
                            else:
                                for ci in range(c):
                                    acc += abs(x[i, yy, xq, ci]) * abs(w[o, r, q, ci])
                    s[i, y, xx, o] = acc
    return s


def test_abs_bounds_are_the_absolute_sums():
    """The rounding scales S = sum |x||w| + |b| that decide which ReLU and
    max-pool decisions a float32 run may take differently (and the depthwise
    kernels' tolerance) against direct loops: a wrong scale would silently widen
    or narrow the accepted set."""
    rng = np.random.default_rng(11)
    x = rng.standard_normal((2, 4, 5, 3))
    w = rng.standard_normal((4, 3, 3, 3))
    b = rng.standard_normal(4)
    conv = L.Conv3x3(L.Param("w", w), L.Param("b", b))
    np.testing.assert_allclose(conv.abs_bound(x), _brute_abs_conv(x, w, b, False), rtol=1e-13)
    assert np.all(conv.abs_bound(x) >= np.abs(conv.forward(x)[0]))
    wd = rng.standard_normal((3, 3, 3))
    dw = L.DepthwiseConv3x3(L.Param("w", wd), L.Param("b", b[:3]))
    np.testing.assert_allclose(dw.abs_bound(x), _brute_abs_conv(x, wd, b[:3], True), rtol=1e-13)
    xl = rng.standard_normal((5, 7))
    wl = rng.standard_normal((3, 7))
    lin = L.Linear(L.Param("w", wl), L.Param("b", b[:3]))
    want = np.array([[sum(abs(xl[m, k] * wl[n, k]) for k in range(7)) + abs(b[n])
                      for n in range(3)] for m in range(5)])
    np.testing.assert_allclose(lin.abs_bound(xl), want, rtol=1e-13)
