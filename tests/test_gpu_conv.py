"""GPU parity of the convolution and max-pool entry points against the oracle.

Shapes cover scalar gathers (C = 3), vector gathers, odd sizes, reduction splits
and the VGG-11 layer shapes at batch 128 (first two convolutions in full; the
later ones on a reduced batch).  Max-pool argmax positions are bit-exact.
"""
import ctypes

import numpy as np
import pytest

from oracle import layers as OL
from oracle import optim as OO

pytestmark = pytest.mark.gpu

TOL = 1e-4


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.max(np.abs(b))
    return float(np.max(np.abs(a - b)) / (den if den > 0 else 1.0))


@pytest.fixture(scope="module")
def env(gpu):
    import torch
    from paper_2104_00237_amd import _lib as L
    L.load()
    return torch, L, gpu


def _t(torch, dev, a):
    return torch.as_tensor(np.ascontiguousarray(a, dtype=np.float32)).to(dev)


def _ws(torch, dev, nbytes):
    return torch.empty(max(16, (nbytes + 15) // 16 * 4), dtype=torch.float32, device=dev)


SHAPES = [  # N, H, W, C, Cout
    (2, 4, 4, 3, 8), (2, 6, 10, 3, 64), (1, 5, 7, 16, 24), (2, 8, 8, 40, 48),
    (3, 4, 4, 64, 36), (2, 2, 2, 512, 512), (128, 32, 32, 3, 64), (128, 16, 16, 64, 128),
    (16, 8, 8, 128, 256), (16, 4, 4, 256, 512), (32, 2, 2, 512, 512),
]


def _data(N, H, W, C, Co, seed):
    r = np.random.default_rng(seed)
    x = r.standard_normal((N, H, W, C)).astype(np.float32)
    w = (r.standard_normal((Co, 3, 3, C)) * np.sqrt(2.0 / (9 * C))).astype(np.float32)
    b = (r.standard_normal(Co) * 0.1).astype(np.float32)
    dy = (r.standard_normal((N, H, W, Co)) * 1e-2).astype(np.float32)
    return x, w, b, dy


@pytest.mark.parametrize("N,H,W,C,Co", SHAPES)
def test_conv_fwd(env, N, H, W, C, Co):
    torch, L, dev = env
    x, w, b, _ = _data(N, H, W, C, Co, N + H + C + Co)
    op = OL.Conv3x3(OL.Param("w", w.astype(np.float64)), OL.Param("b", b.astype(np.float64)))
    z, _ = op.forward(x.astype(np.float64))
    ref = np.maximum(z, 0)
    d = L.OfConvDesc(N, H, W, C, Co, L.OF_ACT_RELU, 1)
    X, Wt, Bt = _t(torch, dev, x), _t(torch, dev, w), _t(torch, dev, b)
    Y = torch.full((N, H, W, Co), float("nan"), device=dev)
    ws = _ws(torch, dev, L.of_conv_workspace_size(d, L.OF_CONV_FWD))
    L.of_conv_fwd(d, X.data_ptr(), L.OfParam(Wt.data_ptr(), None, None, None, w.size),
                  Bt.data_ptr(), Y.data_ptr(), ws.data_ptr(), ws.numel() * 4, 0)
    torch.cuda.synchronize()
    assert rel(Y.cpu().numpy(), ref) <= TOL


@pytest.mark.parametrize("N,H,W,C,Co", SHAPES)
def test_conv_bwd(env, N, H, W, C, Co):
    torch, L, dev = env
    x, w, b, dy = _data(N, H, W, C, Co, 7 * N + H + C + Co)
    prev = np.maximum(x, 0)   # the input is a ReLU output: mask prev > 0
    op = OL.Conv3x3(OL.Param("w", w.astype(np.float64)), OL.Param("b", b.astype(np.float64)))
    _, xp = op.forward(prev.astype(np.float64))
    (dx,), (dw, db) = op.backward(xp, dy.astype(np.float64))
    dx = np.where(prev > 0, dx, 0.0)
    d = L.OfConvDesc(N, H, W, C, Co, L.OF_ACT_RELU, 1)
    PR, Wt, DY = _t(torch, dev, prev), _t(torch, dev, w), _t(torch, dev, dy)
    DX = torch.full((N, H, W, C), float("nan"), device=dev)
    DW = torch.full((Co, 3, 3, C), float("nan"), device=dev)
    DB = torch.full((Co,), float("nan"), device=dev)
    wsd = _ws(torch, dev, L.of_conv_workspace_size(d, L.OF_CONV_BWD_DATA))
    wsw = _ws(torch, dev, L.of_conv_workspace_size(d, L.OF_CONV_BWD_WEIGHT))
    Wp = L.OfParam(Wt.data_ptr(), None, None, None, w.size)
    L.of_conv_bwd_data(d, DY.data_ptr(), Wp, PR.data_ptr(), L.OF_ACT_RELU, DX.data_ptr(),
                       wsd.data_ptr(), wsd.numel() * 4, 0)
    L.of_conv_bwd_weight(d, DY.data_ptr(), PR.data_ptr(), DW.data_ptr(), DB.data_ptr(), 0,
                         wsw.data_ptr(), wsw.numel() * 4, 0)
    torch.cuda.synchronize()
    assert rel(DX.cpu().numpy(), dx) <= TOL
    assert rel(DW.cpu().numpy(), dw) <= TOL
    assert rel(DB.cpu().numpy(), db) <= TOL


SGD = dict(kind="sgd", lr=0.1, momentum=0.9, weight_decay=5e-4)


@pytest.mark.parametrize("N,H,W,C,Co", [(2, 6, 10, 3, 64), (2, 8, 8, 40, 48), (128, 32, 32, 3, 64),
                                        (16, 4, 4, 256, 512), (32, 2, 2, 512, 512)])
def test_conv_wgrad_fused(env, N, H, W, C, Co):
    """Backward-fusion for a convolution: the filter-gradient contraction's epilogue
    applies SGD with momentum (the policy pi_2) to W and b.  Checked against the
    oracle and bit for bit against the eager pair (filter gradient -> optimizer)."""
    torch, L, dev = env
    x, w, b, dy = _data(N, H, W, C, Co, 3 * N + C)
    r = np.random.default_rng(5)
    mw = (r.standard_normal(w.shape) * 1e-3).astype(np.float32)
    mb = (r.standard_normal(b.shape) * 1e-3).astype(np.float32)
    op = OL.Conv3x3(OL.Param("w", w.astype(np.float64)), OL.Param("b", b.astype(np.float64)))
    _, xp = op.forward(x.astype(np.float64))
    _, (dw, db) = op.backward(xp, dy.astype(np.float64))
    refs = []
    for val, m, g in ((w, mw, dw), (b, mb, db)):
        P = OL.Param("p", val.astype(np.float64))
        P.m = m.astype(np.float64)
        P.step = 4
        P.grad = g
        OO.apply(P, SGD)
        refs.append(P)
    d = L.OfConvDesc(N, H, W, C, Co, L.OF_ACT_RELU, 1)
    X, DY = _t(torch, dev, x), _t(torch, dev, dy)
    bufs = {}
    for path in ("fused", "eager"):
        Wt, Mw, Bt, Mb = (_t(torch, dev, a) for a in (w, mw, b, mb))
        Wp = L.OfParam(Wt.data_ptr(), Mw.data_ptr(), None, None, w.size)
        Bp = L.OfParam(Bt.data_ptr(), Mb.data_ptr(), None, None, b.size)
        ws = _ws(torch, dev, L.of_conv_workspace_size(d, L.OF_CONV_BWD_WEIGHT))
        opt = L.make_opt(SGD, 5)
        if path == "fused":
            L.of_conv_wgrad_fused(d, DY.data_ptr(), X.data_ptr(), Wp, Bp, None, None, opt,
                                  ws.data_ptr(), ws.numel() * 4, 0)
        else:
            DW = torch.empty(w.shape, device=dev)
            DB = torch.empty(b.shape, device=dev)
            L.of_conv_bwd_weight(d, DY.data_ptr(), X.data_ptr(), DW.data_ptr(), DB.data_ptr(), 0,
                                 ws.data_ptr(), ws.numel() * 4, 0)
            arr = (L.OfParam * 2)(Wp, Bp)
            gp = (ctypes.c_void_p * 2)(DW.data_ptr(), DB.data_ptr())
            L.of_optimizer_step(2, arr, gp, opt, 0)
        torch.cuda.synchronize()
        bufs[path] = [t.cpu().numpy() for t in (Wt, Mw, Bt, Mb)]
    fw, fm, fb, fmb = bufs["fused"]
    assert rel(fw, refs[0].value) <= TOL and rel(fm, refs[0].m) <= TOL
    assert rel(fb, refs[1].value) <= TOL and rel(fmb, refs[1].m) <= TOL
    for a, e in zip(bufs["fused"], bufs["eager"]):
        np.testing.assert_array_equal(a, e)


@pytest.mark.parametrize("N,H,W,C", [(2, 4, 4, 3), (128, 32, 32, 64), (3, 6, 2, 5), (2, 2, 2, 512)])
def test_maxpool(env, N, H, W, C):
    torch, L, dev = env
    r = np.random.default_rng(N + H + C)
    # ReLU outputs: many exact zeros, so ties exercise the first-maximum rule
    x = np.maximum(r.standard_normal((N, H, W, C)), 0).astype(np.float32)
    x[:, ::2, ::2, ::3] = x[:, 1::2, 1::2, ::3]   # exact ties between positions 0 and 3
    dy = r.standard_normal((N, H // 2, W // 2, C)).astype(np.float32)
    op = OL.MaxPool2x2()
    y, ctx = op.forward(x.astype(np.float64))
    arg = ctx[1]
    (dx,), _ = op.backward(ctx, dy.astype(np.float64))
    dx_masked = np.where(x > 0, dx, 0.0)
    X, DYt = _t(torch, dev, x), _t(torch, dev, dy)
    Y = torch.empty((N, H // 2, W // 2, C), device=dev)
    A = torch.empty((N, H // 2, W // 2, C), dtype=torch.uint8, device=dev)
    DX = torch.full((N, H, W, C), float("nan"), device=dev)
    DX2 = torch.full((N, H, W, C), float("nan"), device=dev)
    L.of_maxpool2x2_fwd(X.data_ptr(), N, H, W, C, Y.data_ptr(), A.data_ptr(), 0)
    L.of_maxpool2x2_bwd(DYt.data_ptr(), A.data_ptr(), None, N, H, W, C, DX.data_ptr(), 0)
    L.of_maxpool2x2_bwd(DYt.data_ptr(), A.data_ptr(), X.data_ptr(), N, H, W, C, DX2.data_ptr(), 0)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(Y.cpu().numpy(), y)
    np.testing.assert_array_equal(A.cpu().numpy().astype(np.int32), arg)
    np.testing.assert_array_equal(DX.cpu().numpy(), dx)
    np.testing.assert_array_equal(DX2.cpu().numpy(), dx_masked)
