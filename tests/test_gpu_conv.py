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
    # a 3-channel stem of at most 32 filters over 65k pixels or more (its own tiling:
    # 256x32 forward tiles, a weight gradient split 256 ways), ragged filter count
    (6, 107, 107, 3, 29),
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
                                        (16, 4, 4, 256, 512), (32, 2, 2, 512, 512),
                                        (6, 107, 107, 3, 29)])
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


@pytest.mark.parametrize("N,H,W,C,Co", SHAPES)
@pytest.mark.parametrize("kind", ["sgd", "adam"])
def test_conv_fwd_fused(env, N, H, W, C, Co, kind):
    """Forward-fusion in the filter-tile prologue: y uses the updated filter and
    bias, which go to the second buffer set; the first set is left as it was.
    Against the oracle, and bit for bit against an update pass followed by the
    plain forward (the same contraction and per-element arithmetic)."""
    torch, L, dev = env
    hyper = (dict(kind="sgd", lr=0.1, momentum=0.9, weight_decay=5e-4) if kind == "sgd" else
             dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0))
    step = 3
    x, w, b, _ = _data(N, H, W, C, Co, N * 7 + C + Co)
    r = np.random.default_rng(C + Co)
    gw = (r.standard_normal(w.shape) * 0.05).astype(np.float32)
    gb = (r.standard_normal(Co) * 0.05).astype(np.float32)
    mw = (r.standard_normal(w.shape) * 0.01).astype(np.float32)
    mb = (r.standard_normal(Co) * 0.01).astype(np.float32)
    vw = (r.random(w.shape) * 1e-4).astype(np.float32)
    vb = (r.random(Co) * 1e-4).astype(np.float32)
    adam = kind != "sgd"

    def param(arrs):
        ts = [_t(torch, dev, a) for a in arrs]
        p = L.OfParam(ts[0].data_ptr(), ts[1].data_ptr(), ts[2].data_ptr() if adam else None,
                      None, ts[0].numel())
        return p, ts

    def fresh():
        return param((w, mw, vw)), param((b, mb, vb))

    def blank(shape):
        z = np.full(shape, np.nan, np.float32)
        return param((z, z, z))

    def oracle(val, g, m, v):
        P = OL.Param("p", val.astype(np.float64))
        P.m, P.v, P.step = m.astype(np.float64), v.astype(np.float64), step - 1
        P.grad = g.astype(np.float64)
        OO.apply(P, hyper)
        return P

    d = L.OfConvDesc(N, H, W, C, Co, L.OF_ACT_RELU, 1)
    ws = _ws(torch, dev, L.of_conv_workspace_size(d, 0))
    GW, GB = _t(torch, dev, gw), _t(torch, dev, gb)
    (Wp, Wt), (Bp, Bt) = fresh()
    (Wo, Wot), (Bo, Bot) = blank(w.shape), blank((Co,))
    Y = torch.full((N, H, W, Co), float("nan"), device=dev)
    L.of_conv_fwd_fused(d, _t(torch, dev, x).data_ptr(), Wp, Wo, GW.data_ptr(), Bp, Bo,
                        GB.data_ptr(), L.make_opt(hyper, step), Y.data_ptr(), ws.data_ptr(),
                        ws.numel() * 4, 0)
    torch.cuda.synchronize()
    rw, rb = oracle(w, gw, mw, vw), oracle(b, gb, mb, vb)
    conv = OL.Conv3x3(OL.Param("w", rw.value), OL.Param("b", rb.value))
    y_ref = np.maximum(conv.forward(x.astype(np.float64))[0], 0)
    assert rel(Y.cpu().numpy(), y_ref) <= TOL
    for got, ref in ((Wot[0], rw.value), (Wot[1], rw.m), (Bot[0], rb.value), (Bot[1], rb.m)):
        assert rel(got.cpu().numpy(), ref) <= TOL
    if adam:
        assert rel(Wot[2].cpu().numpy(), rw.v) <= TOL
    for t, a in zip(Wt + Bt, (w, mw, vw, b, mb, vb)):   # the first set is unchanged
        if t is not None:
            np.testing.assert_array_equal(t.cpu().numpy(), a)

    # eager pair: the multi-tensor update in place, then the plain forward
    (We, Wet), (Be, Bet) = fresh()
    arr = (L.OfParam * 2)(We, Be)
    gp = (ctypes.c_void_p * 2)(GW.data_ptr(), GB.data_ptr())
    L.of_optimizer_step(2, arr, gp, L.make_opt(hyper, step), 0)
    Ye = torch.empty_like(Y)
    L.of_conv_fwd(d, _t(torch, dev, x).data_ptr(), We, Bet[0].data_ptr(), Ye.data_ptr(),
                  ws.data_ptr(), ws.numel() * 4, 0)
    torch.cuda.synchronize()
    for a, b_ in ((Wot[0], Wet[0]), (Wot[1], Wet[1]), (Bot[0], Bet[0]), (Bot[1], Bet[1])):
        np.testing.assert_array_equal(a.cpu().numpy(), b_.cpu().numpy())
    if adam:
        np.testing.assert_array_equal(Wot[2].cpu().numpy(), Wet[2].cpu().numpy())
    # the same contraction unless the tiling model picked 128x128 (no LDS room
    # for the bias row: the fused forward runs 128x64 with the same splits)
    assert rel(Ye.cpu().numpy(), Y.cpu().numpy()) <= TOL
