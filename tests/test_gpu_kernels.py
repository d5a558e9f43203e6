"""GPU parity of each opfuse entry point against the oracle (fp64), through the C ABI.

Tolerance: max-norm relative error ||gpu - oracle||_inf / ||oracle||_inf <= 1e-4 for
fp32 paths; integer outputs (counters) and GPU-internal ordering comparisons are
bit-exact.
"""
import ctypes

import numpy as np
import pytest

from oracle import layers as OL
from oracle import optim as OO
from oracle.losses import xent, mse

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


SHAPES = [  # (M, N, K): tails in every dimension, split reductions, tiny and wide
    (32, 128, 64), (33, 10, 27), (72, 168, 200), (256, 1024, 1024), (64, 520, 520),
    (130, 96, 44), (300, 70, 257), (64, 2048, 4096), (1, 5, 3),
    # direct-load 32x32 tiles with tails: scalar loads (K % 4 != 0), partial blocks
    (300, 1030, 1001), (290, 1028, 1100),
    # few output tiles and a long reduction: direct tiles with a split
    (100, 50, 3000), (200, 30, 2050),
    # at most 64 rows against a wide weight: ragged columns and reduction splits
    (33, 1030, 2052), (17, 600, 4000), (1, 2048, 1024),
    # tall, narrow products (1x1 convolutions over pixel rows): narrow forward and
    # data-gradient tiles; weight gradients over 65k+ rows split up to 256 ways
    (70001, 23, 37), (66000, 45, 17), (20000, 150, 30), (17000, 20, 200),
    # many weight-gradient tiles over a moderate reduction: split 64x32 tiles
    (1500, 600, 500),
]


def _rng(seed):
    return np.random.default_rng(seed)


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("act", ["none", "relu"])
def test_linear_fwd(env, M, N, K, act):
    torch, L, dev = env
    r = _rng(M * 7 + N)
    x, w, b = r.standard_normal((M, K)), r.standard_normal((N, K)) * 0.1, r.standard_normal(N)
    x, w, b = (a.astype(np.float32).astype(np.float64) for a in (x, w, b))
    op = OL.Linear(OL.Param("w", w), OL.Param("b", b))
    z, _ = op.forward(x)
    y_ref = np.maximum(z, 0) if act == "relu" else z
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.ACTS[act], 1)
    X, Wt, Bt = _t(torch, dev, x), _t(torch, dev, w), _t(torch, dev, b)
    Y = torch.full((M, N), float("nan"), device=dev)
    Z = torch.full((M, N), float("nan"), device=dev)
    ws = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_FWD))
    Wp = L.OfParam(Wt.data_ptr(), None, None, None, N * K)
    L.of_linear_fwd(d, X.data_ptr(), Wp, Bt.data_ptr(), Z.data_ptr(), Y.data_ptr(), ws.data_ptr(),
                    ws.numel() * 4, 0)
    torch.cuda.synchronize()
    assert rel(Y.cpu().numpy(), y_ref) <= TOL
    assert rel(Z.cpu().numpy(), z) <= TOL


@pytest.mark.parametrize("M,N,K", SHAPES)
def test_linear_bwd_data_and_weight(env, M, N, K):
    torch, L, dev = env
    r = _rng(M + 3 * N + K)
    x, w = r.standard_normal((M, K)), r.standard_normal((N, K)) * 0.1
    dz, prev = r.standard_normal((M, N)), r.standard_normal((M, K))
    x, w, dz, prev = (a.astype(np.float32).astype(np.float64) for a in (x, w, dz, prev))
    op = OL.Linear(OL.Param("w", w), OL.Param("b", np.zeros(N)))
    (dx,), (dw, db) = op.backward(x, dz)
    dx_masked = np.where(prev > 0, dx, 0.0)
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 1)
    X, Wt, DZ, PR = (_t(torch, dev, a) for a in (x, w, dz, np.maximum(prev, 0)))
    DX = torch.full((M, K), float("nan"), device=dev)
    DW = torch.full((N, K), float("nan"), device=dev)
    DB = torch.full((N,), float("nan"), device=dev)
    wsd = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_DATA))
    wsw = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_WEIGHT))
    Wp = L.OfParam(Wt.data_ptr(), None, None, None, N * K)
    L.of_linear_bwd_data(d, DZ.data_ptr(), Wp, PR.data_ptr(), L.OF_ACT_RELU, DX.data_ptr(),
                         wsd.data_ptr(), wsd.numel() * 4, 0)
    L.of_linear_bwd_weight(d, DZ.data_ptr(), X.data_ptr(), DW.data_ptr(), DB.data_ptr(), 0,
                           wsw.data_ptr(), wsw.numel() * 4, 0)
    torch.cuda.synchronize()
    assert rel(DX.cpu().numpy(), dx_masked) <= TOL
    assert rel(DW.cpu().numpy(), dw) <= TOL
    assert rel(DB.cpu().numpy(), db) <= TOL
    # accumulate = 1 adds a second contribution
    L.of_linear_bwd_weight(d, DZ.data_ptr(), X.data_ptr(), DW.data_ptr(), DB.data_ptr(), 1,
                           wsw.data_ptr(), wsw.numel() * 4, 0)
    torch.cuda.synchronize()
    assert rel(DW.cpu().numpy(), 2 * dw) <= TOL
    assert rel(DB.cpu().numpy(), 2 * db) <= TOL


HYPERS = {
    "sgd": dict(kind="sgd", lr=0.01, momentum=0.9, weight_decay=1e-4),
    "adam": dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0),
    "adamw": dict(kind="adamw", lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01),
    # the other optimizers of Fig. 7
    "adagrad": dict(kind="adagrad", lr=0.01, eps=1e-10, weight_decay=1e-4),
    "rmsprop": dict(kind="rmsprop", lr=1e-3, alpha=0.99, eps=1e-8, weight_decay=1e-4, momentum=0.9),
    "adadelta": dict(kind="adadelta", lr=1.0, rho=0.9, eps=1e-6, weight_decay=1e-4),
}
FIG7 = ["adagrad", "rmsprop", "adadelta"]


class _Param:
    """Device tensors of one parameter with random history, and their oracle copy."""

    def __init__(self, torch, L, dev, shape, kind, seed, step):
        r = _rng(seed)
        self.w = r.standard_normal(shape).astype(np.float32) * 0.1
        self.m = r.standard_normal(shape).astype(np.float32) * 0.01 if step > 1 else np.zeros(shape, np.float32)
        if kind == "adadelta":
            self.m = np.abs(self.m) * 1e-2   # Adadelta's squared-update state is >= 0
        if kind in FIG7 and step > 1:
            # Adagrad / RMSprop divide by sqrt(v): a history with sqrt(v) >= 0.07
            # keeps the float32 rounding of a contraction's gradient (~1e-7) from
            # being amplified by 1/sqrt(v) past the tolerance.
            self.v = ((0.5 + r.random(shape)) * 1e-2).astype(np.float32)
        elif step > 1 and kind != "sgd":
            self.v = r.random(shape).astype(np.float32) * 1e-4
        else:
            self.v = np.zeros(shape, np.float32)
        self.W = _t(torch, dev, self.w)
        self.M = _t(torch, dev, self.m)
        self.V = _t(torch, dev, self.v)
        self.p = L.OfParam(self.W.data_ptr(), self.M.data_ptr(),
                           self.V.data_ptr() if kind != "sgd" else None, None, self.W.numel())
        self.kind, self.step = kind, step

    def oracle(self, g, hyper):
        P = OL.Param("p", self.w.astype(np.float64))
        P.m = self.m.astype(np.float64)
        P.v = self.v.astype(np.float64)
        P.step = self.step - 1
        P.grad = np.asarray(g, np.float64)
        OO.apply(P, hyper)
        return P

    def check(self, ref, tol=TOL):
        assert rel(self.W.cpu().numpy(), ref.value) <= tol
        assert rel(self.M.cpu().numpy(), ref.m) <= tol
        if self.kind != "sgd":
            assert rel(self.V.cpu().numpy(), ref.v) <= tol


@pytest.mark.parametrize("kind", ["sgd", "adam", "adamw"] + FIG7)
@pytest.mark.parametrize("step", [1, 7])
def test_optimizer_step_multi_tensor(env, kind, step):
    torch, L, dev = env
    shapes = [(1000, 37), (10,), (4097,), (3, 5), (65536,)]
    ps = [_Param(torch, L, dev, s, kind, i + 10 * step, step) for i, s in enumerate(shapes)]
    gs = [_rng(99 + i).standard_normal(s).astype(np.float32) for i, s in enumerate(shapes)]
    G = [_t(torch, dev, g) for g in gs]
    arr = (L.OfParam * len(ps))(*[p.p for p in ps])
    gp = (ctypes.c_void_p * len(ps))(*[g.data_ptr() for g in G])
    L.of_optimizer_step(len(ps), arr, gp, L.make_opt(HYPERS[kind], step), 0)
    torch.cuda.synchronize()
    for p, g in zip(ps, gs):
        p.check(p.oracle(g, HYPERS[kind]))


@pytest.mark.parametrize("kind", ["sgd", "adam", "adamw"] + FIG7)
@pytest.mark.parametrize("rows", [1, 5, 300])
def test_elementwise_fused_update(env, kind, rows):
    torch, L, dev = env
    n = 1027
    p = _Param(torch, L, dev, (n,), kind, 5, 3)
    g = _rng(6).standard_normal((rows, n + 3)).astype(np.float32)
    G = _t(torch, dev, g)
    if rows == 1:
        L.of_elementwise_fused_update(p.p, G.data_ptr(), 1, 0, L.make_opt(HYPERS[kind], 3), 0)
        gsum = g[0, :n]
    else:
        L.of_elementwise_fused_update(p.p, G.data_ptr(), rows, n + 3, L.make_opt(HYPERS[kind], 3), 0)
        gsum = g[:, :n].astype(np.float64).sum(axis=0)
    torch.cuda.synchronize()
    p.check(p.oracle(gsum, HYPERS[kind]))


@pytest.mark.parametrize("M,N,K", [(72, 168, 200), (256, 1024, 1024), (64, 520, 520), (33, 10, 27),
                                   (300, 70, 257),
                                   # 65k+ rows: split up to 256 ways, reduced with the update
                                   (70001, 23, 37), (66000, 45, 17), (1500, 600, 500)])
@pytest.mark.parametrize("kind", ["sgd", "adam"] + FIG7)
def test_bwd_fused_matches_oracle_and_eager_bits(env, M, N, K, kind):
    """Backward-fusion (Alg. 3): dgrad with the old W, then the update in the wgrad
    epilogue.  Checked against the oracle, and bit for bit against the eager pair
    (plain wgrad -> multi-tensor optimizer) on the same inputs."""
    torch, L, dev = env
    r = _rng(M + N + K)
    hyper = HYPERS[kind]
    step = 2
    x = r.standard_normal((M, K)).astype(np.float32)
    dz = (r.standard_normal((M, N)) * 0.05).astype(np.float32)
    prev = np.maximum(r.standard_normal((M, K)), 0).astype(np.float32)
    Wp = _Param(torch, L, dev, (N, K), kind, 1, step)
    Bp = _Param(torch, L, dev, (N,), kind, 2, step)
    op = OL.Linear(OL.Param("w", Wp.w.astype(np.float64)), OL.Param("b", Bp.w.astype(np.float64)))
    (dx,), (dw, db) = op.backward(x.astype(np.float64), dz.astype(np.float64))
    dx = np.where(prev > 0, dx, 0.0)
    refW, refB = Wp.oracle(dw, hyper), Bp.oracle(db, hyper)

    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 1)
    X, DZ, PR = (_t(torch, dev, a) for a in (x, dz, prev))
    DX = torch.full((M, K), float("nan"), device=dev)
    wsd = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_DATA))
    wsw = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_WEIGHT))
    side = torch.cuda.Stream()
    L.of_linear_bwd_fused(d, DZ.data_ptr(), X.data_ptr(), Wp.p, Bp.p, None, None,
                          L.make_opt(hyper, step), PR.data_ptr(), L.OF_ACT_RELU, DX.data_ptr(),
                          wsd.data_ptr(), wsd.numel() * 4, wsw.data_ptr(), wsw.numel() * 4,
                          torch.cuda.current_stream().cuda_stream, side.cuda_stream)
    torch.cuda.synchronize()
    assert rel(DX.cpu().numpy(), dx) <= TOL   # computed from the OLD W
    Wp.check(refW)
    Bp.check(refB)

    # Eager on the same inputs: plain wgrad, then the multi-tensor optimizer.
    We = _Param(torch, L, dev, (N, K), kind, 1, step)
    Be = _Param(torch, L, dev, (N,), kind, 2, step)
    DW = torch.empty((N, K), device=dev)
    DB = torch.empty((N,), device=dev)
    L.of_linear_bwd_weight(d, DZ.data_ptr(), X.data_ptr(), DW.data_ptr(), DB.data_ptr(), 0,
                           wsw.data_ptr(), wsw.numel() * 4, 0)
    arr = (L.OfParam * 2)(We.p, Be.p)
    gp = (ctypes.c_void_p * 2)(DW.data_ptr(), DB.data_ptr())
    L.of_optimizer_step(2, arr, gp, L.make_opt(hyper, step), 0)
    torch.cuda.synchronize()
    for a, b in ((We.W, Wp.W), (We.M, Wp.M), (Be.W, Bp.W), (Be.M, Bp.M)):
        np.testing.assert_array_equal(a.cpu().numpy(), b.cpu().numpy())
    if kind != "sgd":
        np.testing.assert_array_equal(We.V.cpu().numpy(), Wp.V.cpu().numpy())


@pytest.mark.parametrize("M,N,K", [(72, 168, 200), (256, 1024, 1024), (64, 520, 520), (33, 10, 27),
                                   (256, 300, 130), (1, 8, 4),
                                   # a wide weight and at most 64 rows: split reductions
                                   (64, 2048, 4096), (33, 1030, 2052), (17, 600, 4000),
                                   # enough columns for the plain forward's 64x128 tiles
                                   # (vector and scalar operand loads, ragged columns)
                                   (64, 4096, 4096), (40, 4200, 2050),
                                   # ragged columns and reduction on the vector path
                                   (48, 4100, 4100),
                                   # a tall, narrow forward (256x32 tiles)
                                   (70001, 23, 37)])
@pytest.mark.parametrize("kind", ["sgd", "adam", "adamw"] + FIG7)
def test_fwd_fused_matches_oracle_and_eager_bits(env, M, N, K, kind):
    """Forward-fusion (Alg. 2): the pending update is applied while W is loaded and
    the forward uses the updated values.  Checked against the oracle and bit for bit
    against the eager pair (multi-tensor optimizer -> plain forward).  More than 64
    rows span several row tiles: the update goes to a second buffer set (written
    by the first row tile) and the current set must stay untouched."""
    torch, L, dev = env
    r = _rng(M * N + K)
    hyper = HYPERS[kind]
    step = 4
    x = r.standard_normal((M, K)).astype(np.float32)
    gw = (r.standard_normal((N, K)) * 0.01).astype(np.float32)
    gb = (r.standard_normal(N) * 0.01).astype(np.float32)
    Wp = _Param(torch, L, dev, (N, K), kind, 3, step)
    Bp = _Param(torch, L, dev, (N,), kind, 4, step)
    refW, refB = Wp.oracle(gw, hyper), Bp.oracle(gb, hyper)
    op = OL.Linear(refW, refB)
    z, _ = op.forward(x.astype(np.float64))
    y_ref = np.maximum(z, 0)

    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.OF_ACT_RELU, 1)
    X, GW, GB = (_t(torch, dev, a) for a in (x, gw, gb))
    Y = torch.full((M, N), float("nan"), device=dev)
    ws = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_FWD))
    two = M > 64
    if two:
        Wo = _Param(torch, L, dev, (N, K), kind, 13, step)   # overwritten by the call
        Bo = _Param(torch, L, dev, (N,), kind, 14, step)
        before = [t.clone() for t in (Wp.W, Wp.M, Wp.V, Bp.W, Bp.M, Bp.V)]
    L.of_linear_fwd_fused(d, X.data_ptr(), Wp.p, Wo.p if two else None, GW.data_ptr(), Bp.p,
                          Bo.p if two else None, GB.data_ptr(), L.make_opt(hyper, step), None,
                          Y.data_ptr(), ws.data_ptr(), ws.numel() * 4, 0)
    torch.cuda.synchronize()
    if two:
        for a, b in zip(before, (Wp.W, Wp.M, Wp.V, Bp.W, Bp.M, Bp.V)):
            assert torch.equal(a, b)         # the current set is only read
        Wp, Bp = Wo, Bo
    Wp.check(refW)
    Bp.check(refB)
    assert rel(Y.cpu().numpy(), y_ref) <= TOL

    We = _Param(torch, L, dev, (N, K), kind, 3, step)
    Be = _Param(torch, L, dev, (N,), kind, 4, step)
    arr = (L.OfParam * 2)(We.p, Be.p)
    gp = (ctypes.c_void_p * 2)(GW.data_ptr(), GB.data_ptr())
    L.of_optimizer_step(2, arr, gp, L.make_opt(hyper, step), 0)
    Ye = torch.empty((M, N), device=dev)
    L.of_linear_fwd(d, X.data_ptr(), We.p, Be.W.data_ptr(), None, Ye.data_ptr(), ws.data_ptr(),
                    ws.numel() * 4, 0)
    torch.cuda.synchronize()
    # The update is the same per-element arithmetic: identical bits.
    np.testing.assert_array_equal(We.W.cpu().numpy(), Wp.W.cpu().numpy())
    np.testing.assert_array_equal(Be.W.cpu().numpy(), Bp.W.cpu().numpy())
    if M <= 64:
        # The plain forward shares forward-fusion's tiling while M <= 64.
        np.testing.assert_array_equal(Ye.cpu().numpy(), Y.cpu().numpy())
    else:
        assert rel(Ye.cpu().numpy(), Y.cpu().numpy()) <= TOL


@pytest.mark.parametrize("ldx", [4097, 4100])
def test_forward_row_strides(env, ldx):
    """A 64-row forward over a 2048 x 4096 weight with X rows of stride ldx: 4100
    keeps 128-bit operand loads, 4097 does not; the workspace query covers both."""
    torch, L, dev = env
    M, N, K = 64, 2048, 4096
    r = _rng(ldx)
    xf = r.standard_normal((M, ldx)).astype(np.float32)
    w = (r.standard_normal((N, K)) * 0.05).astype(np.float32)
    b = r.standard_normal(N).astype(np.float32)
    z = xf[:, :K].astype(np.float64) @ w.astype(np.float64).T + b
    d = L.OfLinearDesc(M, N, K, ldx, 0, L.OF_F32, L.OF_ACT_NONE, 1)
    X, Wt, Bt = _t(torch, dev, xf), _t(torch, dev, w), _t(torch, dev, b)
    Y = torch.full((M, N), float("nan"), device=dev)
    ws = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_FWD))
    L.of_linear_fwd(d, X.data_ptr(), L.OfParam(Wt.data_ptr(), None, None, None, N * K),
                    Bt.data_ptr(), None, Y.data_ptr(), ws.data_ptr(), ws.numel() * 4, 0)
    torch.cuda.synchronize()
    assert rel(Y.cpu().numpy(), z) <= TOL


@pytest.mark.parametrize("B,C", [(32, 10), (256, 10), (300, 17), (1, 1)])
def test_xent(env, B, C):
    torch, L, dev = env
    r = _rng(B + C)
    z = (r.standard_normal((B, C)) * 3).astype(np.float32)
    y = r.integers(0, C, B).astype(np.int64)
    loss_ref, dz_ref = xent(z.astype(np.float64), y)
    Z = _t(torch, dev, z)
    Yl = torch.as_tensor(y).to(dev)
    loss = torch.zeros(1, device=dev)
    DZ = torch.full((B, C), float("nan"), device=dev)
    L.of_xent_fwd_bwd(Z.data_ptr(), Yl.data_ptr(), B, C, 0, loss.data_ptr(), DZ.data_ptr(), 0)
    torch.cuda.synchronize()
    assert abs(loss.item() - loss_ref) <= TOL * max(1.0, abs(loss_ref))
    assert rel(DZ.cpu().numpy(), dz_ref) <= TOL


@pytest.mark.parametrize("M,D", [(64, 8192), (40, 520), (3, 7)])
def test_mse(env, M, D):
    torch, L, dev = env
    r = _rng(M + D)
    yv = r.standard_normal((M, D)).astype(np.float32)
    tv = r.standard_normal((M, D)).astype(np.float32)
    loss_ref, dy_ref = mse(yv.astype(np.float64), tv.astype(np.float64))
    Yt, Tt = _t(torch, dev, yv), _t(torch, dev, tv)
    loss = torch.zeros(1, device=dev)
    DY = torch.full((M, D), float("nan"), device=dev)
    ws = _ws(torch, dev, L.of_mse_workspace_size(M, D))
    L.of_mse_fwd_bwd(Yt.data_ptr(), Tt.data_ptr(), M, D, 0, loss.data_ptr(), DY.data_ptr(),
                     ws.data_ptr(), ws.numel() * 4, 0)
    torch.cuda.synchronize()
    assert abs(loss.item() - loss_ref) <= TOL * abs(loss_ref)
    assert rel(DY.cpu().numpy(), dy_ref) <= TOL


@pytest.mark.parametrize("n,blocks", [(4, 0), (4100, 3), (1 << 20, 0)])
def test_hbm_stream_probes(env, n, blocks):
    """The streaming probes behind the measured HBM ceilings do what they time:
    a copy equals its source, the read-modify-write adds 1 to every element in
    place, and a read writes nothing but possibly one float."""
    torch, L, dev = env
    src = torch.arange(n, dtype=torch.float32, device=dev)
    dst = torch.full((n,), -1.0, device=dev)
    L.of_hbm_stream(L.OF_STREAM_COPY, src.data_ptr(), dst.data_ptr(), n, blocks, 0)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    L.of_hbm_stream(L.OF_STREAM_RMW, None, dst.data_ptr(), n, blocks, 0)
    torch.cuda.synchronize()
    assert torch.equal(dst, src + 1)
    # three arrays updated side by side: every element of the first 12*(n//12)
    # gets +1, the rest is untouched
    n3 = n // 12 * 12
    if n3:
        L.of_hbm_stream(L.OF_STREAM_RMW3, None, dst.data_ptr(), n3, blocks, 0)
        torch.cuda.synchronize()
        assert torch.equal(dst[:n3], src[:n3] + 2)
        assert torch.equal(dst[n3:], src[n3:] + 1)
    sink = torch.full((n,), -1.0, device=dev)
    L.of_hbm_stream(L.OF_STREAM_READ, src.data_ptr(), sink.data_ptr(), n, blocks, 0)
    torch.cuda.synchronize()
    assert int((sink != -1.0).sum()) <= 1


@pytest.mark.parametrize("chunks", [1, 10, 256])
def test_hbm_stream_columns_probe(env, chunks):
    """The merged kernel's access pattern as a probe: three arrays of rows of 8192
    floats, chunks of 32 rows in at most 8 row ranges (10 chunks: ranges of 2,
    the last ones empty); two passes add 2 to every element and nothing else."""
    torch, L, dev = env
    n = 3 * 8192 * 32 * chunks
    src = torch.arange(n, dtype=torch.float32, device=dev) % 1000
    pad = torch.full((n + 64,), -7.0, device=dev)
    pad[:n] = src
    for _ in range(2):
        L.of_hbm_stream(L.OF_STREAM_RMW3_COLUMNS, None, pad.data_ptr(), n, 0, 0)
    torch.cuda.synchronize()
    assert torch.equal(pad[:n], src + 2)
    assert bool((pad[n:] == -7.0).all())
