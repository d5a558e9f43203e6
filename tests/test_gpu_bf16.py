"""GPU parity of the bf16-operand contractions, LayerNorm, GELU and the
element-wise helpers against the oracle (fp64), through the C ABI.

bf16 contractions: the oracle rounds the same fp32 operands to bf16 and
multiplies in float64; the GPU's products of bf16 values are exact in fp32 and
only the fp32 accumulation differs, so these kernel-level checks hold to the
fp32 tolerance 1e-4 (the 2e-2 bf16 tolerance is for whole training runs).  The
bf16 shadow written by an update is compared bit for bit with the rounding of
the updated fp32 master.
"""
import numpy as np
import pytest

from oracle import layers as OL
from oracle import optim as OO
from oracle.bf16 import round_bf16

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


def _bf16_bits(a32):
    """bf16 bits of float32 values already on the bf16 grid (the shadow layout)."""
    u = np.ascontiguousarray(a32, dtype=np.float32).view(np.uint32)
    return (u >> 16).astype(np.uint16)


def _shadow(torch, dev, w32):
    bits = _bf16_bits(round_bf16(w32).astype(np.float32))
    return torch.as_tensor(bits.view(np.int16)).to(dev)


SHAPES = [  # (M, N, K): ragged tails, vector paths, split reductions, block shapes
    (37, 70, 53), (64, 128, 96), (130, 96, 44), (200, 168, 160), (512, 256, 1024),
    (4096, 1024, 1024), (4096, 3072, 1024), (4096, 1024, 4096),
    # eight-wave 128x256 tiles: a forward with a long reduction (vector and
    # scalar loads, ragged in every dimension), a data gradient with at least
    # 512 output tiles and a ragged reduction
    (2000, 2000, 2056), (1999, 2001, 2050), (4100, 300, 4090),
]


def _data(M, N, K, seed):
    r = np.random.default_rng(seed)
    x = r.standard_normal((M, K)).astype(np.float32).astype(np.float64)
    w = (r.standard_normal((N, K)) / np.sqrt(K)).astype(np.float32).astype(np.float64)
    b = (r.standard_normal(N) * 0.1).astype(np.float32).astype(np.float64)
    dz = (r.standard_normal((M, N)) * 1e-2).astype(np.float32).astype(np.float64)
    return x, w, b, dz


def _desc(L, M, N, K, act, bias=1):
    return L.OfLinearDesc(M, N, K, 0, 0, L.OF_BF16, L.ACTS[act], bias)


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("shadow", [True, False])
def test_bf16_fwd(env, M, N, K, shadow):
    torch, L, dev = env
    x, w, b, _ = _data(M, N, K, M + N + K)
    op = OL.Linear(OL.Param("w", w), OL.Param("b", b), bf16=True)
    z, _ = op.forward(x)
    gelu = OL.GELU().forward(z)[0]
    d = _desc(L, M, N, K, "gelu")
    X, Wt, Bt = _t(torch, dev, x), _t(torch, dev, w), _t(torch, dev, b)
    Wb = _shadow(torch, dev, w) if shadow else None
    Z = torch.full((M, N), float("nan"), device=dev)
    Y = torch.full((M, N), float("nan"), device=dev)
    ws = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_FWD))
    Wp = L.OfParam(Wt.data_ptr(), None, None, Wb.data_ptr() if shadow else None, w.size)
    L.of_linear_fwd(d, X.data_ptr(), Wp, Bt.data_ptr(), Z.data_ptr(), Y.data_ptr(),
                    ws.data_ptr(), ws.numel() * 4, 0)
    torch.cuda.synchronize()
    assert rel(Z.cpu().numpy(), z) <= TOL
    assert rel(Y.cpu().numpy(), gelu) <= TOL


@pytest.mark.parametrize("M,N,K", SHAPES)
def test_bf16_dgrad_wgrad(env, M, N, K):
    """dX = bf16(dZ) bf16(W) times GELU'(prev Z); dW = bf16(dZ)^T bf16(X); db = sum dZ."""
    torch, L, dev = env
    x, w, b, dz = _data(M, N, K, 3 * M + N + K)
    zprev = x   # the previous layer's pre-activation (its GELU derivative is applied)
    op = OL.Linear(OL.Param("w", w), OL.Param("b", b), bf16=True)
    (dx,), (dw, db) = op.backward(x, dz)
    (dx,), _ = OL.GELU().backward(zprev, dx)
    d = _desc(L, M, N, K, "none")
    X, Wt, DZ = _t(torch, dev, x), _t(torch, dev, w), _t(torch, dev, dz)
    Wb = _shadow(torch, dev, w)
    DX = torch.full((M, K), float("nan"), device=dev)
    DW = torch.full((N, K), float("nan"), device=dev)
    DB = torch.full((N,), float("nan"), device=dev)
    wsd = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_DATA))
    wsw = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_WEIGHT))
    Wp = L.OfParam(Wt.data_ptr(), None, None, Wb.data_ptr(), w.size)
    L.of_linear_bwd_data(d, DZ.data_ptr(), Wp, X.data_ptr(), L.OF_ACT_GELU, DX.data_ptr(),
                         wsd.data_ptr(), wsd.numel() * 4, 0)
    L.of_linear_bwd_weight(d, DZ.data_ptr(), X.data_ptr(), DW.data_ptr(), DB.data_ptr(), 0,
                           wsw.data_ptr(), wsw.numel() * 4, 0)
    torch.cuda.synchronize()
    assert rel(DX.cpu().numpy(), dx) <= TOL
    assert rel(DW.cpu().numpy(), dw) <= TOL
    assert rel(DB.cpu().numpy(), db) <= TOL


ADAMW = dict(kind="adamw", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)


@pytest.mark.parametrize("M,N,K", [(37, 70, 53), (200, 168, 160), (4096, 1024, 1024)])
def test_bf16_bwd_fused_adamw(env, M, N, K):
    """Backward-fusion with bf16 operands: the fused wgrad epilogue applies AdamW
    to W and b (fp32 masters) and rewrites the bf16 shadow; equal to the eager pair
    (wgrad -> optimizer) bit for bit and to the oracle within the tolerance."""
    torch, L, dev = env
    x, w, b, dz = _data(M, N, K, 5 * M + K)
    r = np.random.default_rng(9)
    mw = (r.standard_normal(w.shape) * 1e-3).astype(np.float32)
    vw = (r.random(w.shape) * 1e-5).astype(np.float32)
    mb = (r.standard_normal(b.shape) * 1e-3).astype(np.float32)
    vb = (r.random(b.shape) * 1e-5).astype(np.float32)
    op = OL.Linear(OL.Param("w", w), OL.Param("b", b), bf16=True)
    (dx_ref,), (dw, db) = op.backward(x, dz)
    refs = []
    for val, m, v, g in ((w, mw, vw, dw), (b, mb, vb, db)):
        P = OL.Param("p", val)
        P.m, P.v, P.step, P.grad = m.astype(np.float64), v.astype(np.float64), 6, g
        OO.apply(P, ADAMW)
        refs.append(P)
    d = _desc(L, M, N, K, "none")
    X, DZ = _t(torch, dev, x), _t(torch, dev, dz)
    out = {}
    for path in ("fused", "eager"):
        Wt, Mw, Vw, Bt, Mb, Vb = (_t(torch, dev, a) for a in (w, mw, vw, b, mb, vb))
        Wb = _shadow(torch, dev, w)
        Wp = L.OfParam(Wt.data_ptr(), Mw.data_ptr(), Vw.data_ptr(), Wb.data_ptr(), w.size)
        Bp = L.OfParam(Bt.data_ptr(), Mb.data_ptr(), Vb.data_ptr(), None, b.size)
        opt = L.make_opt(ADAMW, 7)
        wsw = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_WEIGHT))
        wsd = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_DATA))
        DX = torch.full((M, K), float("nan"), device=dev)
        if path == "fused":
            L.of_linear_bwd_fused(d, DZ.data_ptr(), X.data_ptr(), Wp, Bp, None, None, opt,
                                  None, L.OF_ACT_NONE, DX.data_ptr(), wsd.data_ptr(),
                                  wsd.numel() * 4, wsw.data_ptr(), wsw.numel() * 4, 0, None)
        else:
            DW = torch.empty((N, K), device=dev)
            DB = torch.empty((N,), device=dev)
            L.of_linear_bwd_data(d, DZ.data_ptr(), Wp, None, L.OF_ACT_NONE, DX.data_ptr(),
                                 wsd.data_ptr(), wsd.numel() * 4, 0)
            L.of_linear_bwd_weight(d, DZ.data_ptr(), X.data_ptr(), DW.data_ptr(), DB.data_ptr(),
                                   0, wsw.data_ptr(), wsw.numel() * 4, 0)
            import ctypes
            arr = (L.OfParam * 2)(Wp, Bp)
            gp = (ctypes.c_void_p * 2)(DW.data_ptr(), DB.data_ptr())
            L.of_optimizer_step(2, arr, gp, opt, 0)
        torch.cuda.synchronize()
        out[path] = [t.cpu().numpy() for t in (Wt, Mw, Vw, Bt, Mb, Vb, DX)] + \
            [Wb.cpu().numpy().view(np.uint16)]
    fw, fm, fv, fb, fmb, fvb, fdx, fsh = out["fused"]
    assert rel(fdx, dx_ref) <= TOL
    assert rel(fw, refs[0].value) <= TOL and rel(fm, refs[0].m) <= TOL
    assert rel(fv, refs[0].v) <= TOL
    assert rel(fb, refs[1].value) <= TOL and rel(fmb, refs[1].m) <= TOL
    np.testing.assert_array_equal(fsh, _bf16_bits(round_bf16(fw.astype(np.float64)).astype(np.float32)))
    for a, e in zip(out["fused"], out["eager"]):
        np.testing.assert_array_equal(a, e)


@pytest.mark.parametrize("M,D", [(5, 7), (136, 96), (4096, 1024), (33, 1030)])
def test_layernorm(env, M, D):
    torch, L, dev = env
    r = np.random.default_rng(M + D)
    x = (r.standard_normal((M, D)) * 2 + 0.5).astype(np.float32).astype(np.float64)
    g = (1 + 0.1 * r.standard_normal(D)).astype(np.float32).astype(np.float64)
    bt = (0.1 * r.standard_normal(D)).astype(np.float32).astype(np.float64)
    dy = r.standard_normal((M, D)).astype(np.float32).astype(np.float64)
    res = r.standard_normal((M, D)).astype(np.float32).astype(np.float64)
    op = OL.LayerNorm(OL.Param("g", g), OL.Param("b", bt), 1e-5)
    y, ctx = op.forward(x)
    (dx,), (dg, db) = op.backward(ctx, dy)
    X, G, B, DY, RES = (_t(torch, dev, a) for a in (x, g, bt, dy, res))
    Y = torch.full((M, D), float("nan"), device=dev)
    MU = torch.empty(M, device=dev)
    RS = torch.empty(M, device=dev)
    L.of_layernorm_fwd(X.data_ptr(), M, D, G.data_ptr(), B.data_ptr(), 1e-5, Y.data_ptr(),
                       MU.data_ptr(), RS.data_ptr(), 0)
    rows = L.of_layernorm_partial_rows(M)
    assert 1 <= rows <= 64
    DX = torch.full((M, D), float("nan"), device=dev)
    DGR = torch.full((rows, D), float("nan"), device=dev)
    DBR = torch.full((rows, D), float("nan"), device=dev)
    L.of_layernorm_bwd(DY.data_ptr(), X.data_ptr(), MU.data_ptr(), RS.data_ptr(), G.data_ptr(),
                       RES.data_ptr(), M, D, DX.data_ptr(), DGR.data_ptr(), DBR.data_ptr(), 0)
    # the two halves computed by separate calls: the same bits
    DX2 = torch.full((M, D), float("nan"), device=dev)
    DGR2 = torch.full((rows, D), float("nan"), device=dev)
    DBR2 = torch.full((rows, D), float("nan"), device=dev)
    L.of_layernorm_bwd(DY.data_ptr(), X.data_ptr(), MU.data_ptr(), RS.data_ptr(), None, None, M,
                       D, None, DGR2.data_ptr(), DBR2.data_ptr(), 0)
    L.of_layernorm_bwd(DY.data_ptr(), X.data_ptr(), MU.data_ptr(), RS.data_ptr(), G.data_ptr(),
                       RES.data_ptr(), M, D, DX2.data_ptr(), None, None, 0)
    DG = torch.empty(D, device=dev)
    DB = torch.empty(D, device=dev)
    L.of_reduce_rows(DGR.data_ptr(), rows, 0, D, DG.data_ptr(), 0)
    L.of_reduce_rows(DBR.data_ptr(), rows, D, D, DB.data_ptr(), 0)
    torch.cuda.synchronize()
    assert rel(Y.cpu().numpy(), y) <= TOL
    assert rel(RS.cpu().numpy(), ctx[1][:, 0]) <= TOL
    assert rel(DX.cpu().numpy(), dx + res) <= TOL
    assert rel(DG.cpu().numpy(), dg) <= TOL
    assert rel(DB.cpu().numpy(), db) <= TOL
    # the row partials are what the fused update sums: their sum is the gradient
    assert rel(DGR.cpu().numpy().astype(np.float64).sum(0), dg) <= TOL
    for a, b in ((DX2, DX), (DGR2, DGR), (DBR2, DBR)):
        np.testing.assert_array_equal(a.cpu().numpy(), b.cpu().numpy())


@pytest.mark.parametrize("n", [1, 7, 4096, 1 << 20])
def test_add(env, n):
    torch, L, dev = env
    r = np.random.default_rng(n)
    a = r.standard_normal(n).astype(np.float32)
    b = r.standard_normal(n).astype(np.float32)
    A, B = _t(torch, dev, a), _t(torch, dev, b)
    O = torch.empty(n, device=dev)
    L.of_add(A.data_ptr(), B.data_ptr(), n, O.data_ptr(), 0)
    L.of_add(A.data_ptr(), B.data_ptr(), n, A.data_ptr(), 0)   # in place
    torch.cuda.synchronize()
    np.testing.assert_array_equal(O.cpu().numpy(), a + b)
    np.testing.assert_array_equal(A.cpu().numpy(), a + b)
