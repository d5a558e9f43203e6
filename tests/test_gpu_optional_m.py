"""Adagrad and RMSprop without momentum keep no m: every updating entry point takes
m = NULL for them and must then give exactly the W, v (and bf16 shadow) it gives
with an m tensor, which it leaves unchanged; both match the oracle."""
import numpy as np
import pytest

from oracle import layers as OL
from oracle import optim as OO

pytestmark = pytest.mark.gpu

TOL = 1e-4
HYPERS = {
    "adagrad": dict(kind="adagrad", lr=0.01, eps=1e-10, weight_decay=1e-4),
    "rmsprop": dict(kind="rmsprop", lr=1e-3, alpha=0.99, eps=1e-8, weight_decay=1e-4),
}


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
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


def _bf16_bits(a):
    u = np.ascontiguousarray(a, np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


class _P:
    """One parameter with a Fig. 7 optimizer's state; m given or NULL."""

    def __init__(self, torch, L, dev, shape, seed, with_m, shadow=False):
        r = np.random.default_rng(seed)
        self.w = (r.standard_normal(shape) * 0.1).astype(np.float32)
        self.v = ((0.5 + r.random(shape)) * 1e-2).astype(np.float32)
        self.m0 = (r.standard_normal(shape) * 0.01).astype(np.float32)
        self.W, self.V = _t(torch, dev, self.w), _t(torch, dev, self.v)
        self.M = _t(torch, dev, self.m0) if with_m else None
        self.S = (torch.as_tensor(_bf16_bits(self.w).view(np.int16)).to(dev) if shadow else None)
        self.p = L.OfParam(self.W.data_ptr(), self.M.data_ptr() if with_m else None,
                           self.V.data_ptr(), self.S.data_ptr() if shadow else None,
                           self.W.numel())

    def out(self):
        o = [self.W.cpu().numpy(), self.V.cpu().numpy()]
        if self.S is not None:
            o.append(self.S.cpu().numpy())
        return o

    def oracle(self, g, hyper):
        P = OL.Param("p", self.w.astype(np.float64))
        P.v = self.v.astype(np.float64)
        P.step = 2
        P.grad = np.asarray(g, np.float64)
        OO.apply(P, hyper)
        return P


def _run_all(torch, L, dev, hyper, with_m):
    """Every updating entry point once; returns {case: (params, reference grads)}."""
    r = np.random.default_rng(3)
    s = torch.cuda.current_stream().cuda_stream
    out = {}
    opt = L.make_opt(hyper, 3)

    # a7 / a8: vector and rows gradients
    p = _P(torch, L, dev, (3001,), 1, with_m)
    g = (r.standard_normal(3001) * 0.05).astype(np.float32)
    G = _t(torch, dev, g)
    L.of_optimizer_step(1, (L.OfParam * 1)(p.p), (L.c_void_p * 1)(G.data_ptr()), opt, s)
    out["vector"] = (p, g)
    p = _P(torch, L, dev, (1027,), 2, with_m)
    gr = (r.standard_normal((5, 1027)) * 0.05).astype(np.float32)
    GR = _t(torch, dev, gr)
    L.of_elementwise_fused_update(p.p, GR.data_ptr(), 5, 0, opt, s)
    out["rows"] = (p, gr.astype(np.float64).sum(axis=0))

    # a5: backward-fusion, with its bias
    M, N, K = 72, 168, 200
    x = r.standard_normal((M, K)).astype(np.float32)
    dz = (r.standard_normal((M, N)) * 0.05).astype(np.float32)
    X, DZ = _t(torch, dev, x), _t(torch, dev, dz)
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 1)
    W, B = _P(torch, L, dev, (N, K), 3, with_m), _P(torch, L, dev, (N,), 4, with_m)
    ws = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_WEIGHT))
    L.of_linear_bwd_fused(d, DZ.data_ptr(), X.data_ptr(), W.p, B.p, None, None, opt, None, 0,
                          None, None, 0, ws.data_ptr(), ws.numel() * 4, s, None)
    dw = dz.astype(np.float64).T @ x.astype(np.float64)
    out["bwd_fused"] = (W, dw)
    out["bwd_fused_bias"] = (B, dz.astype(np.float64).sum(axis=0))

    # a2: forward-fusion prologue (M <= 64)
    Mf = 40
    xf = r.standard_normal((Mf, K)).astype(np.float32)
    gw = (r.standard_normal((N, K)) * 0.05).astype(np.float32)
    df = L.OfLinearDesc(Mf, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 0)
    WF = _P(torch, L, dev, (N, K), 5, with_m)
    XF, GW, Y = _t(torch, dev, xf), _t(torch, dev, gw), torch.empty((Mf, N), device=dev)
    wsf = _ws(torch, dev, L.of_linear_workspace_size(df, L.OF_LINEAR_FWD))
    L.of_linear_fwd_fused(df, XF.data_ptr(), WF.p, None, GW.data_ptr(), None, None, None, opt,
                          None, Y.data_ptr(), wsf.data_ptr(), wsf.numel() * 4, s)
    out["fwd_fused"] = (WF, gw)

    # a2: an update carried by another forward launch
    WC = _P(torch, L, dev, (N, K), 6, with_m)
    Wp = _P(torch, L, dev, (N, K), 7, True)
    carry = L.make_carry(opt, [(WC.p, GW.data_ptr(), 1)])
    L.of_linear_fwd_carry(df, XF.data_ptr(), Wp.p, None, None, Y.data_ptr(), carry,
                          wsf.data_ptr(), wsf.numel() * 4, s)
    out["carry"] = (WC, gw)

    # f1: merged data gradient + update (64 rows)
    dm = L.OfLinearDesc(64, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 0)
    xm = r.standard_normal((64, K)).astype(np.float32)
    dzm = (r.standard_normal((64, N)) * 0.05).astype(np.float32)
    XM, DZM, DX = _t(torch, dev, xm), _t(torch, dev, dzm), torch.empty((64, K), device=dev)
    WM = _P(torch, L, dev, (N, K), 8, with_m)
    wsm = _ws(torch, dev, L.of_linear_workspace_size(dm, L.OF_LINEAR_BWD_MERGED))
    L.of_linear_bwd_merged(dm, DZM.data_ptr(), XM.data_ptr(), WM.p, None, None, None, opt, None,
                           0, DX.data_ptr(), wsm.data_ptr(), wsm.numel() * 4, s)
    out["merged"] = (WM, dzm.astype(np.float64).T @ xm.astype(np.float64))

    # a6: convolution weight gradient + update
    cd = L.OfConvDesc(4, 6, 6, 8, 16, L.OF_ACT_NONE, 1)
    xc = r.standard_normal((4, 6, 6, 8)).astype(np.float32)
    dyc = (r.standard_normal((4, 6, 6, 16)) * 0.05).astype(np.float32)
    WCV, BCV = _P(torch, L, dev, (16, 3, 3, 8), 9, with_m), _P(torch, L, dev, (16,), 10, with_m)
    XC, DYC = _t(torch, dev, xc), _t(torch, dev, dyc)
    wsc = _ws(torch, dev, L.of_conv_workspace_size(cd, 2))
    L.of_conv_wgrad_fused(cd, DYC.data_ptr(), XC.data_ptr(), WCV.p, BCV.p, None, None, opt,
                          wsc.data_ptr(), wsc.numel() * 4, s)
    conv = OL.Conv3x3(OL.Param("w", WCV.w.astype(np.float64)), OL.Param("b", BCV.w.astype(np.float64)))
    _, ctx = conv.forward(xc.astype(np.float64))
    _, (dwc, dbc) = conv.backward(ctx, dyc.astype(np.float64))
    out["conv"] = (WCV, dwc)

    # bf16 operands: backward-fusion rewrites the bf16 shadow too
    db = L.OfLinearDesc(M, N, K, 0, 0, L.OF_BF16, L.OF_ACT_NONE, 0)
    WB = _P(torch, L, dev, (N, K), 11, with_m, shadow=True)
    wsb = _ws(torch, dev, L.of_linear_workspace_size(db, L.OF_LINEAR_BWD_WEIGHT))
    L.of_linear_bwd_fused(db, DZ.data_ptr(), X.data_ptr(), WB.p, None, None, None, opt, None, 0,
                          None, None, 0, wsb.data_ptr(), wsb.numel() * 4, s, None)
    out["bf16"] = (WB, None)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("kind", sorted(HYPERS))
def test_null_m_matches_given_m_and_oracle(env, kind):
    torch, L, dev = env
    hyper = HYPERS[kind]
    a = _run_all(torch, L, dev, hyper, True)
    b = _run_all(torch, L, dev, hyper, False)
    for case in a:
        pa, g = a[case]
        pb, _ = b[case]
        for x, y in zip(pa.out(), pb.out()):
            np.testing.assert_array_equal(x, y, err_msg=case)
        # with m given, the optimizer leaves it as it was
        np.testing.assert_array_equal(pa.M.cpu().numpy(), pa.m0, err_msg=case)
        if g is not None:
            ref = pa.oracle(g, hyper)
            assert rel(pb.W.cpu().numpy(), ref.value) <= TOL, case
            assert rel(pb.V.cpu().numpy(), ref.v) <= TOL, case
