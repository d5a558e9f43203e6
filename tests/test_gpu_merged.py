"""GPU parity of of_linear_bwd_merged (backward-fusion with the data gradient merged
into the update's read of W) against the oracle (fp64), through the C ABI.

Tolerance: ||gpu - oracle||_inf / ||oracle||_inf <= 1e-4 (fp32 operands).  The merged
kernel sums the data gradient in a different order from of_linear_bwd_fused, so the
two are compared within that tolerance, not bit for bit; two runs of the merged
kernel on the same inputs are bit-identical (fixed reduction order).
"""
import numpy as np
import pytest

from oracle import layers as OL
from oracle import optim as OO

pytestmark = pytest.mark.gpu

TOL = 1e-4

HYPERS = {
    "sgd": dict(kind="sgd", lr=0.01, momentum=0.9, weight_decay=1e-4),
    "adam": dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0),
    "adamw": dict(kind="adamw", lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01),
    "adagrad": dict(kind="adagrad", lr=0.01, eps=1e-10, weight_decay=1e-4),
    "rmsprop": dict(kind="rmsprop", lr=1e-3, alpha=0.99, eps=1e-8, weight_decay=1e-4, momentum=0.9),
    "adadelta": dict(kind="adadelta", lr=1.0, rho=0.9, eps=1e-6, weight_decay=1e-4),
}


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


class _Param:
    """Device tensors of one parameter with a random history, and host copies."""

    def __init__(self, torch, L, dev, shape, kind, seed, step):
        r = np.random.default_rng(seed)
        self.w = (r.standard_normal(shape) * 0.1).astype(np.float32)
        self.m = (r.standard_normal(shape) * 0.01).astype(np.float32)
        if kind == "adadelta":
            self.m = np.abs(self.m) * 1e-2   # squared-update state is >= 0
        self.v = (r.random(shape) * 1e-4).astype(np.float32) if kind != "sgd" else None
        if kind in ("adagrad", "rmsprop", "adadelta"):
            # sqrt(v) >= 0.07: the 1/sqrt(v) sensitivity of the update to the
            # gradient's float32 rounding stays well inside the tolerance
            self.v = ((0.5 + r.random(shape)) * 1e-2).astype(np.float32)
        self.W, self.M = _t(torch, dev, self.w), _t(torch, dev, self.m)
        self.V = _t(torch, dev, self.v) if kind != "sgd" else None
        self.p = L.OfParam(self.W.data_ptr(), self.M.data_ptr(),
                           self.V.data_ptr() if self.V is not None else None, None,
                           self.W.numel())
        self.kind, self.step = kind, step

    def oracle(self, g, hyper, rows=None):
        """The oracle's update of the whole tensor (rows=None) or of some rows."""
        sel = (lambda a: a) if rows is None else (lambda a: a[rows])
        P = OL.Param("p", sel(self.w).astype(np.float64))
        P.m = sel(self.m).astype(np.float64)
        P.v = sel(self.v).astype(np.float64) if self.v is not None else np.zeros_like(P.m)
        P.step = self.step - 1
        P.grad = np.asarray(g, np.float64)
        OO.apply(P, hyper)
        return P

    def check(self, ref, rows=None, tol=TOL):
        sel = (lambda a: a) if rows is None else (lambda a: a[rows])
        assert rel(sel(self.W.cpu().numpy()), ref.value) <= tol
        assert rel(sel(self.M.cpu().numpy()), ref.m) <= tol
        if self.V is not None:
            assert rel(sel(self.V.cpu().numpy()), ref.v) <= tol


def _run_merged(torch, L, dev, d, DZ, X, Wp, Bp, gW, gb, hyper, step, PR, act, DX):
    ws = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_MERGED))
    L.of_linear_bwd_merged(d, DZ.data_ptr(), X.data_ptr(), Wp.p, Bp.p if Bp else None,
                           gW.data_ptr() if gW is not None else None,
                           gb.data_ptr() if gb is not None else None,
                           L.make_opt(hyper, step), PR.data_ptr() if PR is not None else None,
                           act, DX.data_ptr() if DX is not None else None,
                           ws.data_ptr(), ws.numel() * 4,
                           torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()


# (M, N, K): one and several row ranges, M <= 32 and <= 64, tails in N (also N % 4 != 0,
# scalar dZ loads) and in K (partial 128-column strips), a single token row.
SHAPES = [(64, 520, 520), (33, 10, 27), (1, 8, 4), (32, 128, 64), (64, 2048, 4096),
          (40, 1030, 300), (17, 4099, 130), (64, 1024, 1000)]


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("kind", ["sgd", "adam", "adamw", "adagrad", "rmsprop", "adadelta"])
def test_merged_matches_oracle(env, M, N, K, kind):
    """dX with the OLD W, the update of W and b from dZ^T X and sum(dZ)."""
    torch, L, dev = env
    r = np.random.default_rng(M * 7 + N * 3 + K)
    hyper, step = HYPERS[kind], 3
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
    _run_merged(torch, L, dev, d, DZ, X, Wp, Bp, None, None, hyper, step, PR, L.OF_ACT_RELU, DX)
    assert rel(DX.cpu().numpy(), dx) <= TOL
    Wp.check(refW)
    Bp.check(refB)


@pytest.mark.parametrize("M,N,K", [(64, 520, 520), (20, 300, 260)])
def test_merged_extra_gradients_gelu_and_strides(env, M, N, K):
    """A shared parameter's earlier gradient (gW, gb) is added before the update;
    GELU's derivative reads Z; X, prev and dX rows have stride ldx > K and dZ rows
    stride ldy > N."""
    torch, L, dev = env
    r = np.random.default_rng(5)
    hyper, step = HYPERS["adam"], 4
    ldx, ldy = K + 6, N + 3
    xf = r.standard_normal((M, ldx)).astype(np.float32)
    dzf = (r.standard_normal((M, ldy)) * 0.05).astype(np.float32)
    zprev = r.standard_normal((M, ldx)).astype(np.float32)
    x, dz, z = xf[:, :K], dzf[:, :N], zprev[:, :K]
    gw = (r.standard_normal((N, K)) * 0.02).astype(np.float32)
    gb = (r.standard_normal(N) * 0.02).astype(np.float32)
    Wp = _Param(torch, L, dev, (N, K), "adam", 11, step)
    Bp = _Param(torch, L, dev, (N,), "adam", 12, step)
    op = OL.Linear(OL.Param("w", Wp.w.astype(np.float64)), OL.Param("b", Bp.w.astype(np.float64)))
    (dx,), (dw, db) = op.backward(x.astype(np.float64), dz.astype(np.float64))
    z64 = z.astype(np.float64)
    dx = OL.GELU().backward(z64, dx)[0][0]
    refW = Wp.oracle(dw + gw.astype(np.float64), hyper)
    refB = Bp.oracle(db + gb.astype(np.float64), hyper)

    d = L.OfLinearDesc(M, N, K, ldx, ldy, L.OF_F32, L.OF_ACT_NONE, 1)
    X, DZ, PR = (_t(torch, dev, a) for a in (xf, dzf, zprev))
    GW, GB = _t(torch, dev, gw), _t(torch, dev, gb)
    DX = torch.full((M, ldx), float("nan"), device=dev)
    _run_merged(torch, L, dev, d, DZ, X, Wp, Bp, GW, GB, hyper, step, PR, L.OF_ACT_GELU, DX)
    out = DX.cpu().numpy()
    assert rel(out[:, :K], dx) <= TOL
    assert np.isnan(out[:, K:]).all()   # the stride padding is not written
    Wp.check(refW)
    Bp.check(refB)


def test_merged_first_layer_and_determinism(env):
    """With no dX (the first layer) only the update runs; the same inputs give the
    same bits twice, and agree with of_linear_bwd_fused within tolerance."""
    torch, L, dev = env
    M, N, K = 64, 2048, 4096
    r = np.random.default_rng(9)
    hyper, step = HYPERS["adam"], 2
    x = r.standard_normal((M, K)).astype(np.float32)
    dz = (r.standard_normal((M, N)) * 0.05).astype(np.float32)
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 0)
    X, DZ = _t(torch, dev, x), _t(torch, dev, dz)

    W0 = _Param(torch, L, dev, (N, K), "adam", 21, step)
    _run_merged(torch, L, dev, d, DZ, X, W0, None, None, None, hyper, step, None, 0, None)
    dw = dz.astype(np.float64).T @ x.astype(np.float64)
    W0.check(W0.oracle(dw, hyper))

    outs = []
    for _ in range(2):
        Wp = _Param(torch, L, dev, (N, K), "adam", 22, step)
        DX = torch.empty((M, K), device=dev)
        _run_merged(torch, L, dev, d, DZ, X, Wp, None, None, None, hyper, step, None, 0, DX)
        outs.append([t.cpu().numpy() for t in (DX, Wp.W, Wp.M, Wp.V)])
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)

    Wf = _Param(torch, L, dev, (N, K), "adam", 22, step)
    DXf = torch.empty((M, K), device=dev)
    wsd = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_DATA))
    wsw = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_WEIGHT))
    L.of_linear_bwd_fused(d, DZ.data_ptr(), X.data_ptr(), Wf.p, None, None, None,
                          L.make_opt(hyper, step), None, 0, DXf.data_ptr(), wsd.data_ptr(),
                          wsd.numel() * 4, wsw.data_ptr(), wsw.numel() * 4, 0, None)
    torch.cuda.synchronize()
    for a, b in zip(outs[0], (DXf, Wf.W, Wf.M, Wf.V)):
        assert rel(a, b.cpu().numpy()) <= TOL


def test_merged_full_size_sampled(env):
    """A 8192 x 8192 layer with 64 token rows and Adam (the parameter-bound stack's
    layer, in the launch configuration the benchmark times), checked on sampled rows
    of W, m, v and sampled columns of dX that the oracle computes one by one."""
    torch, L, dev = env
    M, N, K = 64, 8192, 8192
    hyper, step = HYPERS["adam"], 5
    g = torch.Generator(device="cpu").manual_seed(0)
    X = torch.randn(M, K, generator=g).to(dev)
    DZ = (torch.randn(M, N, generator=g) * 0.05).to(dev)
    Wd = (torch.randn(N, K, generator=g) * 0.01).to(dev)
    Md = (torch.randn(N, K, generator=g) * 0.001).to(dev)
    Vd = (torch.rand(N, K, generator=g) * 1e-6).to(dev)
    rows = np.sort(np.random.default_rng(1).choice(N, 24, replace=False))
    rows = np.concatenate([rows, [0, 31, 32, 1023, 1024, N - 1]])
    cols = np.sort(np.random.default_rng(2).choice(K, 24, replace=False))
    cols = np.concatenate([cols, [0, 127, 128, K - 1]])
    w_rows, m_rows, v_rows = (t[rows].cpu().numpy().astype(np.float64) for t in (Wd, Md, Vd))
    w_cols = Wd[:, cols].cpu().numpy().astype(np.float64)
    x, dz = X.cpu().numpy().astype(np.float64), DZ.cpu().numpy().astype(np.float64)

    p = L.OfParam(Wd.data_ptr(), Md.data_ptr(), Vd.data_ptr(), None, N * K)
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 0)
    ws = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_MERGED))
    DX = torch.empty((M, K), device=dev)
    L.of_linear_bwd_merged(d, DZ.data_ptr(), X.data_ptr(), p, None, None, None,
                           L.make_opt(hyper, step), None, 0, DX.data_ptr(), ws.data_ptr(),
                           ws.numel() * 4, 0)
    torch.cuda.synchronize()

    assert rel(DX[:, cols].cpu().numpy(), dz @ w_cols) <= TOL   # old W
    P = OL.Param("p", w_rows)
    P.m, P.v, P.step = m_rows, v_rows, step - 1
    P.grad = dz[:, rows].T @ x
    OO.apply(P, hyper)
    assert rel(Wd[rows].cpu().numpy(), P.value) <= TOL
    assert rel(Md[rows].cpu().numpy(), P.m) <= TOL
    assert rel(Vd[rows].cpu().numpy(), P.v) <= TOL


def _train(torch, cfg, steps, dev, merge):
    from paper_2104_00237_amd.trainer import Trainer
    from workloads import make_params, make_batch, make_eval_batch
    tr = Trainer(cfg, make_params(cfg), dev, merge_dgrad=merge)
    assert any(getattr(op, "merge_dgrad", False) for op in tr.ops) == merge
    for t in range(1, steps + 1):
        x, y = make_batch(cfg, t)
        tr.step(torch.as_tensor(x).to(dev), torch.as_tensor(y).to(dev), "bf")
    losses = tr.loss_history()
    xe, ye = make_eval_batch(cfg)
    ev = tr.eval_loss(torch.as_tensor(xe).to(dev), torch.as_tensor(ye).to(dev))
    st = tr.state()
    st.update(losses=losses, eval_loss=ev)
    return st


@pytest.mark.parametrize("name,how", [("mlp3", "full"), ("linear4x8192", "reduced")])
def test_merged_training_parity(env, name, how):
    """Backward-fusion with merged data gradients, K steps free-running, against the
    oracle's eager run (the orderings reach the same trajectory), and against the
    unmerged backward-fusion on the GPU within the same tolerance."""
    import oracle
    from parity import check_param
    from workloads import get_config, reduced_config
    torch, L, dev = env
    cfg = reduced_config(name) if how == "reduced" else get_config(name)
    K = cfg["steps"]
    ref = oracle.run(cfg, "eager", steps=K)
    st = _train(torch, cfg, K, dev, True)
    plain = _train(torch, cfg, K, dev, False)
    assert rel(st["losses"], ref["losses"]) <= TOL, (st["losses"], ref["losses"])
    assert abs(st["eval_loss"] - ref["eval_loss"]) <= TOL * abs(ref["eval_loss"])
    for k in ref["params"]:
        check_param(st["params"][k], ref["params"][k], cfg["opt"], K, TOL,
                    ref["min_sqrt_vhat"].get(k), what=f"merged {k}")
        assert rel(st["m"][k], ref["m"][k]) <= TOL, k
        if cfg["opt"]["kind"] != "sgd":
            assert rel(st["v"][k], ref["v"][k]) <= TOL, k
        assert st["step"][k] == ref["step"][k] == K
        assert st["count"][k] == 0
        assert rel(st["m"][k], plain["m"][k]) <= TOL, k
    assert all(st["updated"])


@pytest.mark.timeout(600)
def test_merged_window_full_size(env):
    """The full 4 x 8192^2 Adam stack, 64 rows: from the oracle's state after steps 0
    and 1 (fp32), one merged backward-fusion step against the oracle's next step.
    The chain has no activation, so the step has one correct outcome."""
    import oracle
    from parity import check_param
    from paper_2104_00237_amd.trainer import Trainer
    from workloads import get_config, make_params, make_batch
    torch, L, dev = env
    cfg = get_config("linear4x8192")
    ref = oracle.run(cfg, "eager", steps=1, snapshots={0, 1})
    for s in (0, 1):
        # the oracle's step s+1 from its state after step s (no ReLU: one outcome)
        _, cand_loss, b = next(iter(oracle.candidate_steps(cfg, ref["snapshots"][s], s + 1)))
        tr = Trainer(cfg, make_params(cfg), dev, merge_dgrad=True)
        assert all(op.merge_dgrad for op in tr.ops)
        a = ref["snapshots"][s]
        tr.load_state(a["params"], a["m"], a["v"], a["step"])
        x, y = make_batch(cfg, s + 1)
        tr.step(torch.as_tensor(x).to(dev), torch.as_tensor(y).to(dev), "bf")
        loss = tr.loss_history()
        st = tr.state()
        del tr
        torch.cuda.empty_cache()
        assert rel(loss, [cand_loss]) <= TOL
        for k in b["params"]:
            assert st["step"][k] == s + 1
            check_param(st["params"][k], b["params"][k], cfg["opt"], 1, TOL,
                        b["min_sqrt_vhat"].get(k), what=f"step {s + 1} {k}")
            assert rel(st["m"][k], b["m"][k]) <= TOL, (s, k)
            assert rel(st["v"][k], b["v"][k]) <= TOL, (s, k)


def test_merged_largest_supported_row(env):
    """K = 2^22, the widest row the merged kernel takes (its 32-bit buffer offsets
    stay in range there): 2 token rows, 8 output rows (128 MB of W), every output
    against the oracle."""
    torch, L, dev = env
    M, N, K = 2, 8, 1 << 22
    r = np.random.default_rng(17)
    hyper, step = HYPERS["adam"], 2
    x = r.standard_normal((M, K)).astype(np.float32)
    dz = (r.standard_normal((M, N)) * 0.05).astype(np.float32)
    Wp = _Param(torch, L, dev, (N, K), "adam", 18, step)
    dw = dz.astype(np.float64).T @ x.astype(np.float64)
    dx = dz.astype(np.float64) @ Wp.w.astype(np.float64)
    refW = Wp.oracle(dw, hyper)
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 0)
    X, DZ = _t(torch, dev, x), _t(torch, dev, dz)
    DX = torch.full((M, K), float("nan"), device=dev)
    _run_merged(torch, L, dev, d, DZ, X, Wp, None, None, None, hyper, step, None, 0, DX)
    assert rel(DX.cpu().numpy(), dx) <= TOL
    Wp.check(refW)
