"""GPU parity of global-norm gradient clipping (forward-fusion's global-information
step, Appendix B.1, Table 1) through the C ABI.

* of_grad_clip_scale against the oracle's clip_scale (float64) on ragged vector
  gradients, row partials, more tensors than one launch takes, the capped
  case and non-finite gradients.
* A gradient scale given to an update is the same as scaling the gradient in
  fp32 first: bit for bit, for the eager optimizer pass, the rows-mode update,
  a carried update and the backward-fusion epilogue; a scale of 1 is
  bit-identical to none.
* K-step training with clipping under eager and forward-fusion against the
  oracle's clipped eager run; backward-fusion refuses the option.
"""
import math

import numpy as np
import pytest

import oracle
from oracle.optim import clip_scale
from parity import rel, check_param
from workloads import get_config, reduced_config, make_params, make_batch, make_eval_batch

pytestmark = pytest.mark.gpu

TOL = 1e-4
TOL_BF16 = 2e-2


@pytest.fixture(scope="module")
def env(gpu):
    import torch
    from paper_2104_00237_amd import _lib as L
    L.load()
    return torch, L, gpu


def _rows_sum_f32(g):
    """Row partials summed in row order in fp32 (the rows-mode update's value)."""
    s = g[0].astype(np.float32)
    for r in range(1, g.shape[0]):
        s = (s + g[r].astype(np.float32)).astype(np.float32)
    return s


def _clip_gpu(torch, L, dev, tensors, max_norm):
    """tensors: list of float32 arrays, 1-D (vector) or 2-D (row partials, padded rows)."""
    bufs, items = [], []
    for a in tensors:
        if a.ndim == 1:
            t = torch.as_tensor(a).to(dev)
            items.append((t.data_ptr(), a.size, 1, 0))
        else:
            rows, numel = a.shape
            ld = numel + 3                              # padded row stride
            pad = np.zeros((rows, ld), np.float32)
            pad[:, :numel] = a
            t = torch.as_tensor(pad).to(dev)
            items.append((t.data_ptr(), numel, rows, ld))
        bufs.append(t)
    out = torch.full((2,), float("nan"), device=dev)
    ws = torch.empty(L.OF_CLIP_WS_BYTES // 4, device=dev)
    L.of_grad_clip_scale(len(items), L.grad_refs(items), max_norm, out.data_ptr(),
                         out.data_ptr() + 4, ws.data_ptr(), L.OF_CLIP_WS_BYTES, 0)
    torch.cuda.synchronize()
    s, n = out.cpu().numpy().tolist()
    return s, n


def _ref(tensors, max_norm):
    vecs = [a if a.ndim == 1 else _rows_sum_f32(a) for a in tensors]
    return clip_scale([v.astype(np.float64) for v in vecs], max_norm)


@pytest.mark.parametrize("case", ["ragged", "rows", "many", "one"])
def test_clip_scale_matches_oracle(env, case):
    torch, L, dev = env
    r = np.random.default_rng({"ragged": 1, "rows": 2, "many": 3, "one": 4}[case])
    f = lambda *s: r.standard_normal(s).astype(np.float32)
    if case == "ragged":
        ts = [f(1000), f(37), f(4096 * 3 + 5), f(1), f(1 << 20)]
    elif case == "rows":
        ts = [f(999), f(5, 999), f(64, 1024), f(1, 7)]
    elif case == "many":   # more tensors than one launch takes
        ts = [f(int(n)) for n in r.integers(1, 3000, size=75)] + [f(3, 301)]
    else:
        ts = [f(12345)]
    ref_s, ref_n = _ref(ts, 1.0)
    s, n = _clip_gpu(torch, L, dev, ts, 1.0)
    assert ref_s < 1.0
    assert abs(n - ref_n) <= 1e-6 * ref_n
    assert abs(s - ref_s) <= 1e-6 * ref_s
    # a bound above the norm leaves the gradients alone: exactly 1
    s, _ = _clip_gpu(torch, L, dev, ts, 2.0 * ref_n)
    assert s == 1.0


def test_clip_scale_non_finite(env):
    torch, L, dev = env
    a = np.ones(100, np.float32)
    a[17] = np.nan
    s, n = _clip_gpu(torch, L, dev, [a], 1.0)
    assert math.isnan(s) and math.isnan(n)
    a[17] = np.inf
    s, n = _clip_gpu(torch, L, dev, [a], 1.0)
    assert s == 0.0 and n == math.inf


OPTS = {
    "sgd": dict(kind="sgd", lr=0.05, momentum=0.9, weight_decay=1e-3),
    "adam": dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-2),
    "adamw": dict(kind="adamw", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-2),
}


class _P:
    """Parameter with history on the device, and a copy for a second path."""

    def __init__(self, torch, L, dev, r, numel, kind, shadow=False):
        self.w0 = r.standard_normal(numel).astype(np.float32)
        self.m0 = (r.standard_normal(numel) * 0.1).astype(np.float32)
        self.v0 = (r.random(numel) * 0.01).astype(np.float32)
        self.torch, self.L, self.dev, self.kind = torch, L, dev, kind
        self.numel, self.shadow = numel, shadow
        self.copies = [self._make() for _ in range(2)]

    def _make(self):
        t = self.torch
        w = t.as_tensor(self.w0).to(self.dev)
        m = t.as_tensor(self.m0).to(self.dev)
        v = t.as_tensor(self.v0).to(self.dev) if self.kind != "sgd" else None
        wb = t.zeros(self.numel, dtype=t.int16, device=self.dev) if self.shadow else None
        return dict(w=w, m=m, v=v, wb=wb, p=self.L.param_of(w, m, v, wb))

    def same(self):
        a, b = self.copies
        for k in ("w", "m", "v", "wb"):
            if a[k] is not None:
                np.testing.assert_array_equal(a[k].cpu().numpy(), b[k].cpu().numpy(), err_msg=k)


@pytest.mark.parametrize("kind", ["sgd", "adam", "adamw"])
def test_scaled_update_is_fp32_scaled_gradient(env, kind):
    """opt.grad_scale = s gives the bits of the unscaled update on fl(g * s)."""
    torch, L, dev = env
    r = np.random.default_rng(7)
    s = np.float32(0.3183099)
    sc = torch.tensor([s, 1.0], dtype=torch.float32, device=dev)
    hyper = OPTS[kind]
    # eager multi-tensor pass (vector paths and a ragged tail)
    ps = [_P(torch, L, dev, r, n, kind) for n in (4096, 1001)]
    gs = [r.standard_normal(p.numel).astype(np.float32) for p in ps]
    G = [torch.as_tensor(g).to(dev) for g in gs]
    Gs = [torch.as_tensor((g * s).astype(np.float32)).to(dev) for g in gs]
    for step in (1, 2):
        for c, grads, scale in ((0, G, sc.data_ptr()), (1, Gs, None)):
            opt = L.make_opt(hyper, step, None, scale)
            arr = (L.OfParam * 2)(*[p.copies[c]["p"] for p in ps])
            L.of_optimizer_step(2, arr, (L.c_void_p * 2)(*[g.data_ptr() for g in grads]), opt, 0)
    torch.cuda.synchronize()
    for p in ps:
        p.same()
    # rows mode: the scale applies to the summed rows
    p = _P(torch, L, dev, r, 777, kind)
    rows = r.standard_normal((5, 777)).astype(np.float32)
    Gr = torch.as_tensor(rows).to(dev)
    Gv = torch.as_tensor((_rows_sum_f32(rows) * s).astype(np.float32)).to(dev)
    L.of_elementwise_fused_update(p.copies[0]["p"], Gr.data_ptr(), 5, 777,
                                  L.make_opt(hyper, 1, None, sc.data_ptr()), 0)
    L.of_elementwise_fused_update(p.copies[1]["p"], Gv.data_ptr(), 1, 0,
                                  L.make_opt(hyper, 1), 0)
    torch.cuda.synchronize()
    p.same()
    # a scale of exactly 1 is the unscaled update
    p = _P(torch, L, dev, r, 3000, kind)
    g = torch.as_tensor(r.standard_normal(3000).astype(np.float32)).to(dev)
    for c, scale in ((0, sc.data_ptr() + 4), (1, None)):
        L.of_optimizer_step(1, (L.OfParam * 1)(p.copies[c]["p"]), (L.c_void_p * 1)(g.data_ptr()),
                            L.make_opt(hyper, 3, None, scale), 0)
    torch.cuda.synchronize()
    p.same()


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_scaled_carry_and_backward_fusion(env, dt):
    """A carried update and the backward-fusion epilogue read the same scale:
    bit-identical to the eager pass with that scale."""
    torch, L, dev = env
    r = np.random.default_rng(11)
    bf16 = dt == "bf16"
    M, N, K = 300, 256, 200
    sc = torch.tensor([0.625], dtype=torch.float32, device=dev)
    hyper = OPTS["adamw"]
    opt = L.make_opt(hyper, 2, None, sc.data_ptr())
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_BF16 if bf16 else L.OF_F32, L.OF_ACT_RELU, 1)
    X = torch.as_tensor(r.standard_normal((M, K)).astype(np.float32)).to(dev)
    DZ = torch.as_tensor((r.standard_normal((M, N)) * 1e-2).astype(np.float32)).to(dev)
    W = _P(torch, L, dev, r, N * K, "adamw", shadow=bf16)
    B = _P(torch, L, dev, r, N, "adamw")
    ws = torch.empty(1 << 24, device=dev)
    wsa = (ws.data_ptr(), ws.numel() * 4)
    # eager: dW, db, then the optimizer pass with the scale (copy 1)
    DW = torch.empty(N, K, device=dev)
    DB = torch.empty(N, device=dev)
    L.of_linear_bwd_weight(d, DZ.data_ptr(), X.data_ptr(), DW.data_ptr(), DB.data_ptr(), 0, *wsa, 0)
    arr = (L.OfParam * 2)(W.copies[1]["p"], B.copies[1]["p"])
    L.of_optimizer_step(2, arr, (L.c_void_p * 2)(DW.data_ptr(), DB.data_ptr()), opt, 0)
    # backward-fusion (copy 0)
    L.of_linear_bwd_fused(d, DZ.data_ptr(), X.data_ptr(), W.copies[0]["p"], B.copies[0]["p"],
                          None, None, opt, None, 0, None, None, 0, *wsa, 0, None)
    torch.cuda.synchronize()
    W.same()
    B.same()
    # forward-fusion: the same updates carried by another forward
    W2 = _P(torch, L, dev, r, N * K, "adamw", shadow=bf16)
    B2 = _P(torch, L, dev, r, N, "adamw")
    arr = (L.OfParam * 2)(W2.copies[1]["p"], B2.copies[1]["p"])
    L.of_optimizer_step(2, arr, (L.c_void_p * 2)(DW.data_ptr(), DB.data_ptr()), opt, 0)
    carry = L.make_carry(opt, [(W2.copies[0]["p"], DW.data_ptr(), 1),
                               (B2.copies[0]["p"], DB.data_ptr(), 1)])
    Wf = _P(torch, L, dev, r, N * K, "adamw", shadow=bf16)
    bf = torch.zeros(N, device=dev)
    Y = torch.empty(M, N, device=dev)
    L.of_linear_fwd_carry(d, X.data_ptr(), Wf.copies[0]["p"], bf.data_ptr(), None, Y.data_ptr(),
                          carry, *wsa, 0)
    torch.cuda.synchronize()
    W2.same()
    B2.same()


def _gpu_run(torch, cfg, ordering, steps, dev):
    from paper_2104_00237_amd.trainer import Trainer
    tr = Trainer(cfg, make_params(cfg), dev)
    scales = []
    for t in range(1, steps + 1):
        x, y = make_batch(cfg, t)
        tr.step(torch.as_tensor(x).to(dev), torch.as_tensor(y).to(dev), ordering)
        scales.append(tr.clip_out.cpu().numpy().tolist())
    losses = tr.loss_history()
    if ordering == "ff":
        tr.flush()
    xe, ye = make_eval_batch(cfg)
    ev = tr.eval_loss(torch.as_tensor(xe).to(dev), torch.as_tensor(ye).to(dev))
    st = tr.state()
    st.update(losses=losses, eval_loss=ev, scales=scales)
    return st


def _clipped(cfg):
    """cfg with clip_norm at half the first step's gradient norm (oracle)."""
    g = oracle.run(cfg, "eager", steps=1, snapshots=(1,))["snapshots"][1]["grad"]
    norm = float(np.linalg.norm(np.concatenate([g[k].ravel() for k in g])))
    cfg = dict(cfg)
    cfg["opt"] = dict(cfg["opt"], clip_norm=0.5 * norm)
    return cfg


@pytest.mark.parametrize("name,how", [("mlp3", "full"), ("mlp8x1024", "reduced"),
                                      ("tblock12", "reduced")])
def test_clipped_training_parity(env, name, how):
    torch, L, dev = env
    cfg = _clipped(reduced_config(name) if how == "reduced" else get_config(name))
    K = cfg["steps"]
    tol = TOL_BF16 if cfg["dtype"] == "bf16" else TOL
    ref = oracle.run(cfg, "eager", steps=K)
    assert ref["clips"][0][0] < 1.0
    runs = {o: _gpu_run(torch, cfg, o, K, dev) for o in ("eager", "ff")}
    for o, st in runs.items():
        for t, ((s, n), (rs, rn)) in enumerate(zip(st["scales"], ref["clips"])):
            assert abs(n - rn) <= tol * rn, (o, t, n, rn)
            assert abs(s - rs) <= tol * rs, (o, t, s, rs)
        assert rel(st["losses"], ref["losses"]) <= tol, (o, st["losses"], ref["losses"])
        assert abs(st["eval_loss"] - ref["eval_loss"]) <= tol * abs(ref["eval_loss"])
        for k in ref["params"]:
            check_param(st["params"][k], ref["params"][k], cfg["opt"], K, tol,
                        ref["min_sqrt_vhat"].get(k), what=f"{o} {k}")
            assert rel(st["m"][k], ref["m"][k]) <= tol, (o, k)
            assert st["step"][k] == K
    if cfg["batch"] <= 64:
        # same contractions in both orderings: identical bits
        for k in ref["params"]:
            np.testing.assert_array_equal(runs["ff"]["params"][k], runs["eager"]["params"][k])
    from paper_2104_00237_amd.trainer import Trainer
    tr = Trainer(cfg, make_params(cfg), dev)
    x, y = make_batch(cfg, 1)
    with pytest.raises(ValueError):
        tr.step(torch.as_tensor(x).to(dev), torch.as_tensor(y).to(dev), "bf")
