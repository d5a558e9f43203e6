"""Pins for the oracle's orderings (Alg. 2, Alg. 3) against the eager definition.

The paper states that forward- and backward-fusion only reorder the same
updates and leave the optimizer algorithm and the training result unchanged.
In float64 with identical per-element arithmetic that means bit-identical
parameters, histories, losses and counters.
"""
import numpy as np
import pytest

from oracle import run, new_model
from oracle import layers as L
from workloads import get_config, reduced_config

CASES = ["mlp3", "mlp8x1024", "linear4x8192", "tblock12", "vgg11", "mbv2"]


def _same(a, b):
    for k in ("params", "m", "v"):
        assert a[k].keys() == b[k].keys()
        for n in a[k]:
            np.testing.assert_array_equal(a[k][n], b[k][n], err_msg=f"{k}[{n}]")
    np.testing.assert_array_equal(a["losses"], b["losses"])
    assert a["eval_loss"] == b["eval_loss"]
    assert a["step"] == b["step"]


@pytest.mark.parametrize("name", CASES)
def test_orderings_bit_identical(name):
    cfg = reduced_config(name)
    e = run(cfg, "eager")
    f = run(cfg, "ff")
    b = run(cfg, "bf")
    _same(e, f)
    _same(e, b)
    K = cfg["steps"]
    assert all(s == K for s in e["step"].values())
    assert all(c == 0 for c in b["count"].values())
    # FF: every node that ran backward holds a pending update until the flush.
    assert not any(f["updated_before_flush"])
    assert all(f["updated"])
    # Training moved the parameters and the loss is finite.
    assert np.all(np.isfinite(e["losses"]))
    init = new_model(cfg).params
    assert any(np.any(e["params"][k] != init[k].value) for k in init)


def test_full_size_mlp3_orderings():
    cfg = get_config("mlp3")
    e, f, b = run(cfg, "eager"), run(cfg, "ff"), run(cfg, "bf")
    _same(e, f)
    _same(e, b)
    assert len(e["losses"]) == 5


@pytest.mark.parametrize("name", ["mlp3", "vgg11", "tblock12", "mbv2"])
def test_planted_dependency_violation_is_caught(name):
    """Updating theta before the input gradient is computed (against the rule after
    Alg. 3) must change the result: the invariant test can see the race."""
    cfg = reduced_config(name)
    e = run(cfg, "eager")
    bad = run(cfg, "bf", race_bug=True)
    # NaN (a diverged wrong run) counts as a difference too.
    assert any(np.any(~(np.abs(e["params"][k] - bad["params"][k]) <= 1e-6)) for k in e["params"])


def _shared_model(cfg):
    """x -> A -> relu -> B -> relu -> A (same operator again) -> relu -> C: A is used twice."""
    rng = np.random.default_rng(11)
    d = 12
    A = L.Linear(L.Param("A.w", rng.uniform(-0.5, 0.5, (d, d))), L.Param("A.b", np.zeros(d)))
    B = L.Linear(L.Param("B.w", rng.uniform(-0.5, 0.5, (d, d))), L.Param("B.b", np.zeros(d)))
    C = L.Linear(L.Param("C.w", rng.uniform(-0.5, 0.5, (4, d))), None)
    nodes = [(A, ["input"], "a1"), (L.ReLU(), ["a1"], "r1"), (B, ["r1"], "b"),
             (L.ReLU(), ["b"], "r2"), (A, ["r2"], "a2"), (L.ReLU(), ["a2"], "r3"),
             (C, ["r3"], "output")]
    params = {p.name: p for op in (A, B, C) for p in op.params}
    from oracle.train import Model
    return Model(nodes, params, "xent", cfg["opt"]), A


@pytest.mark.parametrize("opt", ["sgd", "adam"])
def test_shared_operator_updated_once_per_step(opt):
    cfg = get_config("mlp3" if opt == "sgd" else "mlp8x1024")
    rng = np.random.default_rng(12)
    batches = [(rng.standard_normal((6, 12)), rng.integers(0, 4, 6)) for _ in range(4)]
    results = {}
    for ordering in ("eager", "ff", "bf"):
        model, A = _shared_model(cfg)
        losses = []
        for x, y in batches:
            if ordering == "eager":
                losses.append(model.step_eager(x, y))
            elif ordering == "ff":
                losses.append(model.step_ff(x, y))
                assert A.updated is False
            else:
                losses.append(model.step_bf(x, y))
                assert all(p.count == 0 for p in model.params.values())
        if ordering == "ff":
            model.flush()
        assert all(p.step == len(batches) for p in model.params.values())
        results[ordering] = (losses, {k: p.value.copy() for k, p in model.params.items()})
    for ordering in ("ff", "bf"):
        assert results[ordering][0] == results["eager"][0]
        for k, v in results["eager"][1].items():
            np.testing.assert_array_equal(results[ordering][1][k], v)


def test_bf_counts_forward_uses():
    cfg = get_config("mlp3")
    model, A = _shared_model(cfg)
    x, y = np.ones((2, 12)), np.array([0, 1])
    out, _ = model.forward(x, before_node=lambda op: [setattr(p, "count", p.count + 1)
                                                      for p in op.params])
    assert A.w.count == 2 and model.params["B.w"].count == 1


def test_ff_first_iteration_applies_nothing():
    cfg = reduced_config("mlp3")
    model = new_model(cfg)
    before = {k: p.value.copy() for k, p in model.params.items()}
    x = np.random.default_rng(0).standard_normal((32, 64))
    y = np.zeros(32, dtype=np.int64)
    model.step_ff(x, y)
    for k, p in model.params.items():
        np.testing.assert_array_equal(p.value, before[k])
        assert p.step == 0 and p.grad is not None


@pytest.mark.parametrize("name,over", [
    ("mlp3", dict(dims=[5, 7, 6, 4], batch=3, classes=4)),
    # layer 3 applies layer 2's parameters again: their gradient sums both uses
    ("mlp4tied", dict(dims=[5, 6, 6, 6, 4], batch=3, classes=4)),
    ("linear4x8192", dict(dims=[6] * 5, batch=3)),
    ("tblock12", dict(blocks=2, hidden=6, ffn=10, batch=4, dtype="f32")),
    ("vgg11", dict(channels=[3, 4, 4, 4, 5, 5, 5, 5], batch=2)),
    # stride-1 and stride-2 depthwise layers, t = 1 and expanded blocks, a residual
    ("mbv2", dict(image=5, stem=3, blocks=[[1, 4, 1, 1], [2, 3, 1, 2], [2, 3, 1, 1]], head=5,
                  batch=2)),
])
def test_whole_model_gradient_finite_differences(name, over):
    """Backward through the whole graph (wiring, residuals, pooling, loss) vs float64
    central differences of the training loss, for every parameter element."""
    cfg = reduced_config(name, **over)
    from workloads import make_batch
    model = new_model(cfg)
    if name == "mbv2":
        # Zero biases leave exact zeros at ReLU inputs here (a depthwise pixel whose
        # neighbourhood is dead or padding sums to exactly 0), where central
        # differences straddle the kink; nonzero biases keep every input off it.
        rb = np.random.default_rng(1)
        for p in model.params.values():
            if p.name.endswith(".bias"):
                p.value[...] = rb.standard_normal(p.value.shape) * 0.1
    x, y = make_batch(cfg, 1)
    x = x.astype(np.float64)
    y = y if y.dtype == np.int64 else y.astype(np.float64)
    out, tape = model.forward(x)
    _, dout = model.loss_and_grad(out, y)
    model.backward(tape, dout)
    h = 1e-6
    rng = np.random.default_rng(0)
    for p in model.params.values():
        flat = p.value.reshape(-1)
        for i in rng.choice(flat.size, size=min(flat.size, 6), replace=False):
            old = flat[i]
            flat[i] = old + h
            lp = model.loss_and_grad(model.forward(x)[0], y)[0]
            flat[i] = old - h
            lm = model.loss_and_grad(model.forward(x)[0], y)[0]
            flat[i] = old
            num = (lp - lm) / (2 * h)
            assert p.grad.reshape(-1)[i] == pytest.approx(num, rel=1e-5, abs=1e-8), p.name


def test_ambiguous_decisions_and_candidates():
    """A pre-activation placed within float32 rounding of 0 is reported, and the
    candidate steps are the plain step (no flip) and the flipped one."""
    from oracle.train import ambiguous_relu_decisions, candidate_steps, Model
    cfg = reduced_config("mlp3", dims=[4, 3, 2], batch=2, classes=2, steps=1)
    from workloads import make_batch, make_params
    init = make_params(cfg)
    x, _ = make_batch(cfg, 1)
    # Make z[0, 1] of the first layer tiny: shift its bias so the value is ~1e-12.
    z = x.astype(np.float64) @ init["fc1.weight"].astype(np.float64).T
    init["fc1.bias"] = init["fc1.bias"].astype(np.float64)
    init["fc1.bias"][1] = -z[0, 1] + 1e-12
    model = new_model(cfg, init=init)
    dec = ambiguous_relu_decisions(model, x.astype(np.float64))
    assert [(d[1], d[2]) for d in dec] == [(0, 1)]
    state = dict(params=init, m={k: np.zeros(np.shape(v)) for k, v in init.items()},
                 v={k: np.zeros(np.shape(v)) for k, v in init.items()},
                 step={k: 0 for k in init})
    cands = list(candidate_steps(cfg, state, 1))
    assert len(cands) == 2 and cands[0][0] == () and len(cands[1][0]) == 1
    plain = run(cfg, "eager", steps=1, init=init)
    for k in plain["params"]:
        np.testing.assert_array_equal(cands[0][2]["params"][k], plain["params"][k])
    # the flip moves the first layer's gradient row of unit 1 only
    d = np.abs(cands[1][2]["params"]["fc1.weight"] - cands[0][2]["params"]["fc1.weight"])
    assert d[1].max() > 0 and d[0].max() == 0 and d[2].max() == 0


def _zero_state(init):
    z = {k: np.zeros(np.shape(v)) for k, v in init.items()}
    return dict(params=init, m=z, v=dict(z), step={k: 0 for k in init})


@pytest.mark.parametrize("name", ["mlp3", "vgg11"])
def test_decision_search_without_flips_is_the_eager_step(name):
    """Settling every node with no flipped decision reproduces the eager step."""
    from oracle.train import DecisionSearch
    from workloads import make_params
    cfg = reduced_config(name, steps=1)
    init = make_params(cfg)
    plain = run(cfg, "eager", steps=1, init=init)
    s = DecisionSearch(cfg, _zero_state(init), 1)
    assert s.loss == plain["losses"][0]
    while not s.done:
        s.accept(())
    st = s.finish()
    for k in plain["params"]:
        np.testing.assert_array_equal(st["params"][k], plain["params"][k])
        np.testing.assert_array_equal(st["m"][k], plain["m"][k])
        assert st["step"][k] == 1


def _settle_with(s, kind):
    """Walk the search, flipping the first open decision of `kind` met; return it.
    ReLU decisions are taken where no max-pool follows (there the incoming
    gradient is dense, so the flip changes the step)."""
    from oracle import layers as OLY
    chosen = None
    nodes = s.model.nodes
    while not s.done:
        pick = ()
        if chosen is None:
            for d in s.open_decisions():
                if d[0] == kind and not (kind == "relu" and
                                         isinstance(nodes[d[1] + 1][0], OLY.MaxPool2x2)):
                    pick = (d,)
                    chosen = d
                    break
        s.accept(pick)
    return chosen, s.finish()


def test_decision_search_relu_flip_is_a_flipped_mask():
    """A flipped ReLU decision equals the step of a model whose backward mask is
    inverted at that element (the oracle's own flip mechanism)."""
    from oracle.train import DecisionSearch, new_model
    from workloads import make_params, make_batch
    cfg = reduced_config("vgg11", steps=1)
    init = make_params(cfg)
    # a huge c makes every decision "ambiguous", so the walk has choices
    d, st = _settle_with(DecisionSearch(cfg, _zero_state(init), 1, c=1e12), "relu")
    assert d is not None
    model = new_model(cfg, init=init)
    _, i, idx, _ = d
    op = model.nodes[i][0]
    x, y = make_batch(cfg, 1)
    out, tape = model.forward(np.asarray(x, np.float64))
    op.flip = np.zeros(tape[i].shape, bool)
    op.flip[idx] = True
    loss, dout = model.loss_and_grad(out, y)
    model.backward(tape, dout)
    from oracle.optim import apply
    for p in model.params.values():
        apply(p, cfg["opt"])
    changed = 0
    for k, p in model.params.items():
        np.testing.assert_array_equal(st["params"][k], p.value)
        changed += int(np.any(st["params"][k] != run(cfg, "eager", steps=1, init=init)["params"][k]))
    assert changed > 0


def test_decision_search_pool_flip_routes_the_gradient():
    """A flipped max-pool decision equals the step of a model whose pool picks
    that window entry in the backward pass."""
    from oracle.train import DecisionSearch, new_model
    from oracle import layers as OLY
    from oracle.optim import apply
    from workloads import make_params, make_batch
    cfg = reduced_config("vgg11", steps=1)
    init = make_params(cfg)
    d, st = _settle_with(DecisionSearch(cfg, _zero_state(init), 1, c=1e12), "pool")
    assert d is not None
    _, i, idx, q = d
    model = new_model(cfg, init=init)
    op = model.nodes[i][0]
    assert isinstance(op, OLY.MaxPool2x2)
    x, y = make_batch(cfg, 1)
    out, tape = model.forward(np.asarray(x, np.float64))
    shape, arg = tape[i]
    assert arg[idx] != q
    arg = arg.copy()
    arg[idx] = q
    tape[i] = (shape, arg)
    loss, dout = model.loss_and_grad(out, y)
    model.backward(tape, dout)
    for p in model.params.values():
        apply(p, cfg["opt"])
    for k, p in model.params.items():
        np.testing.assert_array_equal(st["params"][k], p.value)


def test_tied_mlp_orderings_and_counts():
    """The tied MLP workload: eager, forward-fusion and backward-fusion give the same
    bits, each shared tensor is updated once per step (step = K) and has two forward
    uses per step, and its gradient is the sum of both uses' contributions (it differs
    from either use alone)."""
    cfg = get_config("mlp4tied")
    runs = {o: run(cfg, o) for o in ("eager", "ff", "bf")}
    for o in ("ff", "bf"):
        np.testing.assert_array_equal(runs[o]["losses"], runs["eager"]["losses"])
        for k in runs["eager"]["params"]:
            np.testing.assert_array_equal(runs[o]["params"][k], runs["eager"]["params"][k])
    assert set(runs["eager"]["step"].values()) == {cfg["steps"]}
    assert "fc3.weight" not in runs["eager"]["params"]
    model = new_model(cfg)
    x = np.random.default_rng(0).standard_normal((cfg["batch"], cfg["dims"][0]))
    model.forward(x, before_node=lambda op: [setattr(p, "count", p.count + 1) for p in op.params])
    assert model.params["fc2.weight"].count == 2 and model.params["fc1.weight"].count == 1


def test_ambiguous_depthwise_decision_and_flip():
    """A depthwise pre-activation placed within float32 rounding of 0 (through
    its bias) is reported with its NHWC index; the candidate that flips it
    differs from the plain step exactly as a hand-flipped ReLU mask does."""
    from oracle.train import ambiguous_relu_decisions, candidate_steps
    from workloads import make_batch, make_params
    cfg = reduced_config("mbv2", image=5, stem=3, blocks=[[2, 3, 1, 1]], head=4, batch=1, steps=1)
    init = {k: np.asarray(v, np.float64) for k, v in make_params(cfg).items()}
    rng = np.random.default_rng(4)
    for k in init:
        if k.endswith(".bias"):
            init[k] = rng.standard_normal(init[k].shape) * 0.1
    x, _ = make_batch(cfg, 1)
    x = x.astype(np.float64)
    model = new_model(cfg, init=init)
    env = {"input": x}
    for i, (op, ins, name) in enumerate(model.nodes):
        env[name] = op.forward(*[env[n] for n in ins])[0]
        if name == "blk1.d":
            node_relu = i + 1
    z = env["blk1.d"]
    # move channel 1's bias so that pixel (0, 2, 3) sits 1e-12 above zero
    init["blk1.dw.bias"][1] -= z[0, 2, 3, 1] - 1e-12
    model = new_model(cfg, init=init)
    dec = ambiguous_relu_decisions(model, x)
    assert [d[:-1] for d in dec] == [(node_relu, 0, 2, 3, 1)]
    state = dict(params=init, m={k: np.zeros(np.shape(v)) for k, v in init.items()},
                 v={k: np.zeros(np.shape(v)) for k, v in init.items()}, step={k: 0 for k in init})
    cands = list(candidate_steps(cfg, state, 1))
    assert len(cands) == 2 and len(cands[1][0]) == 1
    m2 = new_model(cfg, init=init)
    m2.nodes[node_relu][0].flip = np.zeros(z.shape, bool)
    m2.nodes[node_relu][0].flip[0, 2, 3, 1] = True
    _, y = make_batch(cfg, 1)
    m2.step_eager(x, y)
    for k, p in m2.params.items():
        np.testing.assert_array_equal(cands[1][2]["params"][k], p.value)
    assert any(np.any(cands[1][2]["params"][k] != cands[0][2]["params"][k]) for k in init)
