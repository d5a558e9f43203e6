"""K-step training parity on the GPU: every ordering against the oracle's eager
run on the same seeded inputs, and the three GPU orderings bit for bit against
each other.  Steps and counters are compared exactly."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
from parity import rel, check_param, check_update, teachers, undetermined, _f32
from workloads import get_config, reduced_config, make_params, make_batch, make_eval_batch

pytestmark = pytest.mark.gpu

TOL = 1e-4
TOL_BF16 = 2e-2   # bf16 operands, fp32 accumulation


def _gpu_run(torch, cfg, ordering, steps, dev):
    from paper_2104_00237_amd.trainer import Trainer
    tr = Trainer(cfg, make_params(cfg), dev)
    for t in range(1, steps + 1):
        x, y = make_batch(cfg, t)
        tr.step(torch.as_tensor(x).to(dev), torch.as_tensor(y).to(dev), ordering)
    pending = [op.updated for op in tr.ops]
    losses = tr.loss_history()
    if ordering == "ff":
        tr.flush()
    xe, ye = make_eval_batch(cfg)
    ev = tr.eval_loss(torch.as_tensor(xe).to(dev), torch.as_tensor(ye).to(dev))
    st = tr.state()
    st.update(losses=losses, eval_loss=ev, pending=pending)
    return st


CASES = [
    ("mlp3", "full"),
    ("mlp8x1024", "reduced"),
    ("linear4x8192", "reduced"),
    ("vgg11", "reduced"),
    ("tblock12", "reduced"),
]


def _cfg(name, how):
    return reduced_config(name) if how == "reduced" else get_config(name)


@pytest.mark.parametrize("name,how", CASES)
def test_training_parity(gpu, name, how):
    import torch
    cfg = _cfg(name, how)
    K = cfg["steps"]
    tol = TOL_BF16 if cfg["dtype"] == "bf16" else TOL
    ref = oracle.run(cfg, "eager", steps=K)
    runs = {o: _gpu_run(torch, cfg, o, K, gpu) for o in ("eager", "ff", "bf")}
    worst = 0.0
    for o, st in runs.items():
        assert rel(st["losses"], ref["losses"]) <= tol, (o, st["losses"], ref["losses"])
        assert abs(st["eval_loss"] - ref["eval_loss"]) <= tol * abs(ref["eval_loss"])
        for k in ref["params"]:
            check_param(st["params"][k], ref["params"][k], cfg["opt"], K, tol,
                        ref["min_sqrt_vhat"].get(k), what=f"{o} {k}")
            assert rel(st["m"][k], ref["m"][k]) <= tol, (o, k)
            worst = max(worst, rel(st["m"][k], ref["m"][k]))
            if cfg["opt"]["kind"] != "sgd":
                assert rel(st["v"][k], ref["v"][k]) <= tol, (o, k)
            assert st["step"][k] == ref["step"][k] == K
            assert st["count"][k] == 0
        assert all(st["updated"])
    print(f"{name}: largest relative error of m over all tensors and orderings {worst:.2e}")
    assert not any(runs["ff"]["pending"])   # Alg. 2: every layer pending before the flush
    # The orderings only move the same updates in time: identical bits on the GPU
    # wherever they run the same contractions (forward-fusion's forward shares the
    # plain forward's tiling while the batch is <= 64 rows).
    for o in (("ff", "bf") if cfg["batch"] <= 64 else ("bf",)):
        np.testing.assert_array_equal(runs[o]["losses"], runs["eager"]["losses"])
        for k in ref["params"]:
            np.testing.assert_array_equal(runs[o]["params"][k], runs["eager"]["params"][k])
            np.testing.assert_array_equal(runs[o]["m"][k], runs["eager"]["m"][k])
            np.testing.assert_array_equal(runs[o]["v"][k], runs["eager"]["v"][k])


def test_vgg_pool_argmax(gpu):
    """Max-pool window choices of the first forward are the oracle's, bit for bit."""
    import torch
    from paper_2104_00237_amd.trainer import Trainer
    cfg = reduced_config("vgg11")
    ref = oracle.run(cfg, "eager", steps=1)
    tr = Trainer(cfg, make_params(cfg), gpu)
    x, y = make_batch(cfg, 1)
    tr.step(torch.as_tensor(x).to(gpu), torch.as_tensor(y).to(gpu), "eager")
    got = tr.argmax()
    want = [ref["argmax"][k] for k in sorted(ref["argmax"])]
    assert len(got) == len(want) == len(cfg["pool_after"])
    for (i, g), w in zip(sorted(got.items()), want):
        np.testing.assert_array_equal(g, w, err_msg=f"pool after layer {i + 1}")


WINDOWS = [  # full-size workloads: one-step windows starting from the oracle's own state
    ("mlp8x1024", (0, 1, 9, 19)),
    ("linear4x8192", (0, 1, 5, 9)),
]


def _mismatch(st, loss, cand_loss, cand, cfg, start, teach):
    """None if a GPU state equals one oracle candidate within the parity rules,
    else the first violated rule."""
    try:
        assert rel(loss, [cand_loss]) <= TOL, f"loss {loss} vs {cand_loss}"
        for k in cand["params"]:
            r = rel(st["m"][k], cand["m"][k])
            assert r <= TOL, f"m {k}: rel {r:.2e}"
            r = rel(st["v"][k], cand["v"][k])
            assert r <= TOL, f"v {k}: rel {r:.2e}"
            und = undetermined(st["m"][k], cand["m"][k], start, k, cfg["opt"], TOL) \
                if k in teach else None
            check_param(st["params"][k], cand["params"][k], cfg["opt"], 1, TOL,
                        cand["min_sqrt_vhat"].get(k), what=k, exclude=und, covered=k in teach)
            check_update(st["params"][k], _f32(start["params"][k]), cand["params"][k],
                         start["params"][k], cfg["opt"], TOL, cand["min_sqrt_vhat"].get(k),
                         what=f"update {k}", undetermined=und, teacher=teach.get(k))
        return None
    except AssertionError as e:
        return str(e)


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("name,starts", WINDOWS)
def test_windowed_parity_full_size(gpu, progress, name, starts):
    """Full-size workloads, whose K-step trajectory is chaotic in float32 (Adam's
    first steps move eps-dominated elements by O(lr), which shifts later ReLU
    decisions).  The GPU restarts from the oracle's state after step s (rounded to
    fp32) and computes step s+1; forward-fusion restarts one update earlier,
    holding the oracle's gradient of step s as its pending update, so its fused
    forward applies update s and its flush applies update s+1.

    A backward ReLU decision on a pre-activation within float32 rounding of 0 can
    go either way, so the oracle enumerates the step's outcomes over its ambiguous
    decisions (fewest flips first) and each ordering must equal one of them under
    the parity rules; which one is reported.  Besides the values, the update
    itself is compared (check_update): each element's move against the oracle's,
    and against the update rule applied to the GPU's own gradient."""
    import torch
    from paper_2104_00237_amd.trainer import Trainer
    cfg = get_config(name)
    last = max(starts) + 1
    want = set(starts) | {s - 1 for s in starts if s > 0}
    progress(f"{name}: oracle, {last} steps")
    ref = oracle.run(cfg, "eager", steps=last, snapshots=want,
                     on_step=lambda t: progress(f"{name}: oracle step {t} done"))
    for s in starts:
        progress(f"{name}: window {s} -> {s + 1}")
        results = {}
        for o in ("eager", "ff", "bf"):
            # built on the state it loads: no random initial values to draw
            a = ref["snapshots"][s - 1 if o == "ff" and s > 0 else s]
            tr = Trainer(cfg, a["params"], gpu)
            if o == "ff" and s > 0:
                tr.load_state(a["params"], a["m"], a["v"], a["step"],
                              pending=ref["snapshots"][s]["grad"])
            else:
                tr.load_state(a["params"], a["m"], a["v"], a["step"])
            x, y = make_batch(cfg, s + 1)
            tr.step(torch.as_tensor(x).to(gpu), torch.as_tensor(y).to(gpu), o)
            loss = tr.loss_history()
            if o == "ff":
                tr.flush()
            st = tr.state()
            assert all(v == s + 1 for v in st["step"].values())
            results[o] = (st, loss, teachers(st, ref["snapshots"][s], cfg["opt"]))
            del tr
            torch.cuda.empty_cache()
        np.testing.assert_array_equal(results["bf"][0]["params"]["fc1.weight"],
                                      results["eager"][0]["params"]["fc1.weight"])
        progress(f"{name}: window {s} -> {s + 1}: the three GPU orderings done")
        matched = {}
        why = {}
        with ThreadPoolExecutor(max_workers=len(results)) as pool:
            for flips, cand_loss, cand in oracle.candidate_steps(cfg, ref["snapshots"][s], s + 1):
                # One step from the oracle's own state: the sensitivity of this step's
                # update is set by this outcome's sqrt(v_hat) alone (cand["min_sqrt_vhat"]).
                # The orderings' checks are independent: one thread each (numpy
                # leaves the interpreter lock in its element-wise loops).
                jobs = {o: pool.submit(_mismatch, st, loss, cand_loss, cand, cfg,
                                       ref["snapshots"][s], teach)
                        for o, (st, loss, teach) in results.items() if o not in matched}
                for o, job in jobs.items():
                    msg = job.result()
                    if msg is None:
                        matched[o] = flips
                    else:
                        why.setdefault(o, []).append((len(flips), msg))
                if len(matched) == len(results):
                    break
        progress(f"{name} step {s + 1}: matched candidates "
                 f"{ {o: len(f) for o, f in matched.items()} }")
        print(f"{name} step {s + 1}: matched candidates", {o: len(f) for o, f in matched.items()},
              flush=True)
        for o in set(results) - set(matched):
            for n, msg in why[o][:12]:
                print(f"  {o}: candidate with {n} flips rejected: {msg}")
        assert set(matched) == set(results), f"step {s + 1}: no oracle outcome for " \
            f"{sorted(set(results) - set(matched))}"
        del results
    del ref


MBV2_DECISION_C = 32.0


def test_mbv2_windows_and_orderings(gpu):
    """The MobileNetV2-like network (reduced: every block kind, stride 2,
    residuals).  Its float32 trajectory is chaotic under Adam (a first step of
    +-lr on elements whose gradient sign is within rounding shifts later
    forwards), so each step is checked as a one-step window from the oracle's
    state, values and updates under the parity rules, for every ordering,
    against the oracle's outcomes over the step's ambiguous ReLU decisions
    (pre-activations within float32 rounding of 0 after a linear, depthwise or
    convolution layer); and the three orderings, run free for K steps, are
    bit-identical on the GPU."""
    import torch
    from paper_2104_00237_amd.trainer import Trainer
    cfg = reduced_config("mbv2")
    K = cfg["steps"]
    ref = oracle.run(cfg, "eager", steps=K, snapshots=set(range(K + 1)))
    for s in range(K):
        results = {}
        for o in ("eager", "ff", "bf"):
            # built on the state it loads: no random initial values to draw
            a = ref["snapshots"][s - 1 if o == "ff" and s > 0 else s]
            tr = Trainer(cfg, a["params"], gpu)
            if o == "ff" and s > 0:
                tr.load_state(a["params"], a["m"], a["v"], a["step"],
                              pending=ref["snapshots"][s]["grad"])
            else:
                tr.load_state(a["params"], a["m"], a["v"], a["step"])
            x, y = make_batch(cfg, s + 1)
            tr.step(torch.as_tensor(x).to(gpu), torch.as_tensor(y).to(gpu), o)
            loss = tr.loss_history()
            if o == "ff":
                tr.flush()
            st = tr.state()
            assert all(v == s + 1 for v in st["step"].values())
            results[o] = (st, loss, teachers(st, ref["snapshots"][s], cfg["opt"]))
        matched, why = {}, {}
        # c = 32: seventeen blocks deep, every forward activation carries a few
        # ulps of its tensor's largest value into the next layer (2-4 measured),
        # more than one ulp of a small element's own rounding scale
        for flips, cand_loss, cand in oracle.candidate_steps(cfg, ref["snapshots"][s], s + 1,
                                                              c=MBV2_DECISION_C):
            for o, (st, loss, teach) in results.items():
                if o in matched:
                    continue
                msg = _mismatch(st, loss, cand_loss, cand, cfg, ref["snapshots"][s], teach)
                if msg is None:
                    matched[o] = flips
                else:
                    why.setdefault(o, []).append((len(flips), msg))
            if len(matched) == len(results):
                break
        print(f"mbv2 step {s + 1}: matched candidates", {o: len(f) for o, f in matched.items()},
              flush=True)
        for o in set(results) - set(matched):
            for n, msg in why[o][:8]:
                print(f"  {o}: candidate with {n} flips rejected: {msg}")
        assert set(matched) == set(results), f"step {s + 1}: no oracle outcome for " \
            f"{sorted(set(results) - set(matched))}"
    runs = {o: _gpu_run(torch, cfg, o, K, gpu) for o in ("eager", "ff", "bf")}
    for o in ("ff", "bf"):
        np.testing.assert_array_equal(runs[o]["losses"], runs["eager"]["losses"])
        for k in ref["params"]:
            np.testing.assert_array_equal(runs[o]["params"][k], runs["eager"]["params"][k])
            np.testing.assert_array_equal(runs[o]["m"][k], runs["eager"]["m"][k])
            np.testing.assert_array_equal(runs[o]["v"][k], runs["eager"]["v"][k])
        assert all(v == K for v in runs[o]["step"].values())


@pytest.mark.timeout(400)
def test_vgg_full_size_first_step(gpu):
    """VGG-11 at batch 128, 32x32: the first step under each ordering against the
    oracle's first step (the full learning rate diverges later, so the check is
    one step from the seeded initial state).  The three orderings are bit for bit
    equal on the GPU.  At this size float32 rounding flips a few backward ReLU
    and max-pool decisions, so the oracle's decision search settles the nodes
    from the output down: each node's parameters and momentum must equal the
    oracle's outcome for some set of at most two of its most ambiguous open
    decisions, within the tolerance."""
    import torch
    from paper_2104_00237_amd.trainer import Trainer
    cfg = get_config("vgg11")
    init = make_params(cfg)
    x, y = make_batch(cfg, 1)
    out = {}
    for o in ("eager", "ff", "bf"):
        tr = Trainer(cfg, init, gpu)
        tr.step(torch.as_tensor(x).to(gpu), torch.as_tensor(y).to(gpu), o)
        loss = tr.loss_history()
        if o == "ff":
            tr.flush()
        out[o] = (tr.state(), loss)
        del tr
        torch.cuda.empty_cache()
    st, loss = out["eager"]
    for o in ("ff", "bf"):
        np.testing.assert_array_equal(out[o][1], loss)
        for k in st["params"]:
            np.testing.assert_array_equal(out[o][0]["params"][k], st["params"][k])
            np.testing.assert_array_equal(out[o][0]["m"][k], st["m"][k])
    zero = {k: np.zeros(np.shape(v)) for k, v in init.items()}
    state = dict(params=init, m=zero, v=dict(zero), step={k: 0 for k in init})
    flips = _vgg_search(get_config("vgg11"), state, 1, st, loss, "eager")
    print("vgg11 step 1: flipped decisions per node", flips)


def _tblock_orderings(torch, gpu, cfg, start, prev=None):
    """One step of tblock12 under each ordering from `start` (a state dict);
    forward-fusion starts from `prev` with start's gradient pending when given."""
    from paper_2104_00237_amd.trainer import Trainer
    t = int(next(iter(start["step"].values()))) + 1
    x, y = make_batch(cfg, t)
    out = {}
    for o in ("eager", "ff", "bf"):
        tr = Trainer(cfg, (prev if o == "ff" and prev is not None else start)["params"], gpu)
        if o == "ff" and prev is not None:
            tr.load_state(prev["params"], prev["m"], prev["v"], prev["step"], pending=start["grad"])
        else:
            tr.load_state(start["params"], start["m"], start["v"], start["step"])
        tr.step(torch.as_tensor(x).to(gpu), torch.as_tensor(y).to(gpu), o)
        loss = tr.loss_history()
        if o == "ff":
            tr.flush()
        out[o] = (tr.state(), loss)
        del tr
        torch.cuda.empty_cache()
    return out


def _tblock_check(cfg, out, start, ref, losses, say=print):
    """bf16 parity of one AdamW step: loss, m and v within 2e-2 (max-norm
    relative), the values within 2e-2, and the update element by element
    (check_update) against the oracle and against AdamW applied to the GPU's own
    gradient.  On the first step the elements whose oracle gradient is within
    twice the measured gradient error of zero are left to the second rule."""
    hyper = cfg["opt"]

    def one(o, st, loss):
        assert rel(loss, losses) <= TOL_BF16, (o, loss, losses)
        worst_m, worst_u, und = 0.0, 0.0, []
        teach = teachers(st, start, hyper)
        for k in ref["params"]:
            vh = np.sqrt(ref["v"][k] / (1.0 - hyper["beta2"] ** ref["step"][k]))
            vh = np.where(vh > 0.0, vh, np.inf)
            u = undetermined(st["m"][k], ref["m"][k], start, k, hyper, TOL_BF16)
            check_param(st["params"][k], ref["params"][k], hyper, 1, TOL_BF16, vh, what=f"{o} {k}",
                        exclude=u, covered=True)
            rm = rel(st["m"][k], ref["m"][k])
            assert rm <= TOL_BF16, (o, k, rm)
            assert rel(st["v"][k], ref["v"][k]) <= TOL_BF16, (o, k)
            assert st["step"][k] == ref["step"][k]
            r, n = check_update(st["params"][k], _f32(start["params"][k]), ref["params"][k],
                                start["params"][k], hyper, TOL_BF16, vh, what=f"{o} update {k}",
                                undetermined=u, teacher=teach[k])
            und.append(n / ref["params"][k].size)
            worst_m, worst_u = max(worst_m, rm), max(worst_u, r)
        return (f"tblock12 {o} step {ref['step'][k]}: loss {loss[0]:.6f} (oracle {losses[0]:.6f}), "
                f"largest relative error of m {worst_m:.2e}, of the update {worst_u:.2e}; "
                f"elements left to the own-gradient rule: median {np.median(und):.2%}, "
                f"max {np.max(und):.2%} of a tensor")

    # The orderings' checks are independent: one thread each; results (and the
    # first failed assertion) are taken in ordering order.
    with ThreadPoolExecutor(max_workers=len(out)) as pool:
        jobs = [pool.submit(one, o, st, loss) for o, (st, loss) in out.items()]
        for job in jobs:
            say(job.result())
    for k in ref["params"]:
        np.testing.assert_array_equal(out["bf"][0]["params"][k], out["eager"][0]["params"][k])
        np.testing.assert_array_equal(out["bf"][0]["v"][k], out["eager"][0]["v"][k])


@pytest.mark.timeout(600)
def test_tblock_full_size_first_step(gpu, progress):
    """The 12-block bf16 Transformer stack at 4096 tokens, hidden 1024, FFN 4096:
    the first AdamW step under each ordering against the oracle's first step,
    and backward-fusion bit for bit equal to eager."""
    import torch
    cfg = get_config("tblock12")
    progress("tblock12: oracle step 1")
    ref = oracle.run(cfg, "eager", steps=1, snapshots={0})
    start = ref["snapshots"][0]
    progress("tblock12: step 1 on the GPU, three orderings")
    out = _tblock_orderings(torch, gpu, cfg, start)
    _tblock_check(cfg, out, start, ref, ref["losses"], say=progress)


@pytest.mark.timeout(1200)
def test_tblock_full_size_later_step(gpu, progress):
    """tblock12 at full size, one-step window at a later AdamW step: every
    ordering restarts from the oracle's state after step 5 (forward-fusion from
    step 4 with step 5's gradient pending) and takes step 6, where the moments
    carry five steps of history."""
    import torch
    cfg = get_config("tblock12")
    s = 5
    progress(f"tblock12: oracle, {s + 1} steps")
    ref = oracle.run(cfg, "eager", steps=s + 1, snapshots={s - 1, s},
                     on_step=lambda t: progress(f"tblock12: oracle step {t} done"))
    progress(f"tblock12: step {s + 1} on the GPU, three orderings")
    out = _tblock_orderings(torch, gpu, cfg, ref["snapshots"][s], prev=ref["snapshots"][s - 1])
    _tblock_check(cfg, out, ref["snapshots"][s], ref, ref["losses"][s:], say=progress)


def _vgg_search(cfg, state, t, st, loss, what):
    """Settle the oracle's decision search against one GPU state; returns flips per node."""
    search = oracle.DecisionSearch(cfg, state, t)
    assert rel(loss, [search.loss]) <= TOL, (what, loss, search.loss)
    flips = {}
    while not search.done:
        node, names = search.current()
        chosen, why = None, []
        for subset, upd in search.candidates(max_flips=2):
            errs = {k: (rel(st["params"][k], upd[k][0]), rel(st["m"][k], upd[k][1]))
                    for k in names}
            if all(a <= TOL and b <= TOL for a, b in errs.values()):
                chosen = subset
                break
            why.append((len(subset), errs))
        assert chosen is not None, f"{what} node {node} {names}: no oracle outcome; tried {why[:4]}"
        flips[names[0]] = len(chosen)
        search.accept(chosen)
    ref = search.finish()
    for k in ref["params"]:
        assert st["step"][k] == ref["step"][k] == t
        assert st["count"][k] == 0
    return flips


@pytest.mark.timeout(900)
def test_vgg_full_size_second_step(gpu):
    """VGG-11 at batch 128, one-step window at step 2: eager and backward-fusion
    restart from the oracle's state after step 1 (momentum buffers filled),
    forward-fusion from the initial state with step 1's gradient pending; each
    is settled against the oracle's decision search from that state."""
    import torch
    from paper_2104_00237_amd.trainer import Trainer
    cfg = get_config("vgg11")
    print("vgg11: oracle step 1", flush=True)
    ref = oracle.run(cfg, "eager", steps=1, snapshots={0, 1})
    s0, s1 = ref["snapshots"][0], ref["snapshots"][1]
    x, y = make_batch(cfg, 2)
    out = {}
    for o in ("eager", "ff", "bf"):
        tr = Trainer(cfg, (s0 if o == "ff" else s1)["params"], gpu)
        if o == "ff":
            tr.load_state(s0["params"], s0["m"], s0["v"], s0["step"], pending=s1["grad"])
        else:
            tr.load_state(s1["params"], s1["m"], s1["v"], s1["step"])
        tr.step(torch.as_tensor(x).to(gpu), torch.as_tensor(y).to(gpu), o)
        loss = tr.loss_history()
        if o == "ff":
            tr.flush()
        out[o] = (tr.state(), loss)
        del tr
        torch.cuda.empty_cache()
    st, loss = out["eager"]
    np.testing.assert_array_equal(out["bf"][1], loss)
    for k in st["params"]:
        np.testing.assert_array_equal(out["bf"][0]["params"][k], st["params"][k])
        np.testing.assert_array_equal(out["bf"][0]["m"][k], st["m"][k])
    for o in ("eager", "ff"):
        flips = _vgg_search(cfg, s1, 2, out[o][0], out[o][1], o)
        print(f"vgg11 step 2 {o}: flipped decisions per node", flips, flush=True)


# Adagrad's and RMSprop's first step is g / (|g| sqrt(c) + eps), whose derivative
# in g is up to 1/eps: eps = 1e-4 keeps float32 gradient rounding (~1e-8 here)
# far inside the tolerance (with PyTorch's 1e-10 / 1e-8 an element with |g| near
# eps could move by a sizable fraction of a step in any float32 run).
FIG7_HYPERS = {
    "adagrad": dict(kind="adagrad", lr=0.01, eps=1e-4, weight_decay=1e-4),
    "rmsprop": dict(kind="rmsprop", lr=1e-3, alpha=0.99, eps=1e-4, weight_decay=1e-4, momentum=0.9),
    "rmsprop_nomom": dict(kind="rmsprop", lr=1e-3, alpha=0.99, eps=1e-4, weight_decay=1e-4),
    "adadelta": dict(kind="adadelta", lr=1.0, rho=0.9, eps=1e-6, weight_decay=1e-4),
}


@pytest.mark.parametrize("opt", sorted(FIG7_HYPERS))
def test_fig7_optimizer_training(gpu, opt):
    """The 3-layer MLP trained with each of Fig. 7's other optimizers under the three
    orderings: every ordering against the oracle's eager run, and bit for bit
    against the GPU's eager run (the update is the same per-element arithmetic)."""
    import torch
    cfg = dict(get_config("mlp3"), opt=FIG7_HYPERS[opt])
    K = cfg["steps"]
    ref = oracle.run(cfg, "eager", steps=K)
    runs = {o: _gpu_run(torch, cfg, o, K, gpu) for o in ("eager", "ff", "bf")}
    for o, st in runs.items():
        assert rel(st["losses"], ref["losses"]) <= TOL, (o, st["losses"], ref["losses"])
        assert abs(st["eval_loss"] - ref["eval_loss"]) <= TOL * abs(ref["eval_loss"])
        for k in ref["params"]:
            check_param(st["params"][k], ref["params"][k], cfg["opt"], K, TOL, None,
                        what=f"{o} {k}")
            assert rel(st["m"][k], ref["m"][k]) <= TOL, (o, k)
            assert rel(st["v"][k], ref["v"][k]) <= TOL, (o, k)
            assert st["step"][k] == ref["step"][k] == K
    for o in ("ff", "bf"):
        np.testing.assert_array_equal(runs[o]["losses"], runs["eager"]["losses"])
        for k in ref["params"]:
            np.testing.assert_array_equal(runs[o]["params"][k], runs["eager"]["params"][k])
            np.testing.assert_array_equal(runs[o]["v"][k], runs["eager"]["v"][k])


def _gpu_run_merge(torch, cfg, ordering, steps, dev, merge):
    from paper_2104_00237_amd.trainer import Trainer
    tr = Trainer(cfg, make_params(cfg), dev, merge_dgrad=merge)
    for t in range(1, steps + 1):
        x, y = make_batch(cfg, t)
        tr.step(torch.as_tensor(x).to(dev), torch.as_tensor(y).to(dev), ordering)
    losses = tr.loss_history()
    if ordering == "ff":
        tr.flush()
    st = tr.state()
    st.update(losses=losses)
    return st


@pytest.mark.parametrize("opt", ["sgd", "adam"])
def test_shared_parameter_training(gpu, opt):
    """Layer 3 applies layer 2's weight and bias again.  Eager sums both uses'
    gradients before the optimizer; forward-fusion updates the operator once, at
    its first forward (Alg. 2's `updated` flag); backward-fusion writes the later
    use's gradient to a buffer and the last backward use's fused update adds it
    (Alg. 3's `count`), also with the merged data gradient.  Every ordering against
    the oracle's eager run; the unmerged orderings bit for bit against each other."""
    import torch
    cfg = get_config("mlp4tied")
    if opt == "adam":
        cfg["opt"] = dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                          weight_decay=0.0)
    K = cfg["steps"]
    ref = oracle.run(cfg, "eager", steps=K)
    runs = {o: _gpu_run_merge(torch, cfg, o, K, gpu, False) for o in ("eager", "ff", "bf")}
    runs["bf_merged"] = _gpu_run_merge(torch, cfg, "bf", K, gpu, True)
    for o, st in runs.items():
        assert rel(st["losses"], ref["losses"]) <= TOL, (o, st["losses"], ref["losses"])
        assert sorted(st["params"]) == sorted(ref["params"])
        for k in ref["params"]:
            check_param(st["params"][k], ref["params"][k], cfg["opt"], K, TOL,
                        ref["min_sqrt_vhat"].get(k), what=f"{o} {k}")
            assert rel(st["m"][k], ref["m"][k]) <= TOL, (o, k)
            assert st["step"][k] == ref["step"][k] == K, (o, k)
            assert st["count"][k] == 0
    for o in ("ff", "bf"):
        np.testing.assert_array_equal(runs[o]["losses"], runs["eager"]["losses"])
        for k in ref["params"]:
            np.testing.assert_array_equal(runs[o]["params"][k], runs["eager"]["params"][k])


def test_vgg_conv_prologue_forward_fusion(gpu):
    """Forward-fusion with each convolution's pending update applied in its
    forward's filter-tile loads (two buffer sets alternating) on the reduced
    VGG: against the oracle, and bit for bit against the default forward-fusion,
    which carries the same updates in the previous launch."""
    import torch
    cfg = _cfg("vgg11", "reduced")
    K = cfg["steps"]
    ref = oracle.run(cfg, "eager", steps=K)
    runs = {p: _gpu_run_prologue(torch, cfg, K, gpu, p) for p in (False, True)}
    st = runs[True]
    assert rel(st["losses"], ref["losses"]) <= TOL
    for k in ref["params"]:
        check_param(st["params"][k], ref["params"][k], cfg["opt"], K, TOL, None, what=k)
        assert rel(st["m"][k], ref["m"][k]) <= TOL, k
        assert st["step"][k] == K
        np.testing.assert_array_equal(st["params"][k], runs[False]["params"][k])
        np.testing.assert_array_equal(st["m"][k], runs[False]["m"][k])
    np.testing.assert_array_equal(st["losses"], runs[False]["losses"])


def _gpu_run_prologue(torch, cfg, steps, dev, prologue):
    from paper_2104_00237_amd.trainer import Trainer
    tr = Trainer(cfg, make_params(cfg), dev, conv_prologue=prologue)
    assert any(op.kind == "conv" and op.prologue_ff for op in tr.ops) == prologue
    for t in range(1, steps + 1):
        x, y = make_batch(cfg, t)
        tr.step(torch.as_tensor(x).to(dev), torch.as_tensor(y).to(dev), "ff")
    losses = tr.loss_history()
    tr.flush()
    st = tr.state()
    st.update(losses=losses)
    return st


def test_linear_prologue_forward_fusion(gpu):
    """Forward-fusion with every linear layer's pending update applied in its own
    forward's W-tile loads: the reduced 8-layer MLP (72 rows, more than one row
    tile) writes each update to the second buffer set, which becomes current;
    K steps against the oracle's eager run."""
    import torch
    from paper_2104_00237_amd.trainer import Trainer
    cfg = reduced_config("mlp8x1024")
    assert cfg["batch"] > 64
    K = cfg["steps"]
    ref = oracle.run(cfg, "eager", steps=K)
    tr = Trainer(cfg, make_params(cfg), gpu, linear_prologue=True)
    assert all(op.two_sets() for op in tr.ops if op.kind == "linear")
    for t in range(1, K + 1):
        x, y = make_batch(cfg, t)
        tr.step(torch.as_tensor(x).to(gpu), torch.as_tensor(y).to(gpu), "ff")
    losses = tr.loss_history()
    tr.flush()
    st = tr.state()
    assert rel(losses, ref["losses"]) <= TOL
    for k in ref["params"]:
        check_param(st["params"][k], ref["params"][k], cfg["opt"], K, TOL,
                    ref["min_sqrt_vhat"].get(k), what=k)
        assert rel(st["m"][k], ref["m"][k]) <= TOL, k
        assert rel(st["v"][k], ref["v"][k]) <= TOL, k
        assert st["step"][k] == K
