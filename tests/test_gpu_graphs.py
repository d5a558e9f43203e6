"""Captured training steps (HIP graphs) replay exactly what step() computes.

Each replay is checked bit for bit against an uncaptured trainer stepping in
lockstep on the same batches, with eager device work and synchronisations
between the replays.
"""
import numpy as np
import pytest

from workloads import get_config, reduced_config, make_params, make_batch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["mlp3", "mlp8x1024", "mbv2", "tblock12"])
@pytest.mark.parametrize("ordering", ["eager", "ff", "bf"])
def test_graph_replays_match_steps(gpu, name, ordering):
    import torch
    from paper_2104_00237_amd.trainer import Trainer
    cfg = get_config(name) if name == "mlp3" else reduced_config(name)
    x, y = make_batch(cfg, 1)
    X, Y = torch.as_tensor(x).to(gpu), torch.as_tensor(y).to(gpu)
    ref = Trainer(cfg, make_params(cfg), gpu)
    cap = Trainer(cfg, make_params(cfg), gpu)
    ref.step(X, Y, ordering)
    cap.step(X, Y, ordering)
    replay = cap.capture(X, Y, ordering)
    for k in range(4):
        ref.step(X, Y, ordering)
        replay()
        # eager work on the device between replays
        junk = torch.randn(1000, device=gpu).sum()
        torch.cuda.synchronize()
        a, b = ref.state(), cap.state()
        for n in a["params"]:
            np.testing.assert_array_equal(b["params"][n], a["params"][n], err_msg=f"replay {k} {n}")
            np.testing.assert_array_equal(b["m"][n], a["m"][n])
            np.testing.assert_array_equal(b["v"][n], a["v"][n])
            # forward-fusion holds the latest update back until the next forward
            assert b["step"][n] == a["step"][n] == k + (1 if ordering == "ff" else 2)
        assert float(junk) == float(junk)
    if ordering == "ff":
        ref.flush()
        cap.flush()
        a, b = ref.state(), cap.state()
        for n in a["params"]:
            np.testing.assert_array_equal(b["params"][n], a["params"][n])


def test_conv_prologue_then_capture(gpu):
    """A trainer that uses the convolutions' filter-tile prologue (alternating
    buffer sets) and is then captured: the replays and later launched steps carry
    the updates instead, and every step matches a trainer that always carried
    them, bit for bit."""
    import torch
    from paper_2104_00237_amd.trainer import Trainer
    from workloads import reduced_config, make_params, make_batch
    cfg = reduced_config("vgg11")
    batches = [tuple(torch.as_tensor(a).to(gpu) for a in make_batch(cfg, t)) for t in range(1, 5)]
    runs = []
    for prologue in (True, False):
        tr = Trainer(cfg, make_params(cfg), gpu, conv_prologue=prologue)
        tr.step(*batches[0], "ff")
        tr.step(*batches[1], "ff")          # prologue steps (generations swapped)
        g = tr.capture(*batches[2], "ff")
        g()
        tr.step(*batches[3], "ff")          # launched again after the capture
        tr.flush()
        torch.cuda.synchronize()
        runs.append((tr.state(), tr.loss_history()))
    (a, la), (b, lb) = runs
    np.testing.assert_array_equal(la, lb)
    for k in a["params"]:
        np.testing.assert_array_equal(a["params"][k], b["params"][k])
        np.testing.assert_array_equal(a["m"][k], b["m"][k])
