"""A residual connection added in the forward's epilogue (of_linear_fwd_res),
through the C ABI: Y = act(X W^T + b) + R must equal of_linear_fwd followed by
of_add bit for bit (the sum is rounded once either way), for fp32 and bf16
operands, bf16 storage of X and Y, in place (R is Y), with a carried update
in the same launch, and with split reductions.  The forward alone is held to
the oracle by the other kernel tests."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env(gpu):
    import torch
    from paper_2104_00237_amd import _lib as L
    L.load()
    return torch, L, gpu


def _ws(torch, dev, nbytes):
    return torch.empty(max(16, (nbytes + 15) // 16 * 4), dtype=torch.float32, device=dev)


def _bits(t):
    import torch
    t = t.detach().cpu().contiguous()
    return (t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)).numpy()


# (M, N, K, ldy): ragged tails and scalar epilogues (N or ldy not a multiple of 4),
# a strided Y, split reductions (K = 4096), the 64-row and wide tiles
SHAPES = [(37, 70, 53, 70), (64, 128, 96, 132), (130, 96, 44, 98), (64, 1024, 4096, 1024),
          (4096, 1024, 4096, 1024), (4096, 1024, 1024, 1024), (2000, 2000, 2056, 2000)]
KINDS = [("f32", 0), ("bf16", 0), ("bf16", 1), ("bf16", 3)]   # dtype, io flags
# every bf16 kind on every shape; fp32 on the shapes up to 1024 rows (its tiles and
# split reductions are all reached there)
CASES = [(shape, kind) for shape in SHAPES for kind in KINDS
         if kind[0] == "bf16" or shape[0] <= 1024]


@pytest.mark.parametrize("M,N,K,ldy,kind,io", [(*sh, *k) for sh, k in CASES])
def test_forward_residual_equals_forward_then_add(env, M, N, K, ldy, kind, io):
    torch, L, dev = env
    g = torch.Generator().manual_seed(M * 7 + N + K)
    x = torch.randn((M, K), generator=g).to(dev)
    w = (torch.randn((N, K), generator=g) / K ** 0.5).to(dev)
    b = (0.1 * torch.randn((N,), generator=g)).to(dev)
    r = torch.randn((M, ldy), generator=g).to(dev)
    bf16 = kind == "bf16"
    wb = w.to(torch.bfloat16) if bf16 else None
    xs = x.to(torch.bfloat16) if io & L.OF_IO_X_BF16 else x
    ydt = torch.bfloat16 if io & L.OF_IO_Y_BF16 else torch.float32
    dt = L.OF_BF16 if bf16 else L.OF_F32
    d = L.OfLinearDesc(M, N, K, 0, ldy, dt, L.OF_ACT_RELU, 1, io)
    d0 = L.OfLinearDesc(M, N, K, 0, ldy, dt, L.OF_ACT_RELU, 1, io & L.OF_IO_X_BF16)
    Wp = L.OfParam(w.data_ptr(), None, None, wb.data_ptr() if bf16 else None, w.numel())
    ws = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_FWD))

    # reference: the fp32 forward, then the residual add
    Z0 = torch.full((M, ldy), float("nan"), device=dev)
    Y0 = torch.full((M, ldy), float("nan"), device=dev)
    L.of_linear_fwd(d0, xs.data_ptr(), Wp, b.data_ptr(), Z0.data_ptr(), Y0.data_ptr(),
                    ws.data_ptr(), ws.numel() * 4, 0)
    S0 = torch.full((M, ldy), float("nan"), device=dev)
    if ldy == N:
        L.of_add(Y0.data_ptr(), r.data_ptr(), M * N, S0.data_ptr(), 0)
    else:   # row by row: the padding columns of a strided Y stay untouched
        for i in range(M):
            L.of_add(Y0[i].data_ptr(), r[i].data_ptr(), N, S0[i].data_ptr(), 0)
    torch.cuda.synchronize()
    want = S0[:, :N].cpu()
    if io & L.OF_IO_Y_BF16:
        want = want.to(torch.bfloat16)

    Z = torch.full((M, ldy), float("nan"), device=dev)
    Y = torch.full((M, ldy), float("nan"), device=dev, dtype=ydt)
    L.of_linear_fwd_res(d, xs.data_ptr(), Wp, b.data_ptr(), r.data_ptr(), Z.data_ptr(),
                        Y.data_ptr(), None, ws.data_ptr(), ws.numel() * 4, 0)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(Y[:, :N]), _bits(want))
    assert np.array_equal(_bits(Z[:, :N]), _bits(Z0[:, :N]))
    if ldy > N:   # the padding columns are not written
        assert bool(torch.isnan(Y[:, N:].float()).all())

    if not io & L.OF_IO_Y_BF16:
        # in place: R is Y
        Yi = r.clone()
        L.of_linear_fwd_res(d, xs.data_ptr(), Wp, b.data_ptr(), Yi.data_ptr(), None,
                            Yi.data_ptr(), None, ws.data_ptr(), ws.numel() * 4, 0)
        torch.cuda.synchronize()
        assert np.array_equal(_bits(Yi[:, :N]), _bits(want))


def test_forward_residual_with_carried_update(env):
    """A later operator's pending update carried by the residual forward's launch:
    Y and the carried tensor equal the plain carried forward's, then of_add."""
    torch, L, dev = env
    M, N, K = 512, 256, 1024
    g = torch.Generator().manual_seed(3)
    x = torch.randn((M, K), generator=g).to(dev)
    w = (torch.randn((N, K), generator=g) / K ** 0.5).to(dev)
    b = (0.1 * torch.randn((N,), generator=g)).to(dev)
    r = torch.randn((M, N), generator=g).to(dev)
    wb = w.to(torch.bfloat16)
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_BF16, L.OF_ACT_NONE, 1, 0)
    Wp = L.OfParam(w.data_ptr(), None, None, wb.data_ptr(), w.numel())
    ws = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_FWD))
    n = 300_001
    hyper = dict(kind="adamw", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)
    t0 = [(torch.randn((n,), generator=g) * s).to(dev) for s in (1.0, 1e-3, 1e-3)]
    t0[2] = t0[2].abs()
    gr = (torch.randn((n,), generator=g) * 1e-2).to(dev)

    def run(fused_add):
        cw, cm, cv = (t.clone() for t in t0)
        P = L.OfParam(cw.data_ptr(), cm.data_ptr(), cv.data_ptr(), None, n)
        c = L.make_carry(L.make_opt(hyper, 2), [(P, gr.data_ptr(), 1)])
        Y = torch.full((M, N), float("nan"), device=dev)
        if fused_add:
            L.of_linear_fwd_res(d, x.data_ptr(), Wp, b.data_ptr(), r.data_ptr(), None,
                                Y.data_ptr(), c, ws.data_ptr(), ws.numel() * 4, 0)
        else:
            L.of_linear_fwd_carry(d, x.data_ptr(), Wp, b.data_ptr(), None, Y.data_ptr(), c,
                                  ws.data_ptr(), ws.numel() * 4, 0)
            L.of_add(Y.data_ptr(), r.data_ptr(), M * N, Y.data_ptr(), 0)
        torch.cuda.synchronize()
        return [Y, cw, cm, cv]

    for a, c in zip(run(True), run(False)):
        assert np.array_equal(_bits(a), _bits(c))


# (M, N, K, ldx): ragged tails and scalar epilogues, a strided dX, split reductions
DG_SHAPES = [(37, 70, 53, 53), (130, 96, 44, 49), (64, 4096, 1024, 1024), (401, 96, 576, 576),
             (2048, 2048, 1024, 1024)]


@pytest.mark.parametrize("M,N,K,ldx", DG_SHAPES)
@pytest.mark.parametrize("kind", ["f32", "bf16"])
@pytest.mark.parametrize("act", ["none", "relu", "gelu"])
def test_data_gradient_residual_equals_data_gradient_then_add(env, M, N, K, ldx, kind, act):
    """dX = (dZ W) * act'(prev) + R equals of_linear_bwd_data followed by of_add bit
    for bit, in a separate buffer and in place."""
    torch, L, dev = env
    g = torch.Generator().manual_seed(M + 3 * N + K)
    dz = (torch.randn((M, N), generator=g) * 1e-2).to(dev)
    w = (torch.randn((N, K), generator=g) / K ** 0.5).to(dev)
    prev = torch.randn((M, ldx), generator=g).to(dev)
    r = torch.randn((M, ldx), generator=g).to(dev)
    bf16 = kind == "bf16"
    wb = w.to(torch.bfloat16) if bf16 else None
    a = {"none": L.OF_ACT_NONE, "relu": L.OF_ACT_RELU, "gelu": L.OF_ACT_GELU}[act]
    d = L.OfLinearDesc(M, N, K, ldx, 0, L.OF_BF16 if bf16 else L.OF_F32, L.OF_ACT_NONE, 0, 0)
    Wp = L.OfParam(w.data_ptr(), None, None, wb.data_ptr() if bf16 else None, w.numel())
    ws = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_DATA))
    pp = prev.data_ptr() if a != L.OF_ACT_NONE else None

    D0 = torch.full((M, ldx), float("nan"), device=dev)
    L.of_linear_bwd_data(d, dz.data_ptr(), Wp, pp, a, D0.data_ptr(), ws.data_ptr(),
                         ws.numel() * 4, 0)
    S0 = torch.full((M, ldx), float("nan"), device=dev)
    if ldx == K:
        L.of_add(D0.data_ptr(), r.data_ptr(), M * K, S0.data_ptr(), 0)
    else:
        for i in range(M):
            L.of_add(D0[i].data_ptr(), r[i].data_ptr(), K, S0[i].data_ptr(), 0)
    D1 = torch.full((M, ldx), float("nan"), device=dev)
    L.of_linear_bwd_data_res(d, dz.data_ptr(), Wp, pp, a, r.data_ptr(), D1.data_ptr(),
                             ws.data_ptr(), ws.numel() * 4, 0)
    Di = r.clone()
    L.of_linear_bwd_data_res(d, dz.data_ptr(), Wp, pp, a, Di.data_ptr(), Di.data_ptr(),
                             ws.data_ptr(), ws.numel() * 4, 0)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(D1[:, :K]), _bits(S0[:, :K]))
    assert np.array_equal(_bits(Di[:, :K]), _bits(S0[:, :K]))
    if ldx > K:
        assert bool(torch.isnan(D1[:, K:]).all())
