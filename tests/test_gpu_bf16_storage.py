"""bf16 storage of activations that only bf16-operand contractions read
(of_linear_desc.io, of_layernorm_fwd_bf16), through the C ABI.

Storing such a tensor as its bf16 rounding (round to nearest even) gives the
contraction the value it would round the fp32 tensor to while staging it, so
every result must be bit-identical to the fp32-storage path, which the other
bf16 tests hold to the oracle: forward Z, the bf16 Y against the rounding of the
fp32 Y, weight gradients, backward-fusion's updated W, m, v, shadow and bias,
the LayerNorm output against the rounding of the fp32 one, and whole reduced
tblock12 trainings in every ordering.
"""
import numpy as np
import pytest

from workloads import make_batch, make_params, reduced_config

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
    """Bit patterns of a tensor on the host (int16 for bf16, int32 for fp32)."""
    import torch
    t = t.detach().cpu().contiguous()
    return (t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)).numpy()


def _rne(torch, t32):
    """bf16 rounding (to nearest even) of an fp32 tensor, done by torch on the host."""
    return t32.detach().cpu().to(torch.bfloat16)


def _data(torch, dev, M, N, K, ldx, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((M, ldx), generator=g)
    w = torch.randn((N, K), generator=g) / K ** 0.5
    b = torch.randn((N,), generator=g) * 0.1
    dz = torch.randn((M, N), generator=g) * 1e-2
    return [t.to(dev) for t in (x, w, b, dz)]


# (M, N, K, ldx): ragged tails with scalar loads (K or ldx not a multiple of 8),
# vector loads, a strided X (the V third of a QKV output), split reductions of a
# forward (K = 4096) and a weight gradient (M = 4096), the eight-wave 128x256 tiles
SHAPES = [(37, 70, 53, 53), (64, 128, 96, 96), (130, 96, 44, 132), (136, 96, 96, 288),
          (200, 168, 160, 163), (512, 256, 1024, 1024), (4096, 1024, 4096, 4096),
          (4096, 1024, 1024, 3072), (1999, 2001, 2050, 2050), (2000, 2000, 2056, 2056)]


@pytest.mark.parametrize("M,N,K,ldx", SHAPES)
def test_forward_bf16_x_and_y(env, M, N, K, ldx):
    torch, L, dev = env
    x, w, b, _ = _data(torch, dev, M, N, K, ldx, M + N + K)
    wb = w.to(torch.bfloat16)
    xb = x.to(torch.bfloat16)

    def run(io):
        d = L.OfLinearDesc(M, N, K, ldx, 0, L.OF_BF16, L.OF_ACT_GELU, 1, io)
        Wp = L.OfParam(w.data_ptr(), None, None, wb.data_ptr(), w.numel())
        ydt = torch.bfloat16 if io & L.OF_IO_Y_BF16 else torch.float32
        Z = torch.full((M, N), float("nan"), device=dev)
        Y = torch.full((M, N), float("nan"), device=dev, dtype=ydt)
        ws = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_FWD))
        X = xb if io & L.OF_IO_X_BF16 else x
        L.of_linear_fwd(d, X.data_ptr(), Wp, b.data_ptr(), Z.data_ptr(), Y.data_ptr(),
                        ws.data_ptr(), ws.numel() * 4, 0)
        torch.cuda.synchronize()
        return Z, Y

    Z0, Y0 = run(0)
    for io in (L.OF_IO_X_BF16, L.OF_IO_Y_BF16, L.OF_IO_X_BF16 | L.OF_IO_Y_BF16):
        Z, Y = run(io)
        assert np.array_equal(_bits(Z), _bits(Z0)), io
        want = _rne(torch, Y0) if io & L.OF_IO_Y_BF16 else Y0
        assert np.array_equal(_bits(Y), _bits(want)), io


ADAMW = dict(kind="adamw", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)


@pytest.mark.parametrize("M,N,K,ldx", SHAPES)
def test_weight_gradients_bf16_x(env, M, N, K, ldx):
    """Eager weight gradient and backward-fusion (AdamW, with the data gradient)
    reading X as stored bf16 equal the fp32-X calls bit for bit."""
    torch, L, dev = env
    x, w, b, dz = _data(torch, dev, M, N, K, ldx, 7 * M + K)
    xb = x.to(torch.bfloat16)
    zprev = x   # the previous layer's pre-activation for GELU's derivative

    def wgrad(io):
        d = L.OfLinearDesc(M, N, K, ldx, 0, L.OF_BF16, L.OF_ACT_NONE, 1, io)
        DW = torch.full((N, K), float("nan"), device=dev)
        DB = torch.full((N,), float("nan"), device=dev)
        ws = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_WEIGHT))
        X = xb if io else x
        L.of_linear_bwd_weight(d, dz.data_ptr(), X.data_ptr(), DW.data_ptr(), DB.data_ptr(), 0,
                               ws.data_ptr(), ws.numel() * 4, 0)
        torch.cuda.synchronize()
        return DW, DB

    DW0, DB0 = wgrad(0)
    DW1, DB1 = wgrad(L.OF_IO_X_BF16)
    assert np.array_equal(_bits(DW1), _bits(DW0))
    assert np.array_equal(_bits(DB1), _bits(DB0))

    g = torch.Generator().manual_seed(11)
    m0 = (torch.randn((N, K), generator=g) * 1e-3).to(dev)
    v0 = (torch.rand((N, K), generator=g) * 1e-6).to(dev)
    bm0 = (torch.randn((N,), generator=g) * 1e-3).to(dev)
    bv0 = (torch.rand((N,), generator=g) * 1e-6).to(dev)

    def fused(io):
        d = L.OfLinearDesc(M, N, K, ldx, 0, L.OF_BF16, L.OF_ACT_NONE, 1, io)
        W, m, v, sh = w.clone(), m0.clone(), v0.clone(), w.to(torch.bfloat16)
        B, bm, bv = b.clone(), bm0.clone(), bv0.clone()
        DX = torch.full((M, ldx), float("nan"), device=dev)
        wsd = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_DATA))
        wsu = _ws(torch, dev, L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_WEIGHT))
        Wp = L.OfParam(W.data_ptr(), m.data_ptr(), v.data_ptr(), sh.data_ptr(), W.numel())
        Bp = L.OfParam(B.data_ptr(), bm.data_ptr(), bv.data_ptr(), None, N)
        opt = L.make_opt(ADAMW, 3)
        X = xb if io else x
        L.of_linear_bwd_fused(d, dz.data_ptr(), X.data_ptr(), Wp, Bp, None, None, opt,
                              zprev.data_ptr(), L.OF_ACT_GELU, DX.data_ptr(), wsd.data_ptr(),
                              wsd.numel() * 4, wsu.data_ptr(), wsu.numel() * 4, 0, None)
        torch.cuda.synchronize()
        return [W, m, v, sh, B, bm, bv, DX[:, :K]]

    for a0, a1 in zip(fused(0), fused(L.OF_IO_X_BF16)):
        assert np.array_equal(_bits(a1), _bits(a0))


@pytest.mark.parametrize("M,D", [(136, 96), (4096, 1024), (33, 30), (7, 2052), (64, 2048)])
def test_layernorm_bf16_output(env, M, D):
    """Register-resident rows (D a multiple of 4, at most 2048) and the general
    kernel (other D): the bf16 output is the rounding of the fp32 one, mean and
    rstd are identical."""
    torch, L, dev = env
    g = torch.Generator().manual_seed(M * D)
    x = (torch.randn((M, D), generator=g) * 2 + 0.5).to(dev)
    gamma = (1 + 0.1 * torch.randn((D,), generator=g)).to(dev)
    beta = (0.1 * torch.randn((D,), generator=g)).to(dev)

    def run(bf16):
        y = torch.full((M, D), float("nan"), device=dev,
                       dtype=torch.bfloat16 if bf16 else torch.float32)
        mu = torch.full((M,), float("nan"), device=dev)
        rs = torch.full((M,), float("nan"), device=dev)
        fn = L.of_layernorm_fwd_bf16 if bf16 else L.of_layernorm_fwd
        fn(x.data_ptr(), M, D, gamma.data_ptr(), beta.data_ptr(), 1e-5, y.data_ptr(),
           mu.data_ptr(), rs.data_ptr(), 0)
        torch.cuda.synchronize()
        return y, mu, rs

    y0, mu0, rs0 = run(False)
    y1, mu1, rs1 = run(True)
    assert np.array_equal(_bits(y1), _bits(_rne(torch, y0)))
    assert np.array_equal(_bits(mu1), _bits(mu0)) and np.array_equal(_bits(rs1), _bits(rs0))


@pytest.mark.parametrize("ordering", ["eager", "ff", "bf"])
def test_tblock_training_bf16_storage_bit_identical(env, ordering):
    """Reduced tblock12 (2 blocks, 136 tokens, AdamW, 3 steps): the trainer with
    bf16 activation storage (the default) and with fp32 storage end with the
    same parameters, histories and losses, bit for bit."""
    torch, L, dev = env
    from paper_2104_00237_amd.trainer import Trainer
    cfg = reduced_config("tblock12")
    out = []
    for acts in (True, False):
        tr = Trainer(cfg, make_params(cfg), dev, bf16_acts=acts)
        for t in range(1, cfg["steps"] + 1):
            x, y = make_batch(cfg, t)
            tr.step(torch.as_tensor(x).to(dev), torch.as_tensor(y).to(dev), ordering)
        losses = tr.loss_history()
        if ordering == "ff":
            tr.flush()
        st = tr.state()
        st["losses"] = losses
        out.append(st)
    a, b = out
    assert np.array_equal(a["losses"], b["losses"])
    for k in a["params"]:
        for f in ("params", "m", "v"):
            assert np.array_equal(a[f][k].view(np.int32), b[f][k].view(np.int32)), (f, k)
