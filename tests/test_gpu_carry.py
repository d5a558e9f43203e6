"""A forward launch carrying a later operator's update (forward-fusion).

of_linear_fwd_carry / of_conv_fwd_carry must give the forward's output bit for
bit as the plain forward, and leave the carried tensors (w, m, v, bf16 shadow)
bit for bit as the separate update passes do: of_optimizer_step for a vector
gradient, of_elementwise_fused_update for row partials.  The update passes are
themselves checked against the oracle in test_gpu_kernels.py.
"""
import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

HYPERS = {
    "sgd": dict(kind="sgd", lr=0.1, momentum=0.9, weight_decay=5e-4),
    "adam": dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8),
    "adamw": dict(kind="adamw", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01),
}


@pytest.fixture(scope="module")
def env(gpu):
    import torch
    from paper_2104_00237_amd import _lib as L
    L.load()
    return torch, L, gpu


class _T:
    """A carried tensor (two identical copies: one for the carry, one for the
    reference pass) with history, an optional bf16 shadow and its gradient."""

    def __init__(self, torch, L, dev, n, kind, seed, rows=1, shadow=False, offset=0):
        g = torch.Generator(device="cpu").manual_seed(seed)
        w = torch.randn(n, generator=g) * 0.1
        m = torch.randn(n, generator=g) * 0.01
        v = torch.rand(n, generator=g) * 1e-4
        gr = torch.randn(rows * n, generator=g) * 1e-2
        self.copies = []
        for _ in range(2):
            # `offset` elements in front of every array break 16-byte alignment
            W = torch.zeros(n + offset, device=dev); W[offset:] = w.to(dev)
            Mm = torch.zeros(n + offset, device=dev); Mm[offset:] = m.to(dev)
            V = torch.zeros(n + offset, device=dev); V[offset:] = v.to(dev)
            G = torch.zeros(rows * n + offset, device=dev); G[offset:] = gr.to(dev)
            B = (W[offset:].to(torch.bfloat16).view(torch.int16).contiguous() if shadow else None)
            p = L.OfParam(W[offset:].data_ptr(), Mm[offset:].data_ptr(),
                          V[offset:].data_ptr() if kind != "sgd" else None,
                          B.data_ptr() if B is not None else None, n)
            self.copies.append(dict(W=W, M=Mm, V=V, G=G, B=B, p=p, g=G[offset:].data_ptr()))
        self.rows, self.n = rows, n

    def reference_update(self, L, opt):
        c = self.copies[1]
        if self.rows == 1:
            arr = (L.OfParam * 1)(c["p"])
            gp = (ctypes.c_void_p * 1)(c["g"])
            L.of_optimizer_step(1, arr, gp, opt, 0)
        else:
            L.of_elementwise_fused_update(c["p"], c["g"], self.rows, self.n, opt, 0)

    def same(self, torch):
        a, b = self.copies
        for k in ("W", "M", "V", "B"):
            if a[k] is not None:
                assert torch.equal(a[k], b[k]), k


def _carry(L, opt, *ts):
    return L.make_carry(opt, [(t.copies[0]["p"], t.copies[0]["g"], t.rows) for t in ts])


CASES = [  # (M, N, K, dtype): direct tiles, staged tiles, split reduction, bf16,
    # bf16 on eight-wave 128x256 tiles (512-thread workgroups carry the update)
    (256, 1024, 1024, "f32"), (1024, 512, 256, "f32"), (100, 50, 3000, "f32"),
    (72, 168, 200, "f32"), (512, 1024, 1024, "bf16"), (1024, 4096, 2048, "bf16"),
]


@pytest.mark.parametrize("M,N,K,dt", CASES)
@pytest.mark.parametrize("kind", ["adam", "sgd"])
def test_linear_fwd_carry_bits(env, M, N, K, dt, kind):
    torch, L, dev = env
    g = torch.Generator(device="cpu").manual_seed(M + N + K)
    X = torch.randn(M, K, generator=g).to(dev)
    Wt = (torch.randn(N, K, generator=g) * 0.05).to(dev)
    b = torch.randn(N, generator=g).to(dev)
    bf16 = dt == "bf16"
    Wb = Wt.to(torch.bfloat16).view(torch.int16).contiguous() if bf16 else None
    Wp = L.OfParam(Wt.data_ptr(), Wt.data_ptr(), None, Wb.data_ptr() if bf16 else None, N * K)
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_BF16 if bf16 else L.OF_F32, L.OF_ACT_RELU, 1)
    wsb = L.of_linear_workspace_size(d, L.OF_LINEAR_FWD)
    ws = torch.empty(max(16, wsb) // 4 + 4, device=dev)
    Y0 = torch.empty(M, N, device=dev)
    Y1 = torch.empty(M, N, device=dev)
    opt = L.make_opt(HYPERS[kind], 3)
    t1 = _T(torch, L, dev, 1000 * 37, kind, 1, shadow=bf16)      # ragged float4 tail
    t2 = _T(torch, L, dev, 4097, kind, 2, offset=1)               # misaligned: scalar path
    L.of_linear_fwd(d, X.data_ptr(), Wp, b.data_ptr(), None, Y0.data_ptr(), ws.data_ptr(),
                    ws.numel() * 4, 0)
    t1.reference_update(L, opt)
    t2.reference_update(L, opt)
    L.of_linear_fwd_carry(d, X.data_ptr(), Wp, b.data_ptr(), None, Y1.data_ptr(),
                          _carry(L, opt, t1, t2), ws.data_ptr(), ws.numel() * 4, 0)
    torch.cuda.synchronize()
    assert torch.equal(Y0, Y1)
    t1.same(torch)
    t2.same(torch)


@pytest.mark.parametrize("rows", [1, 5, 64])
def test_linear_fwd_carry_rows(env, rows):
    """A LayerNorm-style pair of vectors with row-partial gradients, and the next
    layer's weight and bias with vector gradients (four carried tensors)."""
    torch, L, dev = env
    M, N, K = 256, 1024, 1024
    X = torch.randn(M, K, device=dev)
    Wt = torch.randn(N, K, device=dev) * 0.05
    Wp = L.OfParam(Wt.data_ptr(), Wt.data_ptr(), None, None, N * K)
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 0)
    wsb = L.of_linear_workspace_size(d, L.OF_LINEAR_FWD)
    ws = torch.empty(max(16, wsb) // 4 + 4, device=dev)
    Y0 = torch.empty(M, N, device=dev)
    Y1 = torch.empty(M, N, device=dev)
    opt = L.make_opt(HYPERS["adamw"], 2)
    gam = _T(torch, L, dev, 1024, "adamw", 3, rows=rows)
    bet = _T(torch, L, dev, 1024, "adamw", 4, rows=rows)
    w2 = _T(torch, L, dev, 4096 * 1024, "adamw", 7, shadow=True)
    b2 = _T(torch, L, dev, 4096, "adamw", 8)
    L.of_linear_fwd(d, X.data_ptr(), Wp, None, None, Y0.data_ptr(), ws.data_ptr(),
                    ws.numel() * 4, 0)
    for t in (gam, bet, w2, b2):
        t.reference_update(L, opt)
    L.of_linear_fwd_carry(d, X.data_ptr(), Wp, None, None, Y1.data_ptr(),
                          _carry(L, opt, gam, bet, w2, b2), ws.data_ptr(), ws.numel() * 4, 0)
    torch.cuda.synchronize()
    assert torch.equal(Y0, Y1)
    for t in (gam, bet, w2, b2):
        t.same(torch)


@pytest.mark.parametrize("N,H,C,Co", [(8, 16, 64, 128), (128, 4, 256, 512), (4, 7, 3, 16)])
def test_conv_fwd_carry_bits(env, N, H, C, Co):
    torch, L, dev = env
    g = torch.Generator(device="cpu").manual_seed(N * H + C)
    X = torch.randn(N, H, H, C, generator=g).to(dev)
    Wt = (torch.randn(Co, 3, 3, C, generator=g) * 0.05).to(dev)
    b = torch.randn(Co, generator=g).to(dev)
    Wp = L.OfParam(Wt.data_ptr(), Wt.data_ptr(), None, None, Wt.numel())
    d = L.OfConvDesc(N, H, H, C, Co, L.OF_ACT_RELU, 1)
    wsb = L.of_conv_workspace_size(d, L.OF_CONV_FWD)
    ws = torch.empty(max(16, wsb) // 4 + 4, device=dev)
    Y0 = torch.empty(N, H, H, Co, device=dev)
    Y1 = torch.empty(N, H, H, Co, device=dev)
    opt = L.make_opt(HYPERS["sgd"], 4)
    t1 = _T(torch, L, dev, 512 * 9 * 512, "sgd", 5)
    t2 = _T(torch, L, dev, 512, "sgd", 6)
    L.of_conv_fwd(d, X.data_ptr(), Wp, b.data_ptr(), Y0.data_ptr(), ws.data_ptr(), ws.numel() * 4, 0)
    t1.reference_update(L, opt)
    t2.reference_update(L, opt)
    L.of_conv_fwd_carry(d, X.data_ptr(), Wp, b.data_ptr(), Y1.data_ptr(), _carry(L, opt, t1, t2),
                        ws.data_ptr(), ws.numel() * 4, 0)
    torch.cuda.synchronize()
    assert torch.equal(Y0, Y1)
    t1.same(torch)
    t2.same(torch)
