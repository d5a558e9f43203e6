"""of_linear_bwd_merged_static, the no-allocation variant of of_linear_bwd_merged
(its data-gradient partials live in a buffer the library holds per device),
against the workspace entry point through the C ABI: the same kernels and plan
run on both, so W, m, v, b and dX must be bit-identical.  Two shapes in a row,
the second smaller, so the second call reuses the buffer the first filled."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

ADAM = dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0)


def _state(torch, L, dev, r, M, N, K):
    t = lambda a: torch.as_tensor(np.ascontiguousarray(a, np.float32)).to(dev)  # noqa: E731
    s = dict(
        x=t(r.standard_normal((M, K))), dz=t(r.standard_normal((M, N)) * 0.05),
        prev=t(np.maximum(r.standard_normal((M, K)), 0)),
        w=t(r.standard_normal((N, K)) * 0.1), m=t(r.standard_normal((N, K)) * 0.01),
        v=t(r.random((N, K)) * 1e-4), b=t(r.standard_normal(N) * 0.1),
        bm=t(r.standard_normal(N) * 0.01), bv=t(r.random(N) * 1e-4))
    return s


def _clone(s):
    return {k: v.clone() for k, v in s.items()}


def _call(torch, L, s, M, N, K, static):
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 1)
    W = L.OfParam(s["w"].data_ptr(), s["m"].data_ptr(), s["v"].data_ptr(), None, N * K)
    B = L.OfParam(s["b"].data_ptr(), s["bm"].data_ptr(), s["bv"].data_ptr(), None, N)
    dx = torch.full((M, K), float("nan"), device=s["x"].device)
    opt = L.make_opt(ADAM, 4)
    stream = torch.cuda.current_stream().cuda_stream
    common = (d, s["dz"].data_ptr(), s["x"].data_ptr(), W, B, None, None, opt,
              s["prev"].data_ptr(), L.OF_ACT_RELU, dx.data_ptr())
    if static:
        L.of_linear_bwd_merged_static(*common, stream)
    else:
        need = L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_MERGED)
        ws = torch.empty(max(4, need // 4), device=s["x"].device)
        L.of_linear_bwd_merged(*common, ws.data_ptr(), ws.numel() * 4, stream)
    torch.cuda.synchronize()
    return dx


@pytest.mark.parametrize("first,second", [((64, 8192, 8192), (33, 1030, 2052)),
                                          ((64, 2048, 4096), (1, 8, 4))])
def test_static_scratch_matches_workspace_entry(gpu, first, second):
    import torch
    from paper_2104_00237_amd import _lib as L
    L.load()
    for i, (M, N, K) in enumerate((first, second)):
        d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 1)
        assert L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_MERGED) <= \
            L.OF_MERGED_STATIC_SCRATCH_BYTES
        print(f"no-alloc merged backward, call {i + 1}: M={M} N={N} K={K}", flush=True)
        r = np.random.default_rng(M + N + K)
        a = _state(torch, L, gpu, r, M, N, K)
        b = _clone(a)
        dx_ws = _call(torch, L, a, M, N, K, static=False)
        dx_st = _call(torch, L, b, M, N, K, static=True)
        assert not torch.isnan(dx_st).any()
        assert torch.equal(dx_st, dx_ws)
        for k in ("w", "m", "v", "b", "bm", "bv"):
            assert torch.equal(b[k], a[k]), k
        # the update moved W (the call did work, not only the data gradient)
        assert not torch.equal(a["w"], _state(torch, L, gpu, np.random.default_rng(M + N + K),
                                              M, N, K)["w"])


def test_static_scratch_rejects_large_shapes(gpu):
    """Partials above the library's buffer: OF_EUNSUPPORTED before any launch,
    and the arrays are left untouched."""
    import torch
    from paper_2104_00237_amd import _lib as L
    L.load()
    M, N, K = 64, 1, (1 << 17) + 4
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 0)
    assert L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_MERGED) > L.OF_MERGED_STATIC_SCRATCH_BYTES
    s = _state(torch, L, gpu, np.random.default_rng(5), M, N, K)
    w0 = s["w"].clone()
    W = L.OfParam(s["w"].data_ptr(), s["m"].data_ptr(), s["v"].data_ptr(), None, N * K)
    dx = torch.zeros((M, K), device=gpu)
    with pytest.raises(L.OpfuseError) as e:
        L.of_linear_bwd_merged_static(d, s["dz"].data_ptr(), s["x"].data_ptr(), W, None, None,
                                      None, L.make_opt(ADAM, 1), None, L.OF_ACT_NONE,
                                      dx.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert e.value.status == L.OF_EUNSUPPORTED and "scratch" in L.of_last_error()
    torch.cuda.synchronize()
    assert torch.equal(s["w"], w0)
