"""C-ABI checks that need no GPU: the library loads, exports every declared
entry point, and rejects bad arguments before any HIP call."""
import ctypes
import os
import re

import pytest

from paper_2104_00237_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "opfuse.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(of_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(L.LIB_PATH):
        pytest.skip("libopfuse.so not built")
    return L.load()


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
        assert n in L.exported_names(), f"binding lacks {n}"
    assert L.of_version() == 1


def _desc(M=8, N=16, K=12, **kw):
    d = L.OfLinearDesc(M, N, K, 0, 0, L.OF_F32, L.OF_ACT_NONE, 0)
    for k, v in kw.items():
        setattr(d, k, v)
    return d


FAKE = 0x10000  # never dereferenced: validation fails before any HIP call


def _status(fn, *args):
    with pytest.raises(L.OpfuseError) as e:
        fn(*args)
    return e.value.status


def _param(numel, w=FAKE, m=FAKE, v=FAKE):
    return L.OfParam(w, m, v, None, numel)


def test_linear_fwd_validation(lib):
    W = _param(16 * 12)
    assert _status(L.of_linear_fwd, None, FAKE, W, None, None, FAKE, None, 0, None) == L.OF_EINVAL
    assert _status(L.of_linear_fwd, _desc(M=0), FAKE, W, None, None, FAKE, None, 0, None) == L.OF_EINVAL
    assert _status(L.of_linear_fwd, _desc(), None, W, None, None, FAKE, None, 0, None) == L.OF_EINVAL
    assert _status(L.of_linear_fwd, _desc(), FAKE, _param(5), None, None, FAKE, None, 0, None) == L.OF_EINVAL
    assert _status(L.of_linear_fwd, _desc(act=7), FAKE, W, None, None, FAKE, None, 0, None) == L.OF_EINVAL
    assert _status(L.of_linear_fwd, _desc(has_bias=1), FAKE, W, None, None, FAKE, None, 0, None) == L.OF_EINVAL
    assert _status(L.of_linear_fwd, _desc(act=L.OF_ACT_GELU), FAKE, W, None, None, FAKE, None, 0,
                   None) == L.OF_EINVAL
    assert _status(L.of_linear_fwd, _desc(), FAKE + 2, W, None, None, FAKE, None, 0, None) == L.OF_EALIGN
    assert _status(L.of_linear_fwd, _desc(ldx=3), FAKE, W, None, None, FAKE, None, 0, None) == L.OF_EINVAL
    assert _status(L.of_linear_fwd, _desc(dtype=5), FAKE, W, None, None, FAKE, None, 0, None) == L.OF_EINVAL
    assert "ldx" in L.of_last_error() or "dtype" in L.of_last_error()


def test_workspace_query_and_check(lib):
    d = _desc(M=64, N=8192, K=8192)
    need = L.of_linear_workspace_size(d, L.OF_LINEAR_FWD)
    assert need > 0  # a reduction split is used for this shape
    W = _param(8192 * 8192)
    assert _status(L.of_linear_fwd, d, FAKE, W, None, None, FAKE, FAKE, need - 4, None) == L.OF_EWORKSPACE
    assert L.of_linear_workspace_size(_desc(M=0), 0) == 0
    assert L.of_linear_workspace_size(_desc(), 9) == 0


def test_optimizer_validation(lib):
    opt = L.make_opt(dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8), 0)
    p = _param(100)
    g = FAKE
    assert _status(L.of_elementwise_fused_update, p, g, 1, 0, opt, None) == L.OF_EINVAL  # step 0
    opt.step = 1
    assert _status(L.of_elementwise_fused_update, _param(100, v=None), g, 1, 0, opt, None) == L.OF_EINVAL
    assert _status(L.of_elementwise_fused_update, p, None, 1, 0, opt, None) == L.OF_EINVAL
    assert _status(L.of_elementwise_fused_update, p, g, 0, 0, opt, None) == L.OF_EINVAL
    assert _status(L.of_elementwise_fused_update, p, g, 2, 50, opt, None) == L.OF_EINVAL
    bad = L.make_opt(dict(kind="adam", lr=1e-3, beta1=1.5, beta2=0.999, eps=1e-8), 1)
    assert _status(L.of_elementwise_fused_update, p, g, 1, 0, bad, None) == L.OF_EINVAL
    bad.kind = 9
    assert _status(L.of_elementwise_fused_update, p, g, 1, 0, bad, None) == L.OF_EINVAL
    arr = (L.OfParam * 2)(p, _param(0))
    grads = (ctypes.c_void_p * 2)(FAKE, FAKE)
    assert _status(L.of_optimizer_step, 2, arr, grads, opt, None) == L.OF_EINVAL
    assert _status(L.of_optimizer_step, 0, arr, grads, opt, None) == L.OF_EINVAL
    # Fig. 7's other optimizers: known kinds, but eps must be positive; v is required
    for k in ("adagrad", "rmsprop", "adadelta"):
        o = L.make_opt(dict(kind=k, lr=0.01, eps=0.0), 1)
        assert _status(L.of_elementwise_fused_update, p, g, 1, 0, o, None) == L.OF_EINVAL
        assert "eps" in L.of_last_error()
        o.eps = 1e-8
        assert _status(L.of_elementwise_fused_update, _param(100, v=None), g, 1, 0, o,
                       None) == L.OF_EINVAL
    # m may be NULL only where the optimizer keeps none (Adagrad, RMSprop without momentum)
    no_m = _param(100, m=None)
    for hy in (dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8),
               dict(kind="rmsprop", lr=1e-3, alpha=0.99, eps=1e-8, momentum=0.9)):
        assert _status(L.of_elementwise_fused_update, no_m, g, 1, 0, L.make_opt(hy, 1),
                       None) == L.OF_EINVAL
        assert "->m is NULL" in L.of_last_error()
    for hy in (dict(kind="adagrad", lr=0.01, eps=1e-10),
               dict(kind="rmsprop", lr=1e-3, alpha=0.99, eps=1e-8)):
        # accepted: validation fails on the missing gradient instead
        assert _status(L.of_elementwise_fused_update, no_m, None, 1, 0, L.make_opt(hy, 1),
                       None) == L.OF_EINVAL
        assert "->m is NULL" not in L.of_last_error()
    sgd = L.make_opt(dict(kind="sgd", lr=0.1, momentum=0.9), 1)
    # SGD needs no v; a NULL m is still an error.
    assert _status(L.of_elementwise_fused_update, _param(10, m=None, v=None), g, 1, 0, sgd,
                   None) == L.OF_EINVAL


def test_fused_entry_validation(lib):
    d = _desc()
    W = _param(16 * 12)
    opt = L.make_opt(dict(kind="sgd", lr=0.1, momentum=0.9), 1)
    # forward-fusion needs the pending gradient
    assert _status(L.of_linear_fwd_fused, d, FAKE, W, None, None, None, None, None, opt, None, FAKE,
                   None, 0, None) == L.OF_EINVAL
    # more than one row tile (M > 64) needs the second buffer set; bf16 operands are refused
    big = _desc(M=65)
    assert _status(L.of_linear_fwd_fused, big, FAKE, W, None, FAKE, None, None, None, opt, None,
                   FAKE, None, 0, None) == L.OF_EUNSUPPORTED
    assert "W_out" in L.of_last_error()
    assert _status(L.of_linear_fwd_fused, _desc(dtype=L.OF_BF16), FAKE, W, _param(16 * 12, FAKE + 64),
                   FAKE, None, None, None, opt, None, FAKE, None, 0, None) == L.OF_EUNSUPPORTED
    # the second set must not share buffers with the first
    assert _status(L.of_linear_fwd_fused, big, FAKE, W, W, FAKE, None, None, None, opt, None,
                   FAKE, None, 0, None) == L.OF_EINVAL
    Wo = _param(16 * 12, FAKE + 64, FAKE + 128, FAKE + 192)
    assert _status(L.of_linear_fwd_fused, _desc(M=65, has_bias=1), FAKE, W, Wo, FAKE,
                   _param(16), None, FAKE, opt, None, FAKE, None, 0, None) == L.OF_EINVAL
    assert "b_out" in L.of_last_error()
    # backward-fusion: bad act_prev, and a dgrad that needs the saved tensor
    assert _status(L.of_linear_bwd_fused, d, FAKE, FAKE, W, None, None, None, opt, None, 4, FAKE,
                   None, 0, None, 0, None, None) == L.OF_EINVAL
    assert _status(L.of_linear_bwd_fused, d, FAKE, FAKE, W, None, None, None, opt, None,
                   L.OF_ACT_RELU, FAKE, None, 0, None, 0, None, None) == L.OF_EINVAL
    opt.step = -1
    assert _status(L.of_linear_bwd_fused, d, FAKE, FAKE, W, None, None, None, opt, None, 0, None,
                   None, 0, None, 0, None, None) == L.OF_EINVAL
    assert "step" in L.of_last_error()


def test_merged_entry_validation(lib):
    opt = L.make_opt(dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8), 1)
    d = _desc(M=64, N=8192, K=8192)
    W = _param(8192 * 8192)
    need = L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_MERGED)
    # partials of a few row ranges: more than nothing, at most an eighth of W
    assert 64 * 8192 * 4 <= need <= 8192 * 8192 * 4 // 8
    args = (FAKE, FAKE, W, None, None, None, opt, None, L.OF_ACT_NONE)
    assert _status(L.of_linear_bwd_merged, d, *args, FAKE, FAKE, need - 4, None) == L.OF_EWORKSPACE
    assert _status(L.of_linear_bwd_merged, d, *args, FAKE, None, need, None) == L.OF_EWORKSPACE
    assert _status(L.of_linear_bwd_merged, d, *args, FAKE, FAKE + 8, need, None) == L.OF_EALIGN
    # unsupported: more than 64 token rows, bf16 operands, very wide rows
    for bad in (_desc(M=65, N=8192, K=8192), _desc(M=64, N=8192, K=8192, dtype=L.OF_BF16),
                _desc(M=8, N=4, K=(1 << 22) + 1)):
        Wb = _param(bad.N * bad.K)
        assert L.of_linear_workspace_size(bad, L.OF_LINEAR_BWD_MERGED) == 0
        assert _status(L.of_linear_bwd_merged, bad, FAKE, FAKE, Wb, None, None, None, opt, None,
                       L.OF_ACT_NONE, FAKE, FAKE, 1 << 30, None) == L.OF_EUNSUPPORTED
    # the usual argument errors
    assert _status(L.of_linear_bwd_merged, d, None, FAKE, W, None, None, None, opt, None, 0,
                   None, None, 0, None) == L.OF_EINVAL
    assert _status(L.of_linear_bwd_merged, d, FAKE, FAKE, _param(7), None, None, None, opt, None,
                   0, None, None, 0, None) == L.OF_EINVAL
    assert _status(L.of_linear_bwd_merged, d, FAKE, FAKE, W, None, None, None, opt, None,
                   L.OF_ACT_RELU, FAKE, FAKE, need, None) == L.OF_EINVAL  # ReLU needs prev
    assert _status(L.of_linear_bwd_merged, d, FAKE, FAKE, W, _param(3), None, None, opt, None, 0,
                   None, None, 0, None) == L.OF_EINVAL  # bias of the wrong size
    opt.step = 0
    assert _status(L.of_linear_bwd_merged, d, *args, FAKE, FAKE, need, None) == L.OF_EINVAL


def test_loss_validation(lib):
    assert _status(L.of_xent_fwd_bwd, FAKE, FAKE, 0, 10, 0, FAKE, FAKE, None) == L.OF_EINVAL
    assert _status(L.of_xent_fwd_bwd, FAKE, FAKE + 4, 4, 10, 0, FAKE, FAKE, None) == L.OF_EALIGN
    assert _status(L.of_mse_fwd_bwd, FAKE, FAKE, 4, 8, 0, FAKE, FAKE, FAKE, 0, None) == L.OF_EWORKSPACE
    assert L.of_mse_workspace_size(4, 8) > 0


def test_bf16_shadow_and_norm_validation(lib):
    # a bf16 shadow with fp32 operands is a caller error
    Ws = L.OfParam(FAKE, FAKE, FAKE, FAKE, 16 * 12)
    assert _status(L.of_linear_fwd, _desc(), FAKE, Ws, None, None, FAKE, None, 0, None) == L.OF_EINVAL
    assert "w_bf16" in L.of_last_error()
    assert _status(L.of_linear_bwd_data, _desc(), FAKE, Ws, None, 0, FAKE, None, 0, None) == L.OF_EINVAL
    # odd shadow address
    Wo = L.OfParam(FAKE, FAKE, FAKE, FAKE + 1, 16 * 12)
    assert _status(L.of_linear_fwd, _desc(dtype=L.OF_BF16), FAKE, Wo, None, None, FAKE, None, 0,
                   None) == L.OF_EALIGN
    # bf16 workspace queries answer for the bf16 kernels (a split for a tall wgrad)
    assert L.of_linear_workspace_size(_desc(M=4096, N=1024, K=1024, dtype=L.OF_BF16),
                                      L.OF_LINEAR_BWD_WEIGHT) > 0
    assert _status(L.of_layernorm_fwd, FAKE, 0, 8, FAKE, FAKE, 1e-5, FAKE, FAKE, FAKE, None) == L.OF_EINVAL
    assert _status(L.of_layernorm_fwd, FAKE, 4, 8, FAKE, FAKE, 0.0, FAKE, FAKE, FAKE, None) == L.OF_EINVAL
    assert _status(L.of_layernorm_fwd, FAKE + 2, 4, 8, FAKE, FAKE, 1e-5, FAKE, FAKE, FAKE,
                   None) == L.OF_EALIGN
    assert _status(L.of_layernorm_bwd, FAKE, FAKE + 64, FAKE, FAKE, FAKE, None, 4, 8, FAKE, FAKE,
                   FAKE, None) == L.OF_EINVAL   # dx aliases dy
    # the halves may be computed apart, but not nothing and not one partial alone
    assert _status(L.of_layernorm_bwd, FAKE, FAKE + 64, FAKE, FAKE, FAKE, None, 4, 8, None, None,
                   None, None) == L.OF_EINVAL
    assert _status(L.of_layernorm_bwd, FAKE, FAKE + 64, FAKE, FAKE, FAKE, None, 4, 8, FAKE + 128,
                   FAKE + 256, None, None) == L.OF_EINVAL
    assert _status(L.of_layernorm_bwd, FAKE, FAKE + 64, FAKE, FAKE, None, None, 4, 8, FAKE + 128,
                   None, None, None) == L.OF_EINVAL   # dx needs gamma
    assert L.of_layernorm_partial_rows(4096) == 64 and L.of_layernorm_partial_rows(1) == 1
    # bf16 output: required, 2-byte aligned (4-byte alignment is not needed)
    assert _status(L.of_layernorm_fwd_bf16, FAKE, 4, 8, FAKE, FAKE, 1e-5, None, FAKE, FAKE,
                   None) == L.OF_EINVAL
    assert _status(L.of_layernorm_fwd_bf16, FAKE, 4, 8, FAKE, FAKE, 1e-5, FAKE + 1, FAKE, FAKE,
                   None) == L.OF_EALIGN
    assert _status(L.of_layernorm_fwd_bf16, FAKE + 2, 4, 8, FAKE, FAKE, 1e-5, FAKE, FAKE, FAKE,
                   None) == L.OF_EALIGN
    assert _status(L.of_reduce_rows, FAKE, 2, 3, 8, FAKE, None) == L.OF_EINVAL   # ld < n
    assert _status(L.of_add, FAKE, None, 8, FAKE, None) == L.OF_EINVAL


def test_carry_validation(lib):
    """of_linear_fwd_carry / of_conv_fwd_carry reject a malformed carried update
    before any HIP call (the forward's own arguments are valid)."""
    d = _desc()
    W = _param(16 * 12)
    adam = L.make_opt(dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8), 1)

    def fwd(carry):
        return _status(L.of_linear_fwd_carry, d, FAKE, W, None, None, FAKE, carry, None, 0, None)

    assert fwd(L.make_carry(adam, [])) == L.OF_EINVAL                      # n = 0
    over = L.make_carry(adam, [(_param(8), FAKE, 1)])
    over.n = L.OF_CARRY_MAX + 1
    assert fwd(over) == L.OF_EINVAL                                        # n > max
    assert fwd(L.make_carry(adam, [(_param(0), FAKE, 1)])) == L.OF_EINVAL  # empty tensor
    assert fwd(L.make_carry(adam, [(_param(8, v=None), FAKE, 1)])) == L.OF_EINVAL  # Adam needs v
    assert fwd(L.make_carry(adam, [(_param(8), None, 1)])) == L.OF_EINVAL  # no gradient
    assert fwd(L.make_carry(adam, [(_param(8), FAKE + 2, 1)])) == L.OF_EALIGN
    assert fwd(L.make_carry(adam, [(_param(8), FAKE, 0)])) == L.OF_EINVAL  # rows 0
    assert fwd(L.make_carry(adam, [(_param(8), FAKE, 1), (_param(4), None, 1)])) == L.OF_EINVAL
    bad = L.make_opt(dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8), 0)
    assert fwd(L.make_carry(bad, [(_param(8), FAKE, 1)])) == L.OF_EINVAL  # step 0
    cd = L.OfConvDesc(2, 4, 4, 3, 8, L.OF_ACT_RELU, 0)
    Wc = _param(8 * 9 * 3)
    assert _status(L.of_conv_fwd_carry, cd, FAKE, Wc, None, FAKE,
                   L.make_carry(adam, [(_param(8), None, 1)]), FAKE, 1 << 20, None) == L.OF_EINVAL


def test_clip_validation(lib):
    """of_grad_clip_scale rejects malformed arguments, and an optimizer with a
    misaligned gradient-scale address is rejected, before any HIP call."""
    ok = [(FAKE, 100, 1, 0), (FAKE, 10, 3, 16)]

    def clip(items, max_norm=1.0, scale=FAKE, norm=None, ws=FAKE, ws_bytes=L.OF_CLIP_WS_BYTES,
             n=None):
        refs = L.grad_refs(items) if items else None
        return _status(L.of_grad_clip_scale, len(items) if n is None else n, refs, max_norm,
                       scale, norm, ws, ws_bytes, None)

    assert clip([], n=0) == L.OF_EINVAL                              # no tensors
    assert clip(ok, max_norm=0.0) == L.OF_EINVAL
    assert clip(ok, max_norm=float("nan")) == L.OF_EINVAL
    assert clip(ok, max_norm=float("inf")) == L.OF_EINVAL
    assert clip(ok, scale=None) == L.OF_EINVAL
    assert clip(ok, scale=FAKE + 2) == L.OF_EALIGN
    assert clip(ok, norm=FAKE + 1) == L.OF_EALIGN
    assert clip(ok, ws=None) == L.OF_EWORKSPACE
    assert clip(ok, ws_bytes=L.OF_CLIP_WS_BYTES - 8) == L.OF_EWORKSPACE
    assert clip(ok, ws=FAKE + 4) == L.OF_EALIGN
    assert clip([(None, 100, 1, 0)]) == L.OF_EINVAL                  # no gradient
    assert clip([(FAKE + 2, 100, 1, 0)]) == L.OF_EALIGN
    assert clip([(FAKE, 0, 1, 0)]) == L.OF_EINVAL                    # empty tensor
    assert clip([(FAKE, 10, 0, 0)]) == L.OF_EINVAL                   # rows 0
    assert clip([(FAKE, 10, 2, 9)]) == L.OF_EINVAL                   # ld < numel
    opt = L.make_opt(dict(kind="sgd", lr=0.1, momentum=0.9), 1, None, FAKE + 2)
    assert _status(L.of_optimizer_step, 1, (L.OfParam * 1)(_param(8)),
                   (ctypes.c_void_p * 1)(FAKE), opt, None) == L.OF_EALIGN


def test_depthwise_validation(lib):
    opt = L.make_opt(dict(kind="sgd", lr=0.1, momentum=0.9), 1)
    d = L.OfConvDesc(2, 5, 7, 3, 3, L.OF_ACT_RELU, 1)
    need = L.of_dwconv_workspace_size(d)
    assert need >= 10 * 3 * 4
    bad = L.OfConvDesc(2, 5, 7, 3, 4, L.OF_ACT_NONE, 1)  # Cout != C
    assert L.of_dwconv_workspace_size(bad) == 0
    assert _status(L.of_dwconv_fwd, bad, FAKE, FAKE, FAKE, FAKE, None) == L.OF_EINVAL
    gelu = L.OfConvDesc(2, 5, 7, 3, 3, L.OF_ACT_GELU, 1)
    assert _status(L.of_dwconv_fwd, gelu, FAKE, FAKE, FAKE, FAKE, None) == L.OF_EUNSUPPORTED
    huge = L.OfConvDesc(1 << 12, 1 << 10, 1 << 10, 3, 3, L.OF_ACT_NONE, 0)
    assert _status(L.of_dwconv_fwd, huge, FAKE, FAKE, None, FAKE, None) == L.OF_EUNSUPPORTED
    assert _status(L.of_dwconv_fwd, d, FAKE, FAKE, None, FAKE, None) == L.OF_EINVAL  # bias
    assert _status(L.of_dwconv_fwd, d, FAKE + 2, FAKE, FAKE, FAKE, None) == L.OF_EALIGN
    assert _status(L.of_dwconv_bwd_data, d, FAKE, FAKE, None, L.OF_ACT_RELU, FAKE,
                   None) == L.OF_EINVAL
    assert _status(L.of_dwconv_bwd_data, d, FAKE, FAKE, FAKE, L.OF_ACT_GELU, FAKE,
                   None) == L.OF_EUNSUPPORTED
    assert _status(L.of_dwconv_bwd_weight, d, FAKE, FAKE, FAKE, None, 0, FAKE, need - 4,
                   None) == L.OF_EWORKSPACE
    assert _status(L.of_dwconv_bwd_weight, d, FAKE, FAKE, FAKE, None, 2, FAKE, need,
                   None) == L.OF_EINVAL
    W, b = _param(27), _param(3)
    assert _status(L.of_dwconv_wgrad_fused, d, FAKE, FAKE, _param(26), b, None, None, opt, FAKE,
                   need, None) == L.OF_EINVAL
    assert _status(L.of_dwconv_wgrad_fused, d, FAKE, FAKE, W, _param(4), None, None, opt, FAKE,
                   need, None) == L.OF_EINVAL
    assert _status(L.of_dwconv_wgrad_fused, d, FAKE, FAKE, W, b, None, None, opt, FAKE + 4,
                   need, None) == L.OF_EALIGN
    opt.step = 0
    assert _status(L.of_dwconv_wgrad_fused, d, FAKE, FAKE, W, b, None, None, opt, FAKE, need,
                   None) == L.OF_EINVAL
    # stride 2 is accepted (its slices follow the smaller output); stride 3 is not, and the
    # implicit-GEMM 3x3 convolutions run with stride 1 only
    s2 = L.OfConvDesc(2, 5, 7, 3, 3, L.OF_ACT_RELU, 1, 2)
    assert 0 < L.of_dwconv_workspace_size(s2) <= need
    s3 = L.OfConvDesc(2, 5, 7, 3, 3, L.OF_ACT_RELU, 1, 3)
    assert L.of_dwconv_workspace_size(s3) == 0
    assert _status(L.of_dwconv_fwd, s3, FAKE, FAKE, FAKE, FAKE, None) == L.OF_EUNSUPPORTED
    c2 = L.OfConvDesc(2, 5, 7, 3, 8, L.OF_ACT_RELU, 1, 2)
    assert L.of_conv_workspace_size(c2, L.OF_CONV_FWD) == 0
    assert "stride" in L.of_last_error()


def test_avgpool_validation(lib):
    assert _status(L.of_avgpool_fwd, None, 2, 49, 8, FAKE, None) == L.OF_EINVAL
    assert _status(L.of_avgpool_fwd, FAKE, 2, 0, 8, FAKE, None) == L.OF_EINVAL
    assert _status(L.of_avgpool_fwd, FAKE + 2, 2, 49, 8, FAKE, None) == L.OF_EALIGN
    assert _status(L.of_avgpool_fwd, FAKE, 1 << 20, 1 << 20, 8, FAKE, None) == L.OF_EUNSUPPORTED
    assert _status(L.of_avgpool_bwd, FAKE, None, 2, 49, 8, None, None) == L.OF_EINVAL
    assert _status(L.of_avgpool_bwd, FAKE, FAKE + 1, 2, 49, 8, FAKE, None) == L.OF_EALIGN


def test_hbm_stream_validation(lib):
    """The streaming probe: modes, required pointers and alignment are checked
    before any launch; the read-modify-write mode takes no source."""
    assert _status(L.of_hbm_stream, 5, FAKE, FAKE, 1024, 0, None) == L.OF_EINVAL
    # the merged kernel's layout: whole 32-row chunks of 8192-float rows, three arrays
    col = 3 * 8192 * 32
    assert _status(L.of_hbm_stream, L.OF_STREAM_RMW3_COLUMNS, None, FAKE, 1024, 0,
                   None) == L.OF_EINVAL
    assert _status(L.of_hbm_stream, L.OF_STREAM_RMW3_COLUMNS, None, FAKE, col + 12, 0,
                   None) == L.OF_EINVAL
    assert _status(L.of_hbm_stream, L.OF_STREAM_RMW3_COLUMNS, None, FAKE + 4, col, 0,
                   None) == L.OF_EALIGN
    # three arrays of float4s: n a multiple of 12
    assert _status(L.of_hbm_stream, L.OF_STREAM_RMW3, None, FAKE, 1024, 0, None) == L.OF_EINVAL
    assert _status(L.of_hbm_stream, L.OF_STREAM_RMW3, None, FAKE + 4, 1032, 0,
                   None) == L.OF_EALIGN
    assert _status(L.of_hbm_stream, L.OF_STREAM_COPY, None, FAKE, 1024, 0, None) == L.OF_EINVAL
    assert _status(L.of_hbm_stream, L.OF_STREAM_RMW, None, None, 1024, 0, None) == L.OF_EINVAL
    assert _status(L.of_hbm_stream, L.OF_STREAM_RMW, None, FAKE, 1022, 0, None) == L.OF_EINVAL
    assert _status(L.of_hbm_stream, L.OF_STREAM_RMW, None, FAKE + 4, 1024, 0, None) == L.OF_EALIGN
    assert _status(L.of_hbm_stream, L.OF_STREAM_COPY, FAKE, FAKE + 4, 1024, 0, None) == L.OF_EALIGN
    assert _status(L.of_hbm_stream, L.OF_STREAM_READ, FAKE, FAKE, 1024, 70000, None) == L.OF_EINVAL


def test_operand_size_limit(lib):
    """Operand tiles are addressed with 32-bit byte offsets from the tile's
    first element: every linear entry point rejects an operand matrix of 2 GiB
    or more (X, W or Y) before any HIP call, instead of reading zeros or
    wrapped data."""
    opt = L.make_opt(dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8), 1)
    cases = [_desc(M=1024, N=8, K=1 << 19),           # X is exactly 2 GiB
             _desc(M=8, N=1 << 19, K=1024),           # W is 2 GiB
             _desc(M=1024, N=8, K=16, ldy=1 << 19),   # Y's rows are 2 GiB apart in total
             _desc(M=2, N=4, K=4, ldx=1 << 62)]       # an absurd stride, no overflow
    for d in cases:
        W = _param(d.N * d.K)
        calls = [
            (L.of_linear_fwd, (d, FAKE, W, None, None, FAKE, FAKE, 1 << 40, None)),
            (L.of_linear_fwd_fused, (d, FAKE, W, None, FAKE, None, None, None, opt, None, FAKE,
                                     FAKE, 1 << 40, None)),
            (L.of_linear_bwd_data, (d, FAKE, W, None, L.OF_ACT_NONE, FAKE, FAKE, 1 << 40, None)),
            (L.of_linear_bwd_weight, (d, FAKE, FAKE, FAKE, None, 0, FAKE, 1 << 40, None)),
            (L.of_linear_bwd_fused, (d, FAKE, FAKE, W, None, None, None, opt, None, 0, FAKE,
                                     FAKE, 1 << 40, None, 0, None, None)),
        ]
        for fn, args in calls:
            assert _status(fn, *args) == L.OF_EUNSUPPORTED, (fn.__name__, d.M, d.N, d.K)
            assert "2 GiB" in L.of_last_error()
        assert L.of_linear_workspace_size(d, L.OF_LINEAR_FWD) == 0
    # just below the limit the shape is accepted (the missing x fails instead)
    d = _desc(M=1023, N=8, K=1 << 19)
    assert _status(L.of_linear_fwd, d, None, _param(8 << 19), None, None, FAKE, None, 0,
                   None) == L.OF_EINVAL


def test_merged_static_validation(lib):
    """The no-allocation merged backward validates like of_linear_bwd_merged and
    rejects shapes whose partials exceed the library's buffer, before any HIP
    call."""
    opt = L.make_opt(dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8), 1)
    big = _desc(M=64, N=1, K=(1 << 17) + 4)
    assert L.of_linear_workspace_size(big, L.OF_LINEAR_BWD_MERGED) > \
        L.OF_MERGED_STATIC_SCRATCH_BYTES
    Wb = _param(big.N * big.K)
    assert _status(L.of_linear_bwd_merged_static, big, FAKE, FAKE, Wb, None, None, None, opt,
                   None, L.OF_ACT_NONE, FAKE, None) == L.OF_EUNSUPPORTED
    assert "scratch" in L.of_last_error()
    d = _desc(M=64, N=8192, K=8192)
    W = _param(8192 * 8192)
    assert L.of_linear_workspace_size(d, L.OF_LINEAR_BWD_MERGED) <= \
        L.OF_MERGED_STATIC_SCRATCH_BYTES
    for bad in (_desc(M=65, N=8192, K=8192), _desc(M=64, N=8192, K=8192, dtype=L.OF_BF16)):
        assert _status(L.of_linear_bwd_merged_static, bad, FAKE, FAKE, _param(bad.N * bad.K),
                       None, None, None, opt, None, L.OF_ACT_NONE, FAKE, None) == \
            L.OF_EUNSUPPORTED
    assert _status(L.of_linear_bwd_merged_static, d, None, FAKE, W, None, None, None, opt, None,
                   0, None, None) == L.OF_EINVAL
    assert _status(L.of_linear_bwd_merged_static, d, FAKE, FAKE, W, None, None, None, opt, None,
                   L.OF_ACT_RELU, FAKE, None) == L.OF_EINVAL   # ReLU needs prev


def test_bf16_activation_storage_validation(lib):
    """of_linear_desc.io: bf16 storage of X / Y needs bf16 operands, known bits,
    the weight's shadow in a forward, and 2-byte (not 4-byte) alignment."""
    Ws = L.OfParam(FAKE, FAKE, FAKE, FAKE, 16 * 12)
    W = _param(16 * 12)
    xb, yb = L.OF_IO_X_BF16, L.OF_IO_Y_BF16
    # fp32 operands take no bf16 storage
    assert _status(L.of_linear_fwd, _desc(io=xb), FAKE, W, None, None, FAKE, None, 0,
                   None) == L.OF_EINVAL
    assert "io" in L.of_last_error()
    assert _status(L.of_linear_bwd_weight, _desc(io=xb), FAKE, FAKE, FAKE, None, 0, None, 0,
                   None) == L.OF_EINVAL
    assert L.of_linear_workspace_size(_desc(io=yb), L.OF_LINEAR_FWD) == 0
    # unknown bits
    assert _status(L.of_linear_fwd, _desc(dtype=L.OF_BF16, io=4), FAKE, Ws, None, None, FAKE,
                   None, 0, None) == L.OF_EINVAL
    # a forward reading bf16 X takes the weight from its bf16 shadow
    assert _status(L.of_linear_fwd, _desc(dtype=L.OF_BF16, io=xb), FAKE, W, None, None, FAKE,
                   None, 0, None) == L.OF_EINVAL
    assert "w_bf16" in L.of_last_error()
    # alignment: odd bf16 addresses fail, fp32 ones need 4 bytes
    assert _status(L.of_linear_fwd, _desc(dtype=L.OF_BF16, io=xb), FAKE + 1, Ws, None, None,
                   FAKE, None, 0, None) == L.OF_EALIGN
    assert _status(L.of_linear_fwd, _desc(dtype=L.OF_BF16, io=yb), FAKE, Ws, None, None,
                   FAKE + 1, None, 0, None) == L.OF_EALIGN
    assert _status(L.of_linear_fwd, _desc(dtype=L.OF_BF16, io=xb), FAKE, Ws, None, None,
                   FAKE + 2, None, 0, None) == L.OF_EALIGN     # y stays fp32
    assert _status(L.of_linear_bwd_weight, _desc(dtype=L.OF_BF16, io=xb), FAKE, FAKE + 1, FAKE,
                   None, 0, None, 0, None) == L.OF_EALIGN
    assert _status(L.of_linear_bwd_weight, _desc(dtype=L.OF_BF16), FAKE, FAKE + 2, FAKE, None, 0,
                   None, 0, None) == L.OF_EALIGN               # fp32 x
    opt = L.make_opt(dict(kind="sgd", lr=0.1, momentum=0.9, weight_decay=0.0), 1)
    assert _status(L.of_linear_bwd_fused, _desc(dtype=L.OF_BF16, io=xb), FAKE, FAKE + 1, Ws,
                   None, None, None, opt, None, 0, None, None, 0, None, 0, None,
                   None) == L.OF_EALIGN
    # forward-fusion and the merged backward take fp32 operands only
    assert _status(L.of_linear_fwd_fused, _desc(io=xb), FAKE, W, None, FAKE, None, None, None,
                   opt, None, FAKE, None, 0, None) == L.OF_EINVAL


def test_linear_fwd_res_validation(lib):
    """of_linear_fwd_res: the residual is required, 4-byte aligned, and either y
    itself (fp32 Y) or apart from y and z."""
    W = _param(16 * 12)
    Ws = L.OfParam(FAKE, FAKE, FAKE, FAKE, 16 * 12)
    d = _desc()                     # M 8, N 16: y spans 512 bytes
    Y = FAKE + 8192

    def st(desc, res, z, y, w=W):
        return _status(L.of_linear_fwd_res, desc, FAKE, w, None, res, z, y, None, None, 0, None)

    assert st(d, None, None, Y) == L.OF_EINVAL
    assert "res" in L.of_last_error()
    assert st(d, Y + 2 + 4096, None, Y) == L.OF_EALIGN
    assert st(d, Y + 64, None, Y) == L.OF_EINVAL            # overlaps y, not in place
    assert st(d, Y - 64, None, Y) == L.OF_EINVAL
    assert st(d, Y + 4096, Y + 4096 + 256, Y) == L.OF_EINVAL   # overlaps z
    # bf16 Y cannot be updated in place from an fp32 residual
    db = _desc(dtype=L.OF_BF16, io=L.OF_IO_Y_BF16)
    assert st(db, Y, None, Y, Ws) == L.OF_EINVAL
    # otherwise the usual checks apply
    assert st(d, Y + 4096, None, None) == L.OF_EINVAL        # y required


def test_linear_bwd_data_res_validation(lib):
    """of_linear_bwd_data_res: the residual gradient is required, 4-byte aligned,
    and either dx itself or apart from it."""
    W = _param(16 * 12)
    d = _desc()                     # M 8, K 12: dx spans 384 bytes
    DX = FAKE + 8192

    def st(res, dx):
        return _status(L.of_linear_bwd_data_res, d, FAKE, W, None, 0, res, dx, None, 0, None)

    assert st(None, DX) == L.OF_EINVAL
    assert st(DX + 4096 + 2, DX) == L.OF_EALIGN
    assert st(DX + 64, DX) == L.OF_EINVAL     # overlaps dx, not in place
    assert st(DX - 64, DX) == L.OF_EINVAL
    assert st(DX + 4096, None) == L.OF_EINVAL   # dx required
