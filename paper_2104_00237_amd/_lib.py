"""ctypes binding of libopfuse.so: argument marshalling only.

Each function has the C name and signature of include/opfuse.h; device
pointers are passed as Python ints, stream handles as ints (0 = null stream),
structs as the ctypes mirrors below.  A status other than OF_OK raises
OpfuseError with the library's message.  There is no fallback: if the
library is not built, loading fails loudly.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("OPFUSE_LIB", os.path.join(_HERE, "libopfuse.so"))

OF_OK, OF_EINVAL, OF_EUNSUPPORTED, OF_EALIGN, OF_EWORKSPACE, OF_EHIP = range(6)
STATUS_NAMES = {0: "OF_OK", 1: "OF_EINVAL", 2: "OF_EUNSUPPORTED", 3: "OF_EALIGN",
                4: "OF_EWORKSPACE", 5: "OF_EHIP"}
OF_F32, OF_BF16 = 0, 1
OF_IO_X_BF16, OF_IO_Y_BF16 = 1, 2   # of_linear_desc.io: bf16 storage of X / Y
OF_ACT_NONE, OF_ACT_RELU, OF_ACT_GELU = 0, 1, 2
OF_OPT_SGD, OF_OPT_ADAM, OF_OPT_ADAMW = 0, 1, 2
OF_OPT_ADAGRAD, OF_OPT_RMSPROP, OF_OPT_ADADELTA = 3, 4, 5
OF_LINEAR_FWD, OF_LINEAR_BWD_DATA, OF_LINEAR_BWD_WEIGHT, OF_LINEAR_BWD_MERGED = 0, 1, 2, 3
OF_CONV_FWD, OF_CONV_BWD_DATA, OF_CONV_BWD_WEIGHT = 0, 1, 2
ACTS = {"none": OF_ACT_NONE, "relu": OF_ACT_RELU, "gelu": OF_ACT_GELU}
OPT_KINDS = {"sgd": OF_OPT_SGD, "adam": OF_OPT_ADAM, "adamw": OF_OPT_ADAMW,
             "adagrad": OF_OPT_ADAGRAD, "rmsprop": OF_OPT_RMSPROP, "adadelta": OF_OPT_ADADELTA}

c_int32, c_int64, c_float, c_void_p, c_size_t = (ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                                  ctypes.c_void_p, ctypes.c_size_t)


class OfOpt(ctypes.Structure):
    _fields_ = [("kind", c_int32), ("lr", c_float), ("weight_decay", c_float),
                ("momentum", c_float), ("beta1", c_float), ("beta2", c_float),
                ("eps", c_float), ("step", c_int64), ("step_dev", c_void_p),
                ("grad_scale", c_void_p)]


class OfParam(ctypes.Structure):
    _fields_ = [("w", c_void_p), ("m", c_void_p), ("v", c_void_p), ("w_bf16", c_void_p),
                ("numel", c_int64)]


OF_CARRY_MAX = 4


class OfCarry(ctypes.Structure):
    _fields_ = [("n", c_int32), ("t", OfParam * OF_CARRY_MAX), ("g", c_void_p * OF_CARRY_MAX),
                ("rows", c_int64 * OF_CARRY_MAX), ("opt", OfOpt)]


OF_CLIP_WS_BYTES = 2048
OF_STREAM_READ, OF_STREAM_COPY, OF_STREAM_RMW, OF_STREAM_RMW3, OF_STREAM_RMW3_COLUMNS = 0, 1, 2, 3, 4
OF_MERGED_STATIC_SCRATCH_BYTES = 32 << 20   # of_linear_bwd_merged_static's buffer per device


class OfGradRef(ctypes.Structure):
    _fields_ = [("g", c_void_p), ("numel", c_int64), ("rows", c_int64), ("ld", c_int64)]


class OfLinearDesc(ctypes.Structure):
    _fields_ = [("M", c_int64), ("N", c_int64), ("K", c_int64), ("ldx", c_int64),
                ("ldy", c_int64), ("dtype", c_int32), ("act", c_int32), ("has_bias", c_int32),
                ("io", c_int32)]


class OfConvDesc(ctypes.Structure):
    _fields_ = [("N", c_int64), ("H", c_int64), ("W", c_int64), ("C", c_int64),
                ("Cout", c_int64), ("act", c_int32), ("has_bias", c_int32),
                ("stride", c_int32)]   # 0 or 1: stride 1; 2: depthwise stride 2


class OpfuseError(RuntimeError):
    def __init__(self, status, fn, msg):
        super().__init__(f"{fn}: {STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


P = ctypes.POINTER
_SIGS = {
    "of_version": (ctypes.c_int, []),
    "of_last_error": (ctypes.c_char_p, []),
    "of_linear_workspace_size": (c_size_t, [P(OfLinearDesc), c_int32]),
    "of_linear_fwd": (c_int32, [P(OfLinearDesc), c_void_p, P(OfParam), c_void_p, c_void_p,
                                c_void_p, c_void_p, c_size_t, c_void_p]),
    "of_linear_fwd_carry": (c_int32, [P(OfLinearDesc), c_void_p, P(OfParam), c_void_p, c_void_p,
                                      c_void_p, P(OfCarry), c_void_p, c_size_t, c_void_p]),
    "of_linear_fwd_res": (c_int32, [P(OfLinearDesc), c_void_p, P(OfParam), c_void_p, c_void_p,
                                    c_void_p, c_void_p, P(OfCarry), c_void_p, c_size_t,
                                    c_void_p]),
    "of_linear_fwd_fused": (c_int32, [P(OfLinearDesc), c_void_p, P(OfParam), P(OfParam),
                                      c_void_p, P(OfParam), P(OfParam), c_void_p, P(OfOpt),
                                      c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "of_linear_bwd_data": (c_int32, [P(OfLinearDesc), c_void_p, P(OfParam), c_void_p, c_int32,
                                     c_void_p, c_void_p, c_size_t, c_void_p]),
    "of_linear_bwd_data_res": (c_int32, [P(OfLinearDesc), c_void_p, P(OfParam), c_void_p,
                                         c_int32, c_void_p, c_void_p, c_void_p, c_size_t,
                                         c_void_p]),
    "of_linear_bwd_weight": (c_int32, [P(OfLinearDesc), c_void_p, c_void_p, c_void_p, c_void_p,
                                       c_int32, c_void_p, c_size_t, c_void_p]),
    "of_linear_bwd_fused": (c_int32, [P(OfLinearDesc), c_void_p, c_void_p, P(OfParam),
                                      P(OfParam), c_void_p, c_void_p, P(OfOpt), c_void_p,
                                      c_int32, c_void_p, c_void_p, c_size_t, c_void_p, c_size_t,
                                      c_void_p, c_void_p]),
    "of_linear_bwd_merged": (c_int32, [P(OfLinearDesc), c_void_p, c_void_p, P(OfParam),
                                       P(OfParam), c_void_p, c_void_p, P(OfOpt), c_void_p,
                                       c_int32, c_void_p, c_void_p, c_size_t, c_void_p]),
    "of_linear_bwd_merged_static": (c_int32, [P(OfLinearDesc), c_void_p, c_void_p, P(OfParam),
                                              P(OfParam), c_void_p, c_void_p, P(OfOpt), c_void_p,
                                              c_int32, c_void_p, c_void_p]),
    "of_hbm_stream": (c_int32, [c_int32, c_void_p, c_void_p, c_int64, c_int32, c_void_p]),
    "of_elementwise_fused_update": (c_int32, [P(OfParam), c_void_p, c_int64, c_int64,
                                              P(OfOpt), c_void_p]),
    "of_optimizer_step": (c_int32, [c_int32, P(OfParam), P(c_void_p), P(OfOpt), c_void_p]),
    "of_step_advance": (c_int32, [c_void_p, c_int64, c_void_p]),
    "of_grad_clip_scale": (c_int32, [c_int32, P(OfGradRef), c_float, c_void_p, c_void_p,
                                     c_void_p, c_size_t, c_void_p]),
    "of_conv_workspace_size": (c_size_t, [P(OfConvDesc), c_int32]),
    "of_conv_fwd": (c_int32, [P(OfConvDesc), c_void_p, P(OfParam), c_void_p, c_void_p, c_void_p,
                              c_size_t, c_void_p]),
    "of_conv_fwd_carry": (c_int32, [P(OfConvDesc), c_void_p, P(OfParam), c_void_p, c_void_p,
                                    P(OfCarry), c_void_p, c_size_t, c_void_p]),
    "of_conv_fwd_fused": (c_int32, [P(OfConvDesc), c_void_p, P(OfParam), P(OfParam), c_void_p,
                                    P(OfParam), P(OfParam), c_void_p, P(OfOpt), c_void_p,
                                    c_void_p, c_size_t, c_void_p]),
    "of_conv_bwd_data": (c_int32, [P(OfConvDesc), c_void_p, P(OfParam), c_void_p, c_int32,
                                   c_void_p, c_void_p, c_size_t, c_void_p]),
    "of_conv_bwd_weight": (c_int32, [P(OfConvDesc), c_void_p, c_void_p, c_void_p, c_void_p,
                                     c_int32, c_void_p, c_size_t, c_void_p]),
    "of_conv_wgrad_fused": (c_int32, [P(OfConvDesc), c_void_p, c_void_p, P(OfParam), P(OfParam),
                                      c_void_p, c_void_p, P(OfOpt), c_void_p, c_size_t,
                                      c_void_p]),
    "of_dwconv_workspace_size": (c_size_t, [P(OfConvDesc)]),
    "of_dwconv_fwd": (c_int32, [P(OfConvDesc), c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]),
    "of_dwconv_bwd_data": (c_int32, [P(OfConvDesc), c_void_p, c_void_p, c_void_p, c_int32,
                                     c_void_p, c_void_p]),
    "of_dwconv_bwd_weight": (c_int32, [P(OfConvDesc), c_void_p, c_void_p, c_void_p, c_void_p,
                                       c_int32, c_void_p, c_size_t, c_void_p]),
    "of_dwconv_wgrad_fused": (c_int32, [P(OfConvDesc), c_void_p, c_void_p, P(OfParam),
                                        P(OfParam), c_void_p, c_void_p, P(OfOpt), c_void_p,
                                        c_size_t, c_void_p]),
    "of_avgpool_fwd": (c_int32, [c_void_p, c_int64, c_int64, c_int64, c_void_p, c_void_p]),
    "of_avgpool_bwd": (c_int32, [c_void_p, c_void_p, c_int64, c_int64, c_int64, c_void_p,
                                 c_void_p]),
    "of_maxpool2x2_fwd": (c_int32, [c_void_p, c_int64, c_int64, c_int64, c_int64, c_void_p,
                                    c_void_p, c_void_p]),
    "of_maxpool2x2_bwd": (c_int32, [c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_int64,
                                    c_int64, c_void_p, c_void_p]),
    "of_layernorm_fwd": (c_int32, [c_void_p, c_int64, c_int64, c_void_p, c_void_p, c_float,
                                   c_void_p, c_void_p, c_void_p, c_void_p]),
    "of_layernorm_fwd_bf16": (c_int32, [c_void_p, c_int64, c_int64, c_void_p, c_void_p, c_float,
                                        c_void_p, c_void_p, c_void_p, c_void_p]),
    "of_layernorm_partial_rows": (c_int64, [c_int64]),
    "of_layernorm_bwd": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                   c_int64, c_int64, c_void_p, c_void_p, c_void_p, c_void_p]),
    "of_reduce_rows": (c_int32, [c_void_p, c_int64, c_int64, c_int64, c_void_p, c_void_p]),
    "of_add": (c_int32, [c_void_p, c_void_p, c_int64, c_void_p, c_void_p]),
    "of_xent_fwd_bwd": (c_int32, [c_void_p, c_void_p, c_int64, c_int64, c_int64, c_void_p,
                                  c_void_p, c_void_p]),
    "of_mse_workspace_size": (c_size_t, [c_int64, c_int64]),
    "of_mse_fwd_bwd": (c_int32, [c_void_p, c_void_p, c_int64, c_int64, c_int64, c_void_p,
                                 c_void_p, c_void_p, c_size_t, c_void_p]),
}

_lib = None


def load():
    """Load libopfuse.so (once).  Raises if it is missing: there is no fallback path."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"opfuse HIP library not found at {LIB_PATH}; build it with "
                               "`python -m paper_2104_00237_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def exported_names():
    return list(_SIGS)


def _wrap(name):
    def call(*args):
        lib = load()
        st = getattr(lib, name)(*args)
        if st != OF_OK:
            raise OpfuseError(st, name, lib.of_last_error().decode())
        return st
    call.__name__ = name
    return call


def of_version():
    return load().of_version()


def of_last_error():
    return load().of_last_error().decode()


def of_linear_workspace_size(desc, op):
    return load().of_linear_workspace_size(ctypes.byref(desc), op)


def of_mse_workspace_size(M, D):
    return load().of_mse_workspace_size(M, D)


def of_conv_workspace_size(desc, op):
    return load().of_conv_workspace_size(ctypes.byref(desc), op)


def of_dwconv_workspace_size(desc):
    return load().of_dwconv_workspace_size(ctypes.byref(desc))


def of_layernorm_partial_rows(M):
    return load().of_layernorm_partial_rows(M)


for _n in ("of_linear_fwd", "of_linear_fwd_carry", "of_linear_fwd_res", "of_conv_fwd_carry", "of_linear_fwd_fused", "of_linear_bwd_data", "of_linear_bwd_data_res", "of_linear_bwd_weight",
           "of_linear_bwd_fused", "of_linear_bwd_merged", "of_linear_bwd_merged_static",
           "of_hbm_stream", "of_elementwise_fused_update", "of_optimizer_step",
           "of_step_advance", "of_grad_clip_scale", "of_xent_fwd_bwd", "of_mse_fwd_bwd", "of_conv_fwd",
           "of_conv_fwd_fused", "of_conv_bwd_data", "of_conv_bwd_weight", "of_conv_wgrad_fused",
           "of_maxpool2x2_fwd", "of_maxpool2x2_bwd", "of_avgpool_fwd", "of_avgpool_bwd",
           "of_layernorm_fwd", "of_layernorm_fwd_bf16", "of_layernorm_bwd",
           "of_reduce_rows", "of_add", "of_dwconv_fwd", "of_dwconv_bwd_data",
           "of_dwconv_bwd_weight", "of_dwconv_wgrad_fused"):
    globals()[_n] = _wrap(_n)
del _n


def make_opt(hyper, step, step_dev=None, grad_scale=None):
    """of_opt from a workload's optimizer dict and the 1-based update index
    (or a device address holding it), with an optional device address of a
    gradient scale (e.g. the global-norm clipping factor)."""
    # the squared-gradient decay travels in beta2 (RMSprop's alpha, Adadelta's rho)
    beta2 = hyper.get("beta2", hyper.get("alpha", hyper.get("rho", 0.0)))
    return OfOpt(OPT_KINDS[hyper["kind"]], hyper["lr"], hyper.get("weight_decay", 0.0),
                 hyper.get("momentum", 0.0), hyper.get("beta1", 0.0), beta2,
                 hyper.get("eps", 0.0), step, step_dev, grad_scale)


def grad_refs(items):
    """HOST array of of_grad_ref from [(device pointer, numel, rows, ld), ...]."""
    return (OfGradRef * len(items))(*[OfGradRef(g, n, r, ld) for g, n, r, ld in items])


def make_carry(opt, tensors):
    """of_carry of [(OfParam, gradient device pointer, rows), ...] (at most
    OF_CARRY_MAX), all updated with `opt`."""
    c = OfCarry()
    c.n = len(tensors)
    for i, (p, g, rows) in enumerate(tensors):
        c.t[i] = p
        c.g[i] = g
        c.rows[i] = rows
    c.opt = opt
    return c


def param_of(w, m, v=None, w_bf16=None):
    """OfParam over torch tensors (device pointers taken once)."""
    return OfParam(w.data_ptr(), m.data_ptr(), v.data_ptr() if v is not None else None,
                   w_bf16.data_ptr() if w_bf16 is not None else None, w.numel())
