"""bfloat16 rounding for the bf16-operand workload.

The transformer-block workload rounds every matmul operand to bfloat16 with
round-to-nearest, ties-to-even, just before the contraction.  This is the
plain definition: the nearest value on the bfloat16 grid (8 significant bits,
exponent range of float32, gradual underflow below 2**-126), ties going to the
value whose last kept bit is 0; results beyond the largest finite bfloat16
value round to infinity; NaN and infinity pass through.

Pinned by: exact tie cases and grid values (tests/test_oracle_bf16.py) and a
comparison with the bit-level rounding of float32 inputs done independently
in that test.
"""
import numpy as np

_MAX_BF16 = (2.0 - 2.0 ** -7) * 2.0 ** 127


def round_bf16(x):
    """Round float64 values to the nearest bfloat16 value (ties to even); float64 out."""
    x = np.asarray(x, dtype=np.float64)
    out = x.copy()
    fin = np.isfinite(x) & (x != 0)
    xf = x[fin]
    _, e = np.frexp(xf)                 # |xf| = m * 2**e with 0.5 <= m < 1
    e = np.maximum(e, -125)             # below 2**-126 the grid spacing stays 2**-133
    spacing = np.ldexp(1.0, e - 8)      # 8 significant bits
    r = np.round(xf / spacing) * spacing  # numpy rounds halves to even
    r = np.where(np.abs(r) > _MAX_BF16, np.copysign(np.inf, r), r)
    out[fin] = r
    return out
