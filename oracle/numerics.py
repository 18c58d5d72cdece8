"""Storage rounding used by the oracle (test infrastructure only).

The paper does not state a precision. The workloads fix two storage formats:
float32 for the master weights W, the smoothed gradient v and the gradient g,
and bf16 for the operands and activations of the bf16 stages. The oracle
computes in float64 and rounds to those formats where a value is stored.
"""
import numpy as np


def to_f32(x):
    """Round float64 values to the nearest float32 value (IEEE, ties to even)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def to_bf16(x):
    """Round to bf16 the way a float32-producing kernel does: first to float32,
    then to the nearest bf16 (8 significant bits, ties to even).

    Written from the format definition: a normal bf16 number with exponent e
    (value in [2^e, 2^(e+1))) has spacing 2^(e-7); below 2^-126 the spacing
    is the subnormal one, 2^-133. np.rint rounds half to even.
    """
    f = to_f32(x)
    out = np.empty_like(f)
    finite = np.isfinite(f)
    fv = f[finite]
    mant, exp = np.frexp(fv)                 # fv = mant * 2^exp, |mant| in [0.5, 1)
    spacing_exp = np.maximum(exp - 8, -133)  # exponent of the bf16 spacing at fv
    out[finite] = np.ldexp(np.rint(np.ldexp(fv, -spacing_exp)), spacing_exp)
    out[~finite] = f[~finite]
    big = np.abs(out) > 3.3895313892515355e38   # beyond the largest finite bf16
    out[big & finite] = np.sign(out[big & finite]) * np.inf
    return out


def identity(x):
    return np.asarray(x, dtype=np.float64)
