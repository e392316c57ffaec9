"""Round float64 values to the nearest bfloat16 value (ties to even).

bfloat16 keeps fp32's 8 exponent bits and 7 explicit mantissa bits.  The
accelerator rounds its fp32 accumulators to bf16 at storage points; the oracle
rounds its float64 values at the same points with this function.

Test infrastructure only (see the package docstring).
"""
import numpy as np

_MIN_NORMAL = 2.0 ** -126          # smallest normal bf16 (same as fp32)
_SUB_STEP = 2.0 ** -133            # spacing of bf16 subnormals
_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127
_HALF_ULP_MAX = 2.0 ** (127 - 8)   # values at or beyond _MAX + half ulp overflow


def round_bf16(x) -> np.ndarray:
    """Return float64 array of the bf16 values nearest to ``x`` (RNE)."""
    x = np.asarray(x, dtype=np.float64)
    out = np.array(x, dtype=np.float64, copy=True)
    a = np.abs(x)
    normal = np.isfinite(x) & (a >= _MIN_NORMAL)
    # normal range: keep the top 7 of fp64's 52 fraction bits, ties to even
    bits = out.view(np.uint64)
    drop = np.uint64(45)
    lsb = (bits >> drop) & np.uint64(1)
    rounded = (bits + (np.uint64((1 << 44) - 1) + lsb)) & ~np.uint64((1 << 45) - 1)
    bits[normal] = rounded[normal]
    # subnormal range: nearest multiple of 2^-133, ties to even (np.rint)
    sub = np.isfinite(x) & (a < _MIN_NORMAL)
    out[sub] = np.rint(x[sub] / _SUB_STEP) * _SUB_STEP
    # overflow
    big = np.isfinite(x) & (np.abs(out) > _MAX)
    out[big] = np.copysign(np.inf, x[big])
    return out


def identity(x):
    return np.asarray(x, dtype=np.float64)
