"""Rounding onto the bfloat16 grid, written from the format's definition.

bfloat16 keeps the float32 exponent range (8 exponent bits) and 8 significant
bits (7 stored fraction bits plus the implicit one). Rounding is to the nearest
representable value with ties to the even significand, the IEEE-754 default.

This implementation works on float64 inputs with exact arithmetic (frexp,
ldexp and rint are all exact in float64 here), so a float64 value is rounded
once, directly, rather than first to float32 and then to bfloat16.

Test infrastructure only (see the package docstring).
"""

import numpy as np

# Largest finite bfloat16: (2 - 2**-7) * 2**127.
BF16_MAX = float(np.ldexp(2.0 - 2.0 ** -7, 127))
# Exponent (frexp convention, |x| in [2**(e-1), 2**e)) of the smallest normal
# bfloat16 2**-126; below it the grid spacing stays at 2**-133 (subnormals).
_EMIN = -125
_SIG_BITS = 8


def round_bf16(x):
    """Round to the nearest bfloat16 value (ties to even); returns float64.

    Finite values beyond the largest bfloat16 after rounding become +-inf,
    infinities and NaNs pass through unchanged.
    """
    a = np.asarray(x, dtype=np.float64)
    finite = np.isfinite(a)
    safe = np.where(finite, a, 0.0)
    _, e = np.frexp(safe)
    e = np.maximum(e, _EMIN)
    # Grid spacing 2**(e - 8): scale so the grid becomes the integers, round
    # half to even (np.rint), scale back. Both scalings are exact.
    q = np.ldexp(np.rint(np.ldexp(safe, _SIG_BITS - e)), e - _SIG_BITS)
    q = np.where(np.abs(q) > BF16_MAX, np.copysign(np.inf, q), q)
    return np.where(finite, q, a)


def is_bf16_representable(x):
    """True where x lies exactly on the bfloat16 grid."""
    a = np.asarray(x, dtype=np.float64)
    return (round_bf16(a) == a) | ~np.isfinite(a)
