"""bfloat16 rounding for the oracle (test infrastructure only).

bfloat16 keeps the float32 exponent range (8 exponent bits) and 8 significant
bits (7 stored).  ``round_bf16`` rounds a float64 value directly to the
nearest bfloat16 value, ties to even, without an intermediate float32 step,
and returns it as float64.
"""

import numpy as np

_EMIN = -126  # smallest normal exponent of float32 / bfloat16
_P = 8        # significant bits of bfloat16


def round_bf16(x):
    """Round float64 array ``x`` to bfloat16 (RNE); result as float64.

    For |x| in [2^e, 2^(e+1)) the spacing of bfloat16 values is 2^(e-7);
    below the normal range it is the subnormal spacing 2^(-126-7).
    ``np.rint`` rounds half to even, which is exactly RNE on the scaled
    significand.  Values beyond the largest finite bfloat16 become inf.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros_like(x)
    nz = np.isfinite(x) & (x != 0.0)
    xv = x[nz]
    _m, e = np.frexp(xv)  # xv = m * 2**e with 0.5 <= |m| < 1
    e = e - 1             # now |xv| in [2**e, 2**(e+1))
    e = np.maximum(e, _EMIN)
    q = np.ldexp(1.0, e - (_P - 1))
    r = np.rint(xv / q) * q
    big = np.abs(r) > float.fromhex("0x1.fep127")
    r[big] = np.copysign(np.inf, r[big])
    out[nz] = r
    out[~np.isfinite(x)] = x[~np.isfinite(x)]
    # preserve signed zero
    z = x == 0.0
    out[z] = x[z]
    return out
