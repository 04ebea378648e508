"""bf16 rounding for the oracle (test infrastructure only).

bf16 keeps 8 significant bits and the fp32 exponent range.  ``round_bf16``
rounds an exact float64 value to the nearest bf16 value, ties to even, with
gradual underflow below 2^-126 (quantum 2^-133) and overflow to infinity at
or beyond the halfway point above the largest finite value.
"""

import numpy as np

_MIN_QUANTUM_EXP = -133          # bf16 subnormal spacing: 2^-126 * 2^-7


def round_bf16(x):
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)                                   # |x| = m * 2^e, m in [0.5, 1)
    q = np.maximum(e - 8, _MIN_QUANTUM_EXP)              # spacing of bf16 values near x
    r = np.ldexp(np.round(np.ldexp(x, -q)), q)           # np.round: ties to even
    with np.errstate(invalid="ignore"):
        r = np.where(np.abs(r) >= 2.0 ** 128, np.copysign(np.inf, x), r)
    return r


def bf16_bits_to_f64(bits):
    """Exact value of bf16 bit patterns."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def to_f64(a, dtype: str):
    """Exact float64 value of a stored weight/cache array of the model dtype."""
    if dtype == "bf16":
        return bf16_bits_to_f64(a)
    return np.asarray(a, dtype=np.float64)
