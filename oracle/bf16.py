"""bfloat16 grid for the oracle (test infrastructure only).

bfloat16 keeps the float32 exponent range and 8 significant bits.  The oracle
models every tensor the layer stores in bf16 by rounding a float64 value to the
nearest bf16 number, ties to even, directly from float64 (no detour via
float32).
"""
import numpy as np


def round_bf16(x):
    """Nearest bfloat16 value of each element of ``x`` (float64 in, float64 out)."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                      # x = m * 2**e, 0.5 <= |m| < 1
    e = np.maximum(e, -125)                 # below 2**-126 the spacing stays 2**-133
    q = np.rint(np.ldexp(x, 8 - e))         # 8 significant bits, half-to-even
    out = np.ldexp(q, e - 8)
    big = np.abs(out) > 3.3895313892515355e38   # largest finite bf16
    return np.where(big, np.copysign(np.inf, x), out)


def from_bits(u16):
    """bf16 bit patterns (uint16) -> float64 values (exact)."""
    u = np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def to_bits(x):
    """float64 values already on the bf16 grid -> uint16 bit patterns."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    return (f.view(np.uint32) >> 16).astype(np.uint16)
