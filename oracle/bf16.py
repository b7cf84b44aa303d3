"""bfloat16 <-> fp64 conversions for the oracle (test infrastructure only).

bf16 is the upper half of an IEEE binary32: 1 sign bit, 8 exponent bits and
7 stored significand bits.  Decoding is exact (shift into the top half of a
binary32).  Encoding rounds an fp64 value ONCE, to nearest with ties to even,
directly to bf16 -- never through binary32 first, which could round twice.

Non-finite values are outside the contract (inputs must be finite); encoding a
value beyond the largest finite bf16 gives +-inf, as IEEE rounding does.
"""

import numpy as np

F32 = "f32"
BF16 = "bf16"


def bf16_to_f64(bits):
    """Exact value of uint16 bf16 bit patterns, as float64."""
    bits = np.asarray(bits, dtype=np.uint16)
    as_u32 = bits.astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):  # NaN patterns stay NaN
        return as_u32.view(np.float32).astype(np.float64)


def f64_to_bf16(values):
    """Round float64 values to bf16 (nearest, ties to even); return uint16 bits.

    A finite v with frexp(v) = (m, ex), 0.5 <= |m| < 1, lies in the binade
    [2^(ex-1), 2^ex), where bf16's 8 significant bits give a spacing of
    2^(ex-8).  Below the smallest normal (2^-126) the spacing stays at the
    subnormal step 2^-133.  Dividing by a power of two and np.rint (which rounds
    half to even) are exact in fp64, so q = rint(v / ulp) * ulp is the correctly
    rounded bf16 value.  q is exactly representable in binary32, whose upper
    16 bits are then the bf16 pattern.
    """
    v = np.asarray(values, dtype=np.float64)
    _, ex = np.frexp(v)
    ulp_exp = np.maximum(ex.astype(np.int64) - 8, -133)
    ulp = np.ldexp(np.ones_like(v), ulp_exp)
    q = np.rint(v / ulp) * ulp
    with np.errstate(over="ignore"):
        q32 = q.astype(np.float32)  # exact for every finite bf16 value; inf beyond range
    return (q32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def decode(a, dtype):
    """Storage array (float32 or bf16 bits) -> exact float64 values."""
    if dtype == F32:
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    if dtype == BF16:
        return bf16_to_f64(a)
    raise ValueError(f"unknown dtype {dtype!r}")


def encode(v, dtype):
    """float64 values -> storage array, rounded once to nearest-even."""
    if dtype == F32:
        return np.asarray(v, dtype=np.float64).astype(np.float32)
    if dtype == BF16:
        return f64_to_bf16(v)
    raise ValueError(f"unknown dtype {dtype!r}")
