"""bf16 <-> fp32 conversions of the oracle, from the IEEE 754 definitions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper reduces in FP32 and converts the sum back to the element type
``E`` once the sum is complete (Section 3.3, "Deterministic reduction within
the pipeline", Eq. 2).  It does not say how that conversion rounds; the
oracle reads it as IEEE 754 roundTiesToEven, the default rounding of binary
floating point.

bfloat16 is the binary32 format with the low 16 significand bits removed:
1 sign bit, 8 exponent bits, 7 stored significand bits.  Its encoding is the
upper half of a binary32 encoding.
"""

import numpy as np

_F32_INF_AS_F64 = 2.0**128  # the value "one step past max finite" under an unbounded exponent


def widen(h):
    """bf16 encodings (uint16) -> float32, exactly.

    Every bf16 value is a binary32 value whose low 16 encoding bits are zero,
    so widening places the 16 bits in the upper half of a 32-bit word.
    """
    h = np.asarray(h, dtype=np.uint16)
    return (h.astype(np.uint32) << np.uint32(16)).view(np.float32)


def narrow(x):
    """float32 -> bf16 encodings (uint16), round to nearest, ties to even.

    Written as the definition of rounding rather than as a bit trick:

    * the two bf16 candidates that bracket ``x`` are ``lo`` (``x`` truncated
      toward zero: its upper 16 encoding bits) and ``hi`` (the next bf16
      away from zero: encoding ``lo + 1``, which is how sign-magnitude
      encodings step);
    * the result is the candidate nearer to ``x``; on a tie, the one whose
      encoding ends in a 0 bit (the even significand);
    * IEEE 754 rounds as if the exponent range were unbounded and then
      overflows, so when ``hi`` is +-infinity its distance is taken to
      +-2**128, the next value past the largest finite one.  A value at or
      beyond max-finite + half an ulp therefore becomes infinity.

    Distances are computed in float64: ``x``, ``lo`` and ``hi`` are binary32
    values within a factor of two of each other, so their differences are
    exact in float64.

    Readings where the paper is silent: infinities stay infinities; a NaN
    becomes a quiet NaN that keeps its sign and its top significand bits
    (encoding ``upper16 | 0x0040``); denormals are rounded like any other
    value (no flush to zero).
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    lo_bits = (u >> np.uint32(16)).astype(np.uint16)
    exact = (u & np.uint32(0xFFFF)) == 0
    is_nan = np.isnan(x)

    # hi is only needed where x is finite and not exact; guard the encoding
    # step so NaN encodings (upper16 == 0x7FFF / 0xFFFF) cannot wrap.
    hi_bits = np.where(is_nan | exact, lo_bits, lo_bits + np.uint16(1)).astype(np.uint16)

    with np.errstate(invalid="ignore"):  # NaN lanes are overwritten below
        xd = x.astype(np.float64)
        lo = widen(lo_bits).astype(np.float64)
        hi = widen(hi_bits).astype(np.float64)
        hi = np.where(np.isinf(hi), np.copysign(_F32_INF_AS_F64, xd), hi)
        d_lo = np.abs(xd - lo)
        d_hi = np.abs(hi - xd)
    lo_is_even = (lo_bits & np.uint16(1)) == 0
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & ~lo_is_even)

    out = np.where(pick_hi, hi_bits, lo_bits).astype(np.uint16)
    out = np.where(exact, lo_bits, out)
    out = np.where(is_nan, lo_bits | np.uint16(0x0040), out)
    return out.astype(np.uint16)
