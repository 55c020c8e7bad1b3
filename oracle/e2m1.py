"""E2M1 payload of the FP4 formats (test infrastructure; see oracle/__init__).

The paper lists the non-negative E2M1 magnitudes as {0, 1/2, 1, 3/2, 2, 3, 4, 6}
(Sec. "Problem 2: P needs both range and cheap scales") and the seven value
boundaries between them as the midpoints {1/4, 3/4, 5/4, 7/4, 5/2, 7/2, 5}
(eq. e2m1-boundaries).  A 4-bit code is ``sign << 3 | k`` where ``k`` indexes
the magnitude table; bit 0 of ``k`` is the mantissa bit, so "ties to even"
means ties go to the even ``k``.

This module states rounding as its plain definition: the nearest table entry,
ties to the even index, values above 6 saturating to 6 (the largest entry is
also the nearest one).
"""
import numpy as np

MAGNITUDES = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float64)
MAX_MAGNITUDE = 6.0


def round_index(r):
    """Index k in 0..7 of the E2M1 magnitude nearest to ``r`` (>= 0).

    Ties between two neighbours go to the even index.  ``r`` above 6 maps to
    k = 7 (saturation).  ``r`` must be finite and non-negative.
    """
    r = np.asarray(r, dtype=np.float64)
    if np.any(~np.isfinite(r)) or np.any(r < 0):
        raise ValueError("round_index expects finite, non-negative magnitudes")
    r = np.minimum(r, MAX_MAGNITUDE)
    # The nearest entry is one of the two table entries that bracket r.
    hi = np.clip(np.searchsorted(MAGNITUDES, r, side="right"), 1, 7)
    lo = hi - 1
    # Both distances are exact in fp64 (Sterbenz: for r >= 1/2 the bracketing
    # entries lie within a factor of two of r), so equal distances are true ties.
    d_lo = r - MAGNITUDES[lo]
    d_hi = MAGNITUDES[hi] - r
    take_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    return np.where(take_hi, hi, lo).astype(np.uint8)


def round_value(r):
    """E2M1 magnitude nearest to ``r`` (ties to even, saturating at 6)."""
    return MAGNITUDES[round_index(r)]


def encode(v):
    """Signed E2M1 code (uint8 in 0..15) of ``v``: ``signbit << 3 | round_index(|v|)``."""
    v = np.asarray(v, dtype=np.float64)
    return (np.signbit(v).astype(np.uint8) << 3) | round_index(np.abs(v))


def decode(code):
    """Value of a signed E2M1 code (uint8 in 0..15)."""
    code = np.asarray(code, dtype=np.uint8)
    mag = MAGNITUDES[code & 7]
    return np.where(code & 8, -mag, mag)


def pack_nibbles(codes):
    """Pack codes along the last axis two per byte: element 2j in bits 3:0, 2j+1 in bits 7:4."""
    codes = np.asarray(codes, dtype=np.uint8)
    if codes.shape[-1] % 2:
        raise ValueError("last axis must be even")
    return (codes[..., 0::2] & 0xF) | ((codes[..., 1::2] & 0xF) << 4)


def unpack_nibbles(packed):
    """Inverse of :func:`pack_nibbles`."""
    packed = np.asarray(packed, dtype=np.uint8)
    out = np.empty(packed.shape[:-1] + (packed.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = packed & 0xF
    out[..., 1::2] = packed >> 4
    return out
