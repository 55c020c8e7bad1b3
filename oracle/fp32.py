"""Exact IEEE single-precision operations on fp64 carriers (test infrastructure).

The paper computes the Direct-P code map in FP32: scores arrive as FP32
accumulators and the score transform, block exponent and log2(6) term are folded
into the coefficients of one fused multiply-add per score (Sec. "Fix 1", the
paragraph after eq. affine-code-map).  Where such an fp32 value decides an
integer code, the oracle takes the same decision in the same precision, so it
needs a correctly rounded fp32 fused multiply-add.  NumPy has none; this module
builds one from exact fp64 products, Knuth's TwoSum error-free transformation,
and a correction of the one case in which rounding fp64 -> fp32 twice differs
from rounding once (an fp64 sum lying exactly on an fp32 midpoint).
"""
import numpy as np

f32 = np.float32
f64 = np.float64


def _two_sum(a, b):
    """s, e with s = fl64(a + b) and s + e = a + b exactly (Knuth); e = 0 where s
    is infinite (masked scores enter as -inf)."""
    s = a + b
    with np.errstate(invalid="ignore"):
        bb = s - a
        e = (a - (s - bb)) + (b - bb)
    return s, np.where(np.isfinite(s), e, 0.0)


def round_to_f32(s, e):
    """Correctly rounded fp32 of the exact value s + e (s = fl64(s + e), |e| <= ulp(s)/2)."""
    s = np.asarray(s, dtype=f64)
    e = np.asarray(e, dtype=f64)
    with np.errstate(over="ignore"):
        r = s.astype(f32)
    r64 = r.astype(f64)
    toward = np.where(s > r64, np.inf, -np.inf).astype(f32)
    other = np.nextafter(r, toward)
    mid = (r64 + other.astype(f64)) * 0.5
    on_mid = (s == mid) & (e != 0) & (s != r64)
    # On an exact fp32 midpoint the residual e decides the direction.
    hi = np.maximum(r, other)
    lo = np.minimum(r, other)
    fixed = np.where(e > 0, hi, lo)
    return np.where(on_mid, fixed, r).astype(f32)


def mul(a, b):
    """fp32 product of fp32 operands, correctly rounded."""
    p = np.asarray(a, dtype=f32).astype(f64) * np.asarray(b, dtype=f32).astype(f64)
    return p.astype(f32)  # the fp64 product of two fp32 values is exact


def fma(a, b, c):
    """fp32 fused multiply-add a*b + c with a single rounding."""
    p = np.asarray(a, dtype=f32).astype(f64) * np.asarray(b, dtype=f32).astype(f64)
    s, e = _two_sum(p, np.asarray(c, dtype=f32).astype(f64))
    return round_to_f32(s, e)
