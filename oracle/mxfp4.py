"""MXFP4 input quantizer (test infrastructure; see oracle/__init__).

Format (Sec. "Problem 2", Table fp4-formats and eq. mx-scale): blocks of 32
values share one E8M0 byte ``u``; the block amplitude is ``alpha = 2**(u - 127)``
and a value is represented as ``alpha * q / 6`` with ``q`` an E2M1 magnitude and
a sign bit.  The paper stores the amplitude, not the step ``alpha / 6``.

For a block with absolute maximum ``a`` the paper offers two amplitudes,
``2**floor(log2 a)`` and ``2**ceil(log2 a)`` (eq. mx-scale), without a rule to
pick one.  This oracle takes the one with the smaller squared reconstruction
error over the block, and the ceiling on a tie.

The two errors are compared exactly.  With ``r_j = 6|v_j| / 2**e_c`` the ceiling
codes are ``qc_j = Q(r_j)`` and the floor codes ``qf_j = Q(2 r_j)``; in units of
``(2**e_c / 6)**2`` the errors are ``sum (r - qc)**2`` and ``sum (2r - qf)**2 / 4``.
Their difference times four factors as
``delta = sum (2 qc - qf) * (4 r - qf - 2 qc)``; every term and partial sum is
exactly representable in fp64 for fp32 or bf16 inputs, so the sign of
``delta`` is the exact comparison (floor iff ``delta < 0``).

Layout produced (and consumed by :mod:`oracle.directp`):

* ``axis=-1`` (Q, K ``[..., N, d]``): codes ``[..., N, d/2]`` (two per byte, even
  element in the low nibble), scales ``[..., N, d/32]``.
* ``axis=-2`` (V ``[..., N, d]``, blocks along the sequence): the result is
  stored transposed, codes ``[..., d, N/2]`` and scales ``[..., d, N/32]``.

Non-finite blocks get scale byte 255 (E8M0 NaN) and zero code bytes.  An
all-zero block gets scale byte 0; its codes keep each value's sign bit.
Block exponents are clamped to the E8M0 range [-127, 127] and codes are
computed with the clamped exponent.
"""
import numpy as np

from . import e2m1

BLOCK = 32


def _as_f64(x):
    return np.asarray(x, dtype=np.float64)


def _block_exponents(a):
    """(e_floor, e_ceil) with 2**e_floor <= a <= 2**e_ceil, exact via frexp (a > 0)."""
    m, x = np.frexp(a)  # a = m * 2**x, m in [0.5, 1)
    pow2 = m == 0.5
    e_floor = np.where(pow2, x - 1, x - 1)
    e_ceil = np.where(pow2, x - 1, x)
    return e_floor.astype(np.int64), e_ceil.astype(np.int64)


def choose_exponent(blocks):
    """E8M0 exponent chosen for each row of ``blocks`` (shape [..., 32]).

    Returns (exponent int64, finite-and-nonzero mask).  Zero or non-finite blocks
    get exponent 0 and mask False.
    """
    v = _as_f64(blocks)
    mag = np.abs(v)
    a = mag.max(axis=-1)
    ok = np.isfinite(a) & (a > 0)
    a_safe = np.where(ok, a, 1.0)
    e_f, e_c = _block_exponents(a_safe)
    r = np.ldexp(6.0 * np.where(np.isfinite(mag), mag, 0.0), -e_c[..., None])
    qc = e2m1.round_value(r)
    qf = e2m1.round_value(2.0 * r)
    delta = np.sum((2.0 * qc - qf) * (4.0 * r - qf - 2.0 * qc), axis=-1)
    e = np.where((e_f != e_c) & (delta < 0), e_f, e_c)
    e = np.where(ok, e, 0)
    return e, ok


def squared_errors(blocks):
    """Exact (floor, ceil) squared reconstruction errors of each block as Fractions.

    Slow; a check on :func:`choose_exponent` for small inputs.
    """
    from fractions import Fraction

    out = []
    for row in np.asarray(blocks, dtype=np.float64).reshape(-1, BLOCK):
        a = float(np.max(np.abs(row)))
        e_f, e_c = (int(t) for t in _block_exponents(np.array(a)))
        errs = []
        for e in (e_f, e_c):
            step = Fraction(2) ** e / 6
            tot = Fraction(0)
            for x in row:
                r = np.ldexp(6.0 * abs(float(x)), -e)  # exact: 6|x| / 2**e
                q = Fraction(float(e2m1.round_value(r)))
                tot += (Fraction(abs(float(x))) - step * q) ** 2
            errs.append(tot)
        out.append(tuple(errs))
    return out


def quantize(x, axis=-1):
    """MXFP4 codes and E8M0 scales of ``x`` in blocks of 32 along ``axis``.

    ``axis=-1`` keeps the layout; ``axis=-2`` stores the transposed result
    (see module docstring).  Returns (codes uint8 packed, scales uint8).
    """
    x = _as_f64(x)
    ax = axis % x.ndim
    if x.ndim >= 2 and ax == x.ndim - 2:
        x = np.swapaxes(x, -1, -2)
    elif ax != x.ndim - 1:
        raise ValueError("axis must be the last or the second-to-last axis")
    if x.shape[-1] % BLOCK:
        raise ValueError("blocked axis must be a multiple of 32")
    blocks = x.reshape(x.shape[:-1] + (x.shape[-1] // BLOCK, BLOCK))
    e, ok = choose_exponent(blocks)
    finite = np.all(np.isfinite(blocks), axis=-1)
    e = np.clip(e, -127, 127)
    u = (e + 127).astype(np.int64)
    u = np.where(ok, u, 0)
    u = np.where(finite, u, 255).astype(np.uint8)
    mag = np.where(np.isfinite(blocks), np.abs(blocks), 0.0)
    r = np.ldexp(6.0 * mag, -e[..., None])
    codes = (np.signbit(blocks).astype(np.uint8) << 3) | e2m1.round_index(r)
    codes = np.where(finite[..., None], codes, 0).astype(np.uint8)
    codes = codes.reshape(x.shape)
    return e2m1.pack_nibbles(codes), u


def dequantize(codes, scales):
    """Represented values ``2**(u-127) * q / 6`` (fp64), in the stored layout.

    Blocks with scale byte 255 decode to NaN.
    """
    q = e2m1.decode(e2m1.unpack_nibbles(codes))
    s = np.asarray(scales, dtype=np.int64)
    alpha = np.where(s == 255, np.nan, np.ldexp(1.0, s - 127))
    alpha = np.repeat(alpha, BLOCK, axis=-1)
    return alpha * q / 6.0


def scaled_operand(codes, scales):
    """``6 * dequantize``: ``2**(u-127) * q``, the value a block-scaled FP4 matrix unit multiplies."""
    q = e2m1.decode(e2m1.unpack_nibbles(codes))
    s = np.asarray(scales, dtype=np.int64)
    alpha = np.where(s == 255, np.nan, np.ldexp(1.0, s - 127))
    return np.repeat(alpha, BLOCK, axis=-1) * q
