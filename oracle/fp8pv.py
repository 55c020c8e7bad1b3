"""MXFP4 QK with FP8 (E4M3) P and V (test infrastructure; see oracle/__init__).

The paper keeps FP8 probabilities and values as its accuracy control and in
its retained training route (Table accuracy-matched-control, the exact NV/FP8
route; Table causal-precision-contract, "FP8 P and V"; Sec. "Training stability
selects FP8 P/V").  On the block-scaled matrix unit used here the FP8 operand
is MXFP8: an E4M3 payload (bias 7, three mantissa bits, largest finite 448,
subnormals down to 2**-9) with one E8M0 byte per 32 values.  The paper does
not spell out the FP8 encodings, so the readings below are this module's:

1. V (:func:`quantize`): per block of 32 values along the sequence, the
   amplitude ``2**e`` is the smallest power of two with ``amax / 2**e <= 448``
   (no element saturates); payload ``E4M3(v / 2**e)``, nearest with ties to the
   even code; byte ``u = clamp(e + 127, 0, 254)``; an all-zero block has
   ``u = 0``; a block with a non-finite value has ``u = 255`` and zero codes.
   The represented value is ``2**(u - 127) * e4m3(code)``.
2. P (the ideal converter of eq. ideal-code-path with an E4M3 payload): the
   block exponent ``E_B = floor(max_{j in B} y_ij)`` exactly as in Direct-P,
   ``x = y - E_B + 7`` (one fp32 fma: ``x = fma(c_y, raw, 7 - E_B)``), and
   ``q8 = E4M3(fp32(2**x))``: the block maximum lands in [128, 256), every
   payload stays below the E4M3 maximum.  The E8M0 byte is
   ``u_B = clamp(E_B - M_i + 120, 0, 254)``, so ``2**(u_B - 127) q8`` stands for
   ``2**(y - M_i)``.
3. Denominator from the same payload and bytes (Fix 2's principle,
   eq. represented-contributions): ``D_i = sum_B 2**(E_B - M_i - 7) sum_j q8_ij``;
   output ``O_i = sum_B 2**(E_B - M_i - 7) sum_j q8_ij Vhat_j / D_i``.
   The causal form masks keys j > i as :mod:`oracle.directp` does.
"""
import numpy as np

from . import directp, fp32, mxfp4, prange

BLOCK = 32
E4M3 = prange.E4M3          # non-negative finite E4M3 values in code order (0x00 .. 0x7E)
E4M3_MAX = 448.0


def e4m3_index(x):
    """Code index (0 .. 126) of the E4M3 value nearest to ``0 <= x <= 448``, ties to
    the even code."""
    x = np.asarray(x, dtype=np.float64)
    if np.any(x > E4M3_MAX) or np.any(x < 0):
        raise ValueError("E4M3 payloads here stay within [0, 448]")
    hi = np.clip(np.searchsorted(E4M3, x, side="left"), 1, len(E4M3) - 1)
    lo = hi - 1
    d_lo = x - E4M3[lo]
    d_hi = E4M3[hi] - x
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    return np.where(pick_hi, hi, lo).astype(np.uint8)


def block_exponent(amax):
    """Smallest e with amax <= 448 * 2**e (amax > 0), exactly."""
    m, x = np.frexp(np.asarray(amax, dtype=np.float64))     # amax = m 2**x, m in [0.5, 1)
    e = x - 1 - 8                                            # amax / 2**e in [256, 512)
    return np.where(np.ldexp(np.asarray(amax, dtype=np.float64), -e) > E4M3_MAX, e + 1, e).astype(np.int64)


def quantize(x, axis=-1):
    """MXFP8 (E4M3 + E8M0 per 32 values along ``axis``) of fp64 ``x``.

    axis=-1: codes [..., rows, cols] uint8, scales [..., rows, cols/32].
    axis=-2: blocks along rows, stored transposed: codes [..., cols, rows], scales [..., cols, rows/32].
    Code byte = sign << 7 | E4M3 index.
    """
    x = np.asarray(x, dtype=np.float64)
    ax = axis % x.ndim
    if ax == x.ndim - 2:
        x = np.swapaxes(x, -1, -2)
    elif ax != x.ndim - 1:
        raise ValueError("axis must be -1 or -2")
    lead, n = x.shape[:-1], x.shape[-1]
    if n % BLOCK:
        raise ValueError("the blocked extent must be a multiple of 32")
    blk = x.reshape(lead + (n // BLOCK, BLOCK))
    finite = np.all(np.isfinite(blk), axis=-1)
    amax = np.max(np.abs(np.where(np.isfinite(blk), blk, 0.0)), axis=-1)
    pos = finite & (amax > 0)
    e = np.where(pos, block_exponent(np.where(pos, amax, 1.0)), 0)
    e = np.clip(e, -127, 127)
    u = np.where(finite, np.where(amax > 0, e + 127, 0), 255).astype(np.uint8)
    scaled = np.ldexp(np.abs(np.where(np.isfinite(blk), blk, 0.0)), -e[..., None])
    idx = e4m3_index(np.minimum(scaled, E4M3_MAX))
    codes = (idx | np.where(np.signbit(blk), 0x80, 0)).astype(np.uint8)
    codes = np.where(finite[..., None], codes, 0).astype(np.uint8)
    return codes.reshape(lead + (n,)), u


def dequantize(codes, scales):
    """Represented values ``2**(u - 127) e4m3(code)`` [..., n] (blocks along the last axis)."""
    codes = np.asarray(codes, dtype=np.uint8)
    mag = E4M3[np.minimum(codes & 0x7F, 0x7E)]
    val = np.where(codes & 0x80, -mag, mag)
    n = codes.shape[-1]
    w = np.ldexp(1.0, np.repeat(np.asarray(scales).astype(np.int64) - 127, BLOCK, axis=-1))
    return val.reshape(codes.shape[:-1] + (n,)) * w


def p_codes(raw, softmax_scale, visible=None):
    """(E [R, N/32] int64 block exponents, q8 [R, N] E4M3 values, k [R, N] E4M3 indices)."""
    R, N = raw.shape
    nb = N // BLOCK
    if visible is not None:
        raw = np.where(visible, raw, -np.inf)
    c_y, _, _ = directp.fp32_coefficients(softmax_scale, 1.5, 1.2)
    raw32 = raw.astype(np.float32)
    y = fp32.mul(raw32, c_y)
    with np.errstate(invalid="ignore"):
        ymax = y.reshape(R, nb, BLOCK).max(axis=-1).astype(np.float64)
    E = np.where(np.isfinite(ymax), np.floor(np.nan_to_num(ymax, neginf=0.0)), directp.NO_BLOCK).astype(np.int64)
    c7 = np.where(E == directp.NO_BLOCK, 0, 7 - E).astype(np.float32)      # exact for the exponents met
    x = fp32.fma(c_y, raw32, np.repeat(c7, BLOCK, axis=-1)).astype(np.float64)
    with np.errstate(over="ignore"):
        p = np.exp2(x).astype(np.float32).astype(np.float64)                 # fp32(2**x), -inf -> 0
    k = e4m3_index(p)
    return E, E4M3[k], k


def forward_rows(q_codes, q_scales, k_codes, k_scales, vt8_codes, vt8_scales, rows, softmax_scale,
                 causal=False, want_codes=True, exact_p=False):
    """FP8-P/V forward for the query ``rows`` of ONE (batch, head) slice.

    Q, K: MXFP4 as :func:`oracle.mxfp4.quantize`; V^T: MXFP8 from :func:`quantize`
    with ``axis=-2`` (codes [d, N], scales [d, N/32]).  Returns E, M, D (relative
    to 2**M, with the payload's 2**-7 folded in), O, LSE (natural log,
    ``M ln 2 + ln D``: ``2**(E_B - 7) q8`` stands for ``exp(z)``) and, with
    ``want_codes``, the P payload indices.  ``exact_p`` uses unrounded 2**x.
    """
    rows = np.asarray(rows, dtype=np.int64)
    q6 = mxfp4.scaled_operand(q_codes, q_scales)[rows]
    k6 = mxfp4.scaled_operand(k_codes, k_scales)
    v = dequantize(vt8_codes, vt8_scales).T                       # [N, d] represented V
    raw = directp.raw_scores(q6, k6)
    N = raw.shape[1]
    vis = (np.arange(N)[None, :] <= rows[:, None]) if causal else None
    E, q8, k = p_codes(raw, softmax_scale, vis)
    if exact_p:   # fp64 scores, like directp's exp2_exact mode
        y = raw * (float(np.float32(softmax_scale)) / 36.0) * directp.LOG2_E
        if vis is not None:
            y = np.where(vis, y, -np.inf)
        q8 = np.exp2(y - np.repeat(np.where(E == directp.NO_BLOCK, 0, E), BLOCK, axis=-1) + 7)
    if vis is not None:
        q8 = np.where(vis, q8, 0.0)
        k = np.where(vis, k, 0)
    M = E.max(axis=-1)
    w = np.ldexp(1.0, np.maximum(E - M[:, None] - 7, -2000))      # 2**(E_B - M_i - 7)
    R = len(rows)
    D = (w * q8.reshape(R, N // BLOCK, BLOCK).sum(axis=-1)).sum(axis=-1)
    O = (q8 * np.repeat(w, BLOCK, axis=-1)) @ v / D[:, None]
    out = {"E": E, "M": M, "D": D, "O": O, "LSE": M * directp.LN_2 + np.log(D)}
    if want_codes:
        out["codes"] = k
    return out
