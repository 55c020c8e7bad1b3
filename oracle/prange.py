"""Probability-format range diagnostic of Table p-range (test infrastructure).

The paper's Table p-range (Sec. "Problem 2") forms exact Gaussian softmax
probabilities, quantizes them in 32-key blocks, renormalises the represented P
row by row, multiplies by the same V, and reports per format: the fraction of
blocks whose scale encodes as zero, the fraction of zero payloads, the exact
probability mass mapped to zero (mean per row), the relative L2 error of P, and
the cosine and relative L2 error of PV.

Formats:

* NVFP4 with global encode factor G (eq. nv-scale): block scale
  ``s = Q_E4M3(G a_B / 6) / G`` and codes ``Q_E2M1(p / s)``; a zero scale drops
  the whole block.
* MXFP4: the E8M0 amplitude and codes of :mod:`oracle.mxfp4`, applied to P.

Reproducing the paper's MXFP4 row pins the amplitude rule of the input
quantizer, which the paper states only as a choice between two candidates.
"""
import numpy as np

from . import e2m1, mxfp4

BLOCK = 32


def _e4m3_table():
    """All non-negative finite E4M3 values in code order (bias 7, max 448, no infinities)."""
    vals = []
    for code in range(0x7F):  # 0x7F is NaN
        e, m = code >> 3, code & 7
        vals.append(np.ldexp(m / 8.0, -6) if e == 0 else np.ldexp(1.0 + m / 8.0, e - 7))
    return np.array(vals)


E4M3 = _e4m3_table()


def round_e4m3(x):
    """Nearest E4M3 value to ``x >= 0``, ties to the even code, saturating at 448."""
    x = np.asarray(x, dtype=np.float64)
    hi = np.clip(np.searchsorted(E4M3, x, side="left"), 1, len(E4M3) - 1)
    lo = hi - 1
    d_lo = x - E4M3[lo]
    d_hi = E4M3[hi] - x
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    out = np.where(pick_hi, E4M3[hi], E4M3[lo])
    return np.where(x >= E4M3[-1], E4M3[-1], out)


def quantize_p_nvfp4(p, G):
    """Represented P and per-block zero-scale mask under NVFP4 with global factor G."""
    R, N = p.shape
    blocks = p.reshape(R, N // BLOCK, BLOCK)
    a = blocks.max(axis=-1)
    s = round_e4m3(G * a / 6.0) / G
    zero = s == 0
    r = np.where(zero[..., None], 0.0, blocks / np.where(zero, 1.0, s)[..., None])
    q = e2m1.round_value(r)
    return (q * s[..., None]).reshape(R, N), zero


def quantize_p_mxfp4(p):
    """Represented P and per-block zero-scale mask under MXFP4 (oracle.mxfp4 rule)."""
    codes, scales = mxfp4.quantize(p, axis=-1)
    return mxfp4.dequantize(codes, scales), scales == 0


def diagnose(z, v, fmt, G=None):
    """Table p-range metrics for scores ``z`` [R, N] and values ``v`` [N, d].

    ``fmt`` is "nvfp4" (needs G) or "mxfp4".  Returns a dict with keys
    zero_scales, zero_payload, lost_mass, p_rel_l2, pv_cos, pv_rel_l2.
    """
    z = np.asarray(z, dtype=np.float64)
    p = np.exp(z - z.max(axis=-1, keepdims=True))
    p /= p.sum(axis=-1, keepdims=True)
    if fmt == "nvfp4":
        pt, zero = quantize_p_nvfp4(p, G)
    elif fmt == "mxfp4":
        pt, zero = quantize_p_mxfp4(p)
    else:
        raise ValueError(fmt)
    lost = np.where(pt == 0, p, 0.0).sum(axis=-1).mean()
    row = pt.sum(axis=-1, keepdims=True)
    pn = np.where(row > 0, pt / np.where(row > 0, row, 1.0), 0.0)
    o_ref = p @ v
    o = pn @ v
    return {
        "zero_scales": float(zero.mean()),
        "zero_payload": float((pt == 0).mean()),
        "lost_mass": float(lost),
        "p_rel_l2": float(np.linalg.norm(pn - p) / np.linalg.norm(p)),
        "pv_cos": float((o * o_ref).sum() / (np.linalg.norm(o) * np.linalg.norm(o_ref))),
        "pv_rel_l2": float(np.linalg.norm(o - o_ref) / np.linalg.norm(o_ref)),
    }
