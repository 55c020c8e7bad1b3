"""Sampled QK guard for extreme logits (test infrastructure; see oracle/__init__).

What is computed, following Sec. "Fix 3: guard only extreme model logits" and
Alg. 3 (sampled-guard) on top of Alg. 2:

1. Anchor keys.  Before the launch, ``n_anchor`` = 128 globally distributed K/V
   rows are moved into the first key tile; the permutation leaves exact
   attention unchanged.  Reading of "globally distributed": the evenly spaced
   rows ``j * N / n_anchor`` (j = 0 .. n_anchor - 1) in order, then every other
   row in its original order (:func:`anchor_permutation`).  V is quantized
   after the permutation, so its 32-key blocks follow the new key order.
2. Anchor and reference (Alg. 3, steps 1-2): ``a_i`` is the largest score of
   row i over the anchor keys and ``m_i = a_i + M ln 2``.  In the base-2 units
   of the fp32 decision path (``y = fp32(raw * c_y)``, ``c_y = fp32(s log2(e) / 36)``
   as in :mod:`oracle.directp`) the reference is ``R_i = fp32(Y_i + M)`` with
   ``Y_i = max_{j in anchors} y_ij``.
3. Block bytes (Alg. 2 step 2 with reference m_i; Alg. 3 step 3): the block
   exponent ``e_B = floor(fp32(Y_B - R_i))`` with ``Y_B = max_{j in B} y_ij``,
   the byte ``u_B = clamp(e_B + 127, 0, 254)``, the floored working byte
   ``ubar_B = max(u_B, L + 1)`` and ``ebar_B = ubar_B - 127``.  The codes are
   Alg. 2's with ``x = y - R_i - ebar_B + log2 6``, in fp32 like the unguarded
   route: ``T = fp32(R_i + ebar_B)``, affine ``u = fma(c_a, raw, fp32(k0 - A T))``
   and, for native-exponential pairs, ``x = fma(c_y, raw, fp32(k1 - T))``.
   The published byte is ``u'_B = ubar_B - L``.
4. Denominator (Alg. 3, steps 4-5): ``alpha'_B = 2**(u'_B - 127)`` and
   ``D_i = sum_B alpha'_B c_B`` with ``c_B = sum_j q_ij``.  The paper evaluates
   ``alpha'_B (c_B / 6)``; the 1/6 of the represented probability cancels
   against the numerator's, so it is left out here (as in the unguarded route),
   and no quantity formed here can be subnormal for ``u'_B >= 1``.
5. Output (eq. represented-output): ``O_i = sum_B alpha'_B sum_j q_ij (6 Vhat_j) / (6 D_i)``.
   The common ``2**-L`` of numerator and denominator cancels.  The saved row
   normaliser (natural log) is ``LSE_i = (R_i + L) ln 2 + ln(D_i / 6)``: the
   represented ``exp(z_ij)`` is ``2**(R_i + ebar_B) q_ij / 6``.

The margin ``M`` and shift ``L`` are integers with ``M + L <= 126`` (Alg. 3,
step 2), so a block at the anchor publishes a byte of at least 1.
"""
import numpy as np

from . import directp, e2m1, fp32, mxfp4

BLOCK = directp.BLOCK
N_ANCHOR = 128


def anchor_permutation(N, n_anchor=N_ANCHOR):
    """Key order with the anchor rows first: ``permuted[r] = original[perm[r]]``."""
    if N % n_anchor:
        raise ValueError("N must be a multiple of the anchor count")
    stride = N // n_anchor
    anchors = np.arange(n_anchor) * stride
    rest = np.setdiff1d(np.arange(N), anchors)
    return np.concatenate([anchors, rest])


def check_margin_shift(margin, shift):
    if int(margin) != margin or int(shift) != shift or margin < 0 or shift < 0 or margin + shift > 126:
        raise ValueError("margin M and shift L must be non-negative integers with M + L <= 126")


def anchor_reference(raw_anchor, softmax_scale, margin):
    """R_i = fp32(max_{j in anchors} fp32(raw_ij c_y) + M) for the [R, n_anchor] anchor scores."""
    c_y, _, _ = directp.fp32_coefficients(softmax_scale, 1.5, 1.2)
    y = fp32.mul(np.asarray(raw_anchor).astype(np.float32), c_y)
    Y = y.max(axis=-1)
    return fp32.fma(np.float32(1.0), Y, np.float32(margin))


def block_bytes_and_codes(raw, R, softmax_scale, affine_a, affine_b, shift, ex2_pairs=0):
    """Steps 3 of the module docstring for [R, N] scores and fp32 references R [R].

    Returns (e [R, N/32] unclamped block exponents, ubar [R, N/32] working bytes,
    upub [R, N/32] published bytes, q [R, N] code magnitudes, k [R, N] code indices).
    """
    Rn, N = raw.shape
    nb = N // BLOCK
    c_y, c_a, k0 = directp.fp32_coefficients(softmax_scale, affine_a, affine_b)
    raw32 = raw.astype(np.float32)
    y = fp32.mul(raw32, c_y)
    Y_B = y.reshape(Rn, nb, BLOCK).max(axis=-1)
    R32 = np.asarray(R, dtype=np.float32)[:, None]
    e = np.floor(fp32.fma(np.float32(-1.0), R32, Y_B).astype(np.float64)).astype(np.int64)  # fp32(Y_B - R)
    u = np.clip(e + 127, 0, 254)
    ubar = np.maximum(u, shift + 1)
    ebar = ubar - 127
    T = fp32.fma(np.float32(1.0), R32, ebar.astype(np.float32))                               # fp32(R + ebar)
    a32 = np.float32(affine_a)
    c0 = fp32.fma(-a32, T, k0)
    uhat = fp32.fma(c_a, raw32, np.repeat(c0, BLOCK, axis=-1)).astype(np.float64)
    k = e2m1.round_index(np.maximum(uhat, 0.0))
    mask = directp.ex2_key_mask(ex2_pairs)
    if ex2_pairs:
        c1 = fp32.fma(np.float32(-1.0), T, np.float32(directp.LOG2_6))                        # fp32(k1 - T)
        x = fp32.fma(c_y, raw32, np.repeat(c1, BLOCK, axis=-1))
        p = np.exp2(x.astype(np.float64)).astype(np.float32).astype(np.float64)
        k = np.where(np.tile(mask, nb)[None, :], e2m1.round_index(p), k)
    return e, ubar, ubar - shift, e2m1.MAGNITUDES[k], k


def forward_rows(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, rows, softmax_scale,
                 margin, shift, affine_a=1.5, affine_b=1.2, ex2_pairs=0, n_anchor=N_ANCHOR, want_codes=True,
                 reference=None):
    """Guarded Direct-P forward for the query ``rows`` of ONE (batch, head) slice
    whose K and V are already in anchor order (the first ``n_anchor`` keys are
    the anchors).  Operands as :func:`oracle.directp.forward_rows`.

    Returns a dict: ``R`` [R] fp32 references, ``e``/``ebar`` [R, N/32] block and
    working exponents, ``upub`` [R, N/32] published bytes, ``D`` [R]
    (``sum_B 2**(u'_B - 127) c_B``), ``O`` [R, d], ``LSE`` [R], and ``codes`` [R, N].
    ``reference`` replaces the anchor-derived R_i (used by tests).
    """
    check_margin_shift(margin, shift)
    rows = np.asarray(rows, dtype=np.int64)
    q6 = mxfp4.scaled_operand(q_codes, q_scales)[rows]
    k6 = mxfp4.scaled_operand(k_codes, k_scales)
    v6 = mxfp4.scaled_operand(vt_codes, vt_scales).T
    N = k6.shape[0]
    if N < n_anchor:
        raise ValueError("fewer keys than anchors")
    raw = directp.raw_scores(q6, k6)
    R = anchor_reference(raw[:, :n_anchor], softmax_scale, margin) if reference is None else \
        np.asarray(reference, dtype=np.float64)
    e, ubar, upub, q, k = block_bytes_and_codes(raw, R, softmax_scale, affine_a, affine_b, shift, ex2_pairs)
    w = np.ldexp(1.0, upub.astype(np.int64) - 127)                        # alpha'_B
    nb = N // BLOCK
    D = (w * q.reshape(len(rows), nb, BLOCK).sum(axis=-1)).sum(axis=-1)   # sum_B alpha'_B c_B
    acc = (q * np.repeat(w, BLOCK, axis=-1)) @ v6
    out = {"R": R.astype(np.float64), "e": e, "ebar": ubar - 127, "upub": upub, "D": D,
           "O": acc / (6.0 * D[:, None]),
           "LSE": (R.astype(np.float64) + shift) * directp.LN_2 + np.log(D) - directp.LN_6}
    if want_codes:
        out["codes"] = k
    return out
