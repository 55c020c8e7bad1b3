"""Direct-P full-MXFP4 attention forward (test infrastructure; see oracle/__init__).

What is computed, in the paper's order (Sec. "Direct-P: Fixing the FP4
Probability Path"; Alg. 2; eqs. ideal-code-path, affine-code-map,
represented-contributions, represented-output):

1. Scores.  Q and K are MXFP4 operands.  A block-scaled FP4 matrix unit
   multiplies ``2**(u-127) * q`` (six times the represented value), so the
   product it accumulates is ``raw = 36 * Qhat Khat^T``; the paper's 1/36
   correction (Sec. "Problem 2", after eq. mx-scale) and the softmax scale s
   are folded into the score transform: ``y = z * log2(e) = raw * s*log2(e)/36``.
2. Per row i and 32-key block B (keys 32b .. 32b+31): the block exponent
   ``E_B = floor(max_{j in B} y_ij)``, the exponent of the block maximum of
   ``2**y`` (Alg. 2, steps 1-2).
3. Code map (Alg. 2, steps 3-4): ``x = y - E_B + log2(6)`` and
   ``q = Q_E2M1(max(0, A x + B))`` (eq. affine-code-map; A = 1.5, B = 1.2 for
   the ``fast`` fit).  The paper folds the score transform, ``E_B`` and
   ``log2 6`` into the coefficients of one fp32 fused multiply-add per score;
   the default mode ``affine32`` takes exactly that fp32 decision:
   ``u = fma(c_a, raw, c0_B)`` with ``c_a = fp32(A s log2(e) / 36)`` and
   ``c0_B = fp32(A (log2 6 - E_B) + B)`` evaluated as one rounding of
   ``k0 - A E_B`` with ``k0 = fp32(A log2 6 + B)``; the block maximum is
   ``fp32(raw * c_y)`` with ``c_y = fp32(s log2(e) / 36)``.
   Other modes: ``affine64`` (the same map unfused in fp64), ``exp2`` (the ideal
   converter ``Q_E2M1(2**x)``, eq. ideal-code-path) and ``exp2_exact``
   (``2**x`` with no E2M1 rounding, used to check the normalisation).
   Native-exponential mixing (Sec. "Fix 1": a selected pair may use the
   native exponential; the balancing paragraph closing Sec. "Fix 2"; Table
   policy-definition, ``accurate``; Table b300-tuning, EX2 density): with
   ``ex2_pairs = k`` in {1, 2, 4, 8, 16}, pair p of each 32-key block (keys 2p
   and 2p + 1, p = 0..15) takes the ideal converter instead of the affine map
   when ``p % (16 / k) == 0``, i.e. k of the 16 pairs, evenly spaced.  Its fp32
   decision folds the transform into one fma like the affine map:
   ``x = fma(c_y, raw, c1_B)`` with ``c1_B = fp32(k1 - E_B)``,
   ``k1 = fp32(log2 6)``, then ``q = Q_E2M1(fp32(2**x))``.
4. Row reference: the paper's fast path is shiftless (m_i = 0).  Codes do not
   depend on the reference, so this oracle uses the integer reference
   ``M_i = max_B E_B`` and weights ``w_B = 2**(E_B - M_i)``; the E8M0 byte
   published for P is ``u_B = E_B - M_i + 127`` (``u_B = 0`` marks a block
   below the E8M0 range, whose weight is under 2**-126 of the row maximum).
5. Represented denominator (Fix 2, eq. represented-contributions):
   ``c_B = sum_{j in B} q_ij`` from the same codes PV consumes, and
   ``D_i = sum_B w_B c_B``.  No 1/6 appears: the P-side 1/6 cancels between
   numerator and denominator.
6. Output (eq. represented-output): ``O_i = sum_B w_B sum_j q_ij Vhat_j / D_i``
   in fp64, with ``Vhat`` the represented MXFP4 value of V (blocks of 32 keys).

Causal form (the forward of the paper's causal-training route, Sec. "Pass the
forward quantization into backward"): query i sees keys j <= i only.  Masked
scores are -inf: they take code 0, a block with no visible key has no block
exponent (weight 0), and ``M_i`` is the largest exponent over visible blocks.
The saved row normaliser is the natural-log log-sum-exp of the represented
operator, ``LSE_i = M_i ln 2 + ln(D_i / 6)``: with ``2**E_B q_ij / 6`` standing
for ``exp(z_ij)``, ``exp(z_ij - LSE_i)`` is the represented probability
``w_B q_ij / D_i`` that the backward reconstructs.

The online (tiled) form keeps a running integer reference and rescales by
exact powers of two (eq. online-recurrence with ``e**(m - m')`` replaced by
``2**(M - M')``); it gives the same codes and, up to fp64 rounding, the same
output for any tile width.
"""
import numpy as np

from . import e2m1, fp32, mxfp4

# Mathematical constants correctly rounded to fp64.
LOG2_E = 1.4426950408889634
LOG2_6 = 2.584962500721156

BLOCK = 32
MODES = ("affine32", "affine64", "exp2", "exp2_exact")
NO_BLOCK = -(1 << 40)   # block exponent of a block with no visible key (causal mask)
LN_2 = 0.6931471805599453
LN_6 = 1.791759469228055
EX2_PAIRS = (0, 1, 2, 4, 8, 16)


def ex2_key_mask(ex2_pairs):
    """[32] bool: the keys of a 32-key block whose code comes from ``2**x``
    (pair p = key // 2 is selected iff p % (16 / ex2_pairs) == 0)."""
    if ex2_pairs not in EX2_PAIRS:
        raise ValueError(f"ex2_pairs must be one of {EX2_PAIRS}")
    if ex2_pairs == 0:
        return np.zeros(BLOCK, dtype=bool)
    return (np.arange(BLOCK) // 2) % (16 // ex2_pairs) == 0


def fp32_coefficients(softmax_scale, affine_a, affine_b):
    """(c_y, c_a, k0) as fp32 (see step 3 of the module docstring)."""
    s = float(np.float32(softmax_scale))
    a = float(np.float32(affine_a))
    b = float(np.float32(affine_b))
    c_y = np.float32(s * LOG2_E / 36.0)
    c_a = np.float32(a * s * LOG2_E / 36.0)
    k0 = np.float32(a * LOG2_6 + b)
    return c_y, c_a, k0


def raw_scores(q6, k6):
    """``raw = (6 Qhat)(6 Khat)^T`` in fp64.

    Every product of two scaled E2M1 values is exact, and for the block scales
    met in practice every partial sum is exact too; the result is checked to be
    exactly representable in fp32 (the precision of the matrix-unit accumulator),
    and a ValueError is raised otherwise.
    """
    raw = q6 @ k6.T
    if not np.array_equal(raw.astype(np.float32).astype(np.float64), raw, equal_nan=True):
        raise ValueError("raw scores are not exactly representable in fp32")
    return raw


def block_exponents_and_codes(raw, softmax_scale, affine_a, affine_b, mode="affine32", ex2_pairs=0,
                              visible=None):
    """(E [R, N/32] int64, q [R, N] fp64 magnitudes, k [R, N] uint8 code indices or None).

    ``raw`` is the [R, N] score matrix of step 1.  For ``exp2_exact`` the
    returned ``q`` holds the unrounded ``2**x`` and ``k`` is None.
    ``ex2_pairs`` (mode ``affine32`` only) selects native-exponential mixing.
    ``visible`` ([R, N] bool, causal mask): hidden scores get code 0 and a block
    without visible keys gets ``E = NO_BLOCK``.
    """
    if visible is not None:
        E, q, k = block_exponents_and_codes(np.where(visible, raw, -np.inf), softmax_scale, affine_a, affine_b,
                                            mode, ex2_pairs)
        return E, np.where(visible, q, 0.0), (None if k is None else np.where(visible, k, 0).astype(np.uint8))
    if mode not in MODES:
        raise ValueError(f"mode must be one of {MODES}")
    mask = ex2_key_mask(ex2_pairs)
    if ex2_pairs and mode != "affine32":
        raise ValueError("ex2_pairs applies to the fp32 decision (mode affine32)")
    R, N = raw.shape
    if N % BLOCK:
        raise ValueError("key count must be a multiple of 32")
    nb = N // BLOCK
    if mode == "affine32":
        c_y, c_a, k0 = fp32_coefficients(softmax_scale, affine_a, affine_b)
        raw32 = raw.astype(np.float32)
        y = fp32.mul(raw32, c_y)
        E = _floor_exponent(y.reshape(R, nb, BLOCK).max(axis=-1).astype(np.float64))
        a32 = np.float32(affine_a)
        c0 = fp32.fma(-a32, _finite(E).astype(np.float32), k0)
        u = fp32.fma(c_a, raw32, np.repeat(c0, BLOCK, axis=-1)).astype(np.float64)
        k = e2m1.round_index(np.maximum(u, 0.0))
        if ex2_pairs:
            k1 = np.float32(LOG2_6)
            c1 = fp32.fma(np.float32(-1.0), _finite(E).astype(np.float32), k1)  # fp32(k1 - E_B)
            x = fp32.fma(c_y, raw32, np.repeat(c1, BLOCK, axis=-1))
            p = np.exp2(x.astype(np.float64)).astype(np.float32).astype(np.float64)
            keys = np.tile(mask, nb)
            k = np.where(keys[None, :], e2m1.round_index(p), k)
        return E, e2m1.MAGNITUDES[k], k
    # fp64 modes follow eq. ideal-code-path / affine-code-map literally.
    s = float(np.float32(softmax_scale))
    y = raw * (s / 36.0) * LOG2_E
    E = _floor_exponent(y.reshape(R, nb, BLOCK).max(axis=-1))
    x = y - np.repeat(_finite(E), BLOCK, axis=-1) + LOG2_6
    if mode == "affine64":
        a = float(np.float32(affine_a))
        b = float(np.float32(affine_b))
        k = e2m1.round_index(np.maximum(a * x + b, 0.0))
        return E, e2m1.MAGNITUDES[k], k
    p = np.exp2(x)
    if mode == "exp2":
        k = e2m1.round_index(p)
        return E, e2m1.MAGNITUDES[k], k
    return E, p, None


def _floor_exponent(ymax):
    """floor of the block maxima; NO_BLOCK where a block has no finite score."""
    with np.errstate(invalid="ignore"):
        return np.where(np.isfinite(ymax), np.floor(np.nan_to_num(ymax, neginf=0.0)), NO_BLOCK).astype(np.int64)


def _finite(E):
    """Block exponents with NO_BLOCK replaced by 0 (the codes of such blocks are all 0 anyway)."""
    return np.where(E == NO_BLOCK, 0, E)


def lse(M, D):
    """Natural-log row normaliser of the represented operator: M ln 2 + ln(D / 6)."""
    return np.asarray(M, dtype=np.float64) * LN_2 + np.log(np.asarray(D, dtype=np.float64)) - LN_6


def _normalise(E, q, v6, M):
    """Steps 4-6 for one row chunk: (D relative to 2**M, O)."""
    R, N = q.shape
    nb = N // BLOCK
    w = np.ldexp(1.0, np.maximum(E - M[:, None], -2000))    # 2**(E_B - M_i), exact (0 for NO_BLOCK)
    c = q.reshape(R, nb, BLOCK).sum(axis=-1)                 # c_B = sum_j q_ij
    D = (w * c).sum(axis=-1)                                 # represented denominator
    acc = (q * np.repeat(w, BLOCK, axis=-1)) @ v6            # sum_B w_B sum_j q_ij (6 Vhat_j)
    O = acc / (6.0 * D[:, None])
    return D, O


def forward_rows(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, rows,
                 softmax_scale, affine_a=1.5, affine_b=1.2, mode="affine32",
                 chunk=128, want_codes=True, ex2_pairs=0, causal=False):
    """Direct-P forward for the query ``rows`` of ONE (batch, head) slice.

    Operands are single-head MXFP4 arrays as produced by :func:`oracle.mxfp4.quantize`:
    q/k codes [N, d/2] + scales [N, d/32]; vt codes [d, N/2] + scales [d, N/32].
    Returns a dict with ``E`` [R, N/32] (absolute block exponents), ``M`` [R]
    (integer row reference), ``D`` [R] (denominator relative to 2**M), ``O``
    [R, d] (fp64), ``LSE`` [R] (natural log), and when ``want_codes`` ``codes``
    [R, N] (E2M1 magnitude indices 0..7; for ``exp2_exact`` the unrounded
    values instead).  ``causal``: row ``rows[r]`` sees keys ``j <= rows[r]``.
    """
    rows = np.asarray(rows, dtype=np.int64)
    q6 = mxfp4.scaled_operand(q_codes, q_scales)[rows]
    k6 = mxfp4.scaled_operand(k_codes, k_scales)
    v6 = mxfp4.scaled_operand(vt_codes, vt_scales).T         # [N, d], 6 * Vhat
    out = {"E": [], "M": [], "D": [], "O": [], "LSE": [], "codes": []}
    for lo in range(0, len(rows), chunk):
        raw = raw_scores(q6[lo:lo + chunk], k6)
        vis = (np.arange(raw.shape[1])[None, :] <= rows[lo:lo + chunk, None]) if causal else None
        E, q, k = block_exponents_and_codes(raw, softmax_scale, affine_a, affine_b, mode, ex2_pairs, vis)
        M = E.max(axis=-1)
        D, O = _normalise(E, q, v6, M)
        out["E"].append(E)
        out["M"].append(M)
        out["D"].append(D)
        out["O"].append(O)
        out["LSE"].append(lse(M, D))
        if want_codes:
            out["codes"].append(k if k is not None else q)
    res = {key: np.concatenate(val) for key, val in out.items() if val}
    return res


def forward_rows_online(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, rows,
                        softmax_scale, affine_a=1.5, affine_b=1.2, mode="affine32", tile=128, ex2_pairs=0):
    """Online (tiled) form of :func:`forward_rows`: key tiles of width ``tile``.

    A running integer reference ``M`` starts at the first tile's maximum block
    exponent; when a tile raises it, the accumulated numerator and denominator
    are multiplied by ``2**(M_old - M_new)`` (exact).  Returns the same keys as
    :func:`forward_rows`.
    """
    if tile % BLOCK:
        raise ValueError("tile must be a multiple of 32")
    rows = np.asarray(rows, dtype=np.int64)
    q6 = mxfp4.scaled_operand(q_codes, q_scales)[rows]
    k6 = mxfp4.scaled_operand(k_codes, k_scales)
    v6 = mxfp4.scaled_operand(vt_codes, vt_scales).T
    R, N = len(rows), k6.shape[0]
    M = None
    acc = np.zeros((R, v6.shape[1]))
    D = np.zeros(R)
    Es, codes = [], []
    for t0 in range(0, N, tile):
        raw = raw_scores(q6, k6[t0:t0 + tile])
        E, q, k = block_exponents_and_codes(raw, softmax_scale, affine_a, affine_b, mode, ex2_pairs)
        tile_max = E.max(axis=-1)
        M_new = tile_max if M is None else np.maximum(M, tile_max)
        rescale = np.ones(R) if M is None else np.ldexp(1.0, M - M_new)
        w = np.ldexp(1.0, E - M_new[:, None])
        nb = E.shape[1]
        acc = acc * rescale[:, None] + (q * np.repeat(w, BLOCK, axis=-1)) @ v6[t0:t0 + tile]
        D = D * rescale + (w * q.reshape(R, nb, BLOCK).sum(axis=-1)).sum(axis=-1)
        M = M_new
        Es.append(E)
        codes.append(k if k is not None else q)
    return {"E": np.concatenate(Es, axis=1), "M": M, "D": D,
            "O": acc / (6.0 * D[:, None]), "codes": np.concatenate(codes, axis=1)}


def p_scale_bytes(E, M):
    """E8M0 bytes published for P: ``clamp(E_B - M_i + 127, 0, 254)`` (0 = below range)."""
    return np.clip(np.asarray(E) - np.asarray(M)[:, None] + 127, 0, 254).astype(np.uint8)


def represented_probabilities(E, q, M):
    """Normalised represented probabilities ``w_B q_ij / D_i`` [R, N] (rows sum to 1)."""
    R, N = q.shape
    w = np.repeat(np.ldexp(1.0, np.maximum(np.asarray(E) - np.asarray(M)[:, None], -2000)), BLOCK, axis=-1)
    num = w * q
    return num / num.sum(axis=-1, keepdims=True)


def forward(q, k, v, softmax_scale=None, affine_a=1.5, affine_b=1.2, mode="affine32", rows=None):
    """Quantize unquantized Q, K, V ``[B, H, N, d]`` with :mod:`oracle.mxfp4` and run Direct-P.

    ``rows`` selects flattened (b*H + h)*N + i query rows (default: all).
    Returns (O [R, d], rows).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    Bsz, H, N, d = q.shape
    if softmax_scale is None:
        softmax_scale = 1.0 / np.sqrt(d)
    if rows is None:
        rows = np.arange(Bsz * H * N)
    rows = np.asarray(rows, dtype=np.int64)
    O = np.zeros((len(rows), d))
    heads = rows // N
    for bh in np.unique(heads):
        b, h = divmod(int(bh), H)
        sel = np.nonzero(heads == bh)[0]
        qc, qs = mxfp4.quantize(q[b, h], axis=-1)
        kc, ks = mxfp4.quantize(k[b, h], axis=-1)
        vc, vs = mxfp4.quantize(v[b, h], axis=-2)
        res = forward_rows(qc, qs, kc, ks, vc, vs, rows[sel] % N, softmax_scale,
                           affine_a, affine_b, mode, want_codes=False)
        O[sel] = res["O"]
    return O, rows
