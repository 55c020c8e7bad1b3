"""Pins of the sampled-guard oracle (oracle/guard.py, Alg. 3): reductions to the
unguarded route, the cancellation of the stored-scale shift, the no-amplification
property of the floored working byte, range robustness, and plausibility."""
import numpy as np
import pytest

from oracle import directp, exact, guard, mxfp4

S128 = 1 / np.sqrt(128)


def _head(seed, N=512, d=128, scale_q=1.0, permute=True):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((N, d)) * scale_q
    k = rng.standard_normal((N, d))
    v = rng.standard_normal((N, d))
    if permute:
        perm = guard.anchor_permutation(N)
        k, v = k[perm], v[perm]
    ops = mxfp4.quantize(q) + mxfp4.quantize(k) + mxfp4.quantize(v, axis=-2)
    return (q, k, v), ops


def _raw(ops, rows):
    q6 = mxfp4.scaled_operand(*ops[0:2])[rows]
    k6 = mxfp4.scaled_operand(*ops[2:4])
    return directp.raw_scores(q6, k6)


def test_anchor_permutation_is_a_permutation_with_spread_anchors():
    for N in (128, 1024, 4096):
        p = guard.anchor_permutation(N)
        assert np.array_equal(np.sort(p), np.arange(N))
        assert np.array_equal(p[:128], np.arange(128) * (N // 128))
        assert np.all(np.diff(p[128:]) > 0)
    with pytest.raises(ValueError):
        guard.anchor_permutation(1000)


def test_permutation_leaves_exact_attention_unchanged():
    rng = np.random.default_rng(1)
    q, k, v = (rng.standard_normal((256, 64)) for _ in range(3))
    p = guard.anchor_permutation(256)
    assert np.allclose(exact.attention(q, k, v, 0.125), exact.attention(q, k[p], v[p], 0.125), atol=1e-13)


@pytest.mark.parametrize("ex2_pairs", [0, 4])
def test_integer_reference_reduces_to_the_unguarded_codes(ex2_pairs):
    """With an integral reference R and no floor or saturation in play, x = y - R - e_B
    + log2 6 is the unguarded route's x with E_B = R + e_B: identical codes."""
    _, ops = _head(2)
    raw = _raw(ops, np.arange(64))
    E, _, k_ref = directp.block_exponents_and_codes(raw, S128, 1.5, 1.2, ex2_pairs=ex2_pairs)
    R = E.max(axis=-1).astype(np.float64) + 3.0
    e, ubar, upub, _, k = guard.block_bytes_and_codes(raw, R, S128, 1.5, 1.2, shift=0, ex2_pairs=ex2_pairs)
    assert np.all(ubar > 1) and np.all(ubar < 254)
    assert np.array_equal(e, E - R[:, None].astype(np.int64))
    assert np.array_equal(k, k_ref)
    assert np.array_equal(upub, ubar)


def test_codes_invariant_under_integer_shift_of_the_reference():
    _, ops = _head(3)
    raw = _raw(ops, np.arange(32))
    R = guard.anchor_reference(raw[:, :128], S128, margin=20)
    e0, _, _, _, k0 = guard.block_bytes_and_codes(raw, R, S128, 1.5, 1.2, shift=4)
    e1, _, _, _, k1 = guard.block_bytes_and_codes(raw, R + 7.0, S128, 1.5, 1.2, shift=4)
    assert np.array_equal(k0, k1) and np.array_equal(e0 - 7, e1)


def test_stored_scale_shift_cancels():
    """The common 2**-L of numerator and denominator cancels (Alg. 3, last
    paragraph of Sec. "Fix 3"): when no block meets the floor, O does not depend on L."""
    _, ops = _head(4)
    rows = np.arange(0, 512, 3)
    ref = guard.forward_rows(*ops, rows, S128, margin=10, shift=0)
    assert np.all(ref["ebar"] + 127 > 40)
    for L in (8, 24, 39):
        res = guard.forward_rows(*ops, rows, S128, margin=10, shift=L)
        assert np.array_equal(res["codes"], ref["codes"])
        assert np.array_equal(res["upub"].astype(int), ref["upub"].astype(int) - L)
        assert np.allclose(res["O"], ref["O"], rtol=1e-13, atol=1e-15)


def test_floored_blocks_are_never_amplified():
    """Flooring the working byte before forming x and q (Alg. 3 step 3) keeps every
    represented probability within the E2M1 rounding of the exact one; flooring
    only the published byte would amplify blocks below the floor by
    2**(L + 1 - u_B) (the warning after Alg. 3).  Exponential codes (ex2_pairs = 16)
    make the bound exact: p_rep <= 2 p."""
    _, ops = _head(5, scale_q=4.0)
    rows = np.arange(64)
    raw = _raw(ops, rows)
    M, L = 30, 90
    R = guard.anchor_reference(raw[:, :128], S128, M)
    e, ubar, upub, q, _ = guard.block_bytes_and_codes(raw, R, S128, 1.5, 1.2, L, ex2_pairs=16)
    u = np.clip(e + 127, 0, 254)
    assert np.any(u <= L - 3), "the input must put some blocks well below the floor"
    c_y, _, _ = directp.fp32_coefficients(S128, 1.5, 1.2)
    y = raw * np.float64(c_y)
    p_exact = np.exp2(y - R[:, None] - L)                                  # in units of 2**-L, like upub
    p_rep = np.repeat(np.ldexp(1.0, upub.astype(np.int64) - 127), 32, axis=-1) * q / 6
    assert np.all(p_rep <= 2 * p_exact * (1 + 1e-6))
    # the wrong order (codes from the unfloored exponent, only the published byte
    # floored) breaks the bound on the blocks below the floor
    from oracle import e2m1
    e_rep = np.repeat(np.clip(e, -127, 127), 32, axis=-1)
    q_wrong = e2m1.MAGNITUDES[e2m1.round_index(np.exp2(y - R[:, None] - e_rep + directp.LOG2_6))]
    p_wrong = np.repeat(np.ldexp(1.0, np.maximum(u - L, 1) - 127), 32, axis=-1) * q_wrong / 6
    assert np.any(p_wrong > 4 * p_exact)


def test_margin_and_shift_budget():
    for M, L in ((110, 16), (112, 14), (0, 0), (126, 0)):
        guard.check_margin_shift(M, L)
    for M, L in ((110, 17), (-1, 0), (1.5, 0)):
        with pytest.raises(ValueError):
            guard.check_margin_shift(M, L)


def test_extreme_logits_stay_finite():
    """Rows spanning thousands of binades (the Wan layers' logits above 500)
    stay finite; keys above the anchor saturate the byte at 254 instead of overflowing."""
    rng = np.random.default_rng(6)
    N, d = 256, 64
    q = rng.standard_normal((8, d)) * 60
    k = rng.standard_normal((N, d)) * 4
    v = rng.standard_normal((N, d))
    perm = guard.anchor_permutation(N)
    ops = mxfp4.quantize(q) + mxfp4.quantize(k[perm]) + mxfp4.quantize(v[perm], axis=-2)
    res = guard.forward_rows(*ops, np.arange(8), 0.125, margin=110, shift=16)
    assert np.all(np.isfinite(res["O"])) and np.all(res["D"] > 0)
    assert res["upub"].max() <= 254 - 16 and res["upub"].min() >= 1


@pytest.mark.parametrize("M,L,scale_q", [(8, 0, 1.0), (20, 16, 1.0), (110, 16, 8.0), (112, 14, 8.0)])
def test_plausibility_against_exact_attention(M, L, scale_q):
    """The anchor (the largest of 128 spread scores) sits near the row maximum, so
    with a small margin the guarded operator's error equals the unguarded one's.
    The Wan settings (M, L) = (110, 16) and (112, 14) put the anchor's binade on
    the floor, which costs nothing on the peaked rows they serve (logits 8x
    wider here) ..."""
    (q, k, v), ops = _head(7, N=1024, scale_q=scale_q)
    rows = np.arange(0, 1024, 2)
    ref = exact.attention(q[rows], k, v, S128)
    plain = directp.forward_rows(*ops, rows, S128, want_codes=False)
    guarded = guard.forward_rows(*ops, rows, S128, margin=M, shift=L, want_codes=False)
    rel_plain = exact.error_metrics(plain["O"], ref)[1]
    rel_guard = exact.error_metrics(guarded["O"], ref)[1]
    assert abs(rel_guard / rel_plain - 1) < 0.05, (rel_plain, rel_guard)


def test_wan_margin_floors_sub_anchor_blocks_on_flat_rows():
    """... while on flat Gaussian rows every block below the anchor's binade is
    represented with the anchor's amplitude (Alg. 3 step 3 with M + L = 126), so
    the error grows well past the unguarded route's."""
    (q, k, v), ops = _head(7, N=1024)
    rows = np.arange(0, 1024, 2)
    ref = exact.attention(q[rows], k, v, S128)
    plain = exact.error_metrics(directp.forward_rows(*ops, rows, S128, want_codes=False)["O"], ref)[1]
    res = guard.forward_rows(*ops, rows, S128, margin=110, shift=16, want_codes=False)
    assert np.all(res["ebar"] >= -110)
    assert exact.error_metrics(res["O"], ref)[1] > 1.5 * plain


def test_lse_matches_the_online_route_under_an_integral_reference():
    """With an integral reference and no floor in play the guarded operator is the
    online one (same codes, bytes shifted by R - M + L), so its normaliser
    (R + L) ln 2 + ln(D / 6) equals the online M ln 2 + ln(D / 6)."""
    _, ops = _head(8)
    rows = np.arange(0, 512, 5)
    online = directp.forward_rows(*ops, rows, S128)
    R = online["M"].astype(np.float64) + 3.0
    res = guard.forward_rows(*ops, rows, S128, margin=0, shift=9, reference=R)
    assert np.all(res["ebar"] + 127 > 10)
    assert np.array_equal(res["codes"], online["codes"])
    assert np.allclose(res["LSE"], online["LSE"], rtol=0, atol=1e-12)
    assert np.allclose(res["O"], online["O"], rtol=1e-13, atol=1e-15)
