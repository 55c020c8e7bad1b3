"""Pins of the Direct-P oracle (oracle/directp.py): closed forms, invariants,
special cases that reduce to textbook attention, and the paper's error band."""
import os

import numpy as np
import pytest

from oracle import directp, e2m1, exact, mxfp4

SCALE64 = 0.125  # 1/sqrt(64)


def _golden(golden_dir, name, key):
    with open(os.path.join(golden_dir, name)) as f:
        for line in f:
            if line.startswith(key + " "):
                return [float(t) for t in line.split()[1:]]
    raise KeyError(key)


def _quantized_head(rng, N, d, scale_q=1.0):
    q = rng.standard_normal((N, d)) * scale_q
    k = rng.standard_normal((N, d))
    v = rng.standard_normal((N, d))
    ops = mxfp4.quantize(q) + mxfp4.quantize(k) + mxfp4.quantize(v, axis=-2)
    return (q, k, v), ops


def _raw_for_x(xs, softmax_scale, mode):
    """A 32-score block whose maximum has y = 0.5 (E_B = 0) and whose other scores
    have x = y - E_B + log2 6 equal to ``xs``."""
    y = np.concatenate([[0.5], np.asarray(xs) - directp.LOG2_6])
    raw = y / (softmax_scale / 36.0 * directp.LOG2_E)
    if mode == "affine32":
        c_y, _, _ = directp.fp32_coefficients(softmax_scale, 1.5, 1.2)
        raw = (y / np.float64(c_y)).astype(np.float32).astype(np.float64)
    return np.pad(raw, (0, 32 - len(raw)), constant_values=raw[1])[None, :]


@pytest.mark.parametrize("mode,eps", [("affine64", 1e-9), ("affine32", 1e-4)])
@pytest.mark.parametrize("ab_key", ["fast_affine", "wan_affine"])
def test_code_boundaries_closed_form(golden_dir, mode, eps, ab_key):
    """Codes change exactly at x_j = (t_j - B) / A (eq. affine-log-boundaries)."""
    A, B = _golden(golden_dir, "e2m1.txt", ab_key)
    t = _golden(golden_dir, "e2m1.txt", "boundaries")
    # A and B travel as fp32 arguments; the boundaries follow the rounded values
    xj = (np.array(t) - float(np.float32(B))) / float(np.float32(A))
    for j, x in enumerate(xj):
        raw = _raw_for_x([x - eps, x + eps], SCALE64, mode)
        E, _, k = directp.block_exponents_and_codes(raw, SCALE64, A, B, mode)
        assert E[0, 0] == 0
        assert k[0, 1] == j and k[0, 2] == j + 1, (j, x, k[0, :3])
    if ab_key == "fast_affine":
        # the printed (A, B) = (1.5, 1.2) give these boundaries
        assert np.allclose(xj, [-0.63333, -0.3, 0.03333, 0.36667, 0.86667, 1.53333, 2.53333], atol=1e-5)


@pytest.mark.parametrize("mode", ["affine32", "affine64", "exp2"])
def test_block_argmax_gets_code_six(mode):
    rng = np.random.default_rng(10)
    raw = (rng.standard_normal((64, 256)) * 300).astype(np.float32).astype(np.float64)
    E, q, k = directp.block_exponents_and_codes(raw, SCALE64, 1.5, 1.2, mode)
    blocks = k.reshape(64, 8, 32)
    arg = raw.reshape(64, 8, 32).argmax(axis=-1)
    assert np.all(np.take_along_axis(blocks, arg[..., None], axis=-1) == 7)
    # and every other code is at most that
    assert blocks.max() == 7


@pytest.mark.parametrize("mode", ["affine64", "exp2", "exp2_exact"])
def test_codes_invariant_under_integer_log2_shift(mode):
    rng = np.random.default_rng(11)
    raw = rng.standard_normal((32, 256)) * 200
    per_unit = 36.0 / (SCALE64 * directp.LOG2_E)   # raw increment that moves y by one
    for shift in (-7, 3, 40):
        E0, q0, _ = directp.block_exponents_and_codes(raw, SCALE64, 1.5, 1.2, mode)
        E1, q1, _ = directp.block_exponents_and_codes(raw + shift * per_unit, SCALE64, 1.5, 1.2, mode)
        assert np.array_equal(E1, E0 + shift)
        if mode == "exp2_exact":
            assert np.allclose(q0, q1, rtol=1e-9, atol=0)
        else:
            assert np.array_equal(q0, q1)


def test_fp32_decision_agrees_with_fp64_formula():
    rng = np.random.default_rng(12)
    (_, _, _), ops = _quantized_head(rng, 512, 128)
    q6 = mxfp4.scaled_operand(*ops[0:2])
    k6 = mxfp4.scaled_operand(*ops[2:4])
    raw = directp.raw_scores(q6, k6)
    s = 1 / np.sqrt(128)
    E32, _, k32 = directp.block_exponents_and_codes(raw, s, 1.5, 1.2, "affine32")
    E64, _, k64 = directp.block_exponents_and_codes(raw, s, 1.5, 1.2, "affine64")
    assert np.mean(E32 != E64) < 1e-4
    assert np.mean(k32 != k64) < 1e-4


@pytest.mark.parametrize("mode", ["affine32", "exp2"])
def test_represented_probabilities_sum_to_one(mode):
    rng = np.random.default_rng(13)
    _, ops = _quantized_head(rng, 256, 64, scale_q=3.0)
    res = directp.forward_rows(*ops, np.arange(256), SCALE64, mode=mode)
    p = directp.represented_probabilities(res["E"], e2m1.MAGNITUDES[res["codes"]], res["M"])
    assert np.allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-13)
    # the denominator is the same weighted code sum
    w = np.ldexp(1.0, res["E"] - res["M"][:, None])
    c = e2m1.MAGNITUDES[res["codes"]].reshape(256, -1, 32).sum(axis=-1)
    assert np.allclose(res["D"], (w * c).sum(axis=1), rtol=1e-15)


@pytest.mark.parametrize("tile", [32, 64, 128, 512])
def test_online_equals_whole_row(tile):
    rng = np.random.default_rng(14)
    _, ops = _quantized_head(rng, 512, 64, scale_q=4.0)   # peaked rows: the reference moves
    rows = np.arange(0, 512, 3)
    brute = directp.forward_rows(*ops, rows, SCALE64)
    online = directp.forward_rows_online(*ops, rows, SCALE64, tile=tile)
    assert np.array_equal(brute["codes"], online["codes"])
    assert np.array_equal(brute["E"], online["E"])
    assert np.array_equal(brute["M"], online["M"])
    assert np.allclose(online["O"], brute["O"], rtol=0, atol=1e-12 * np.abs(brute["O"]).max())
    assert np.allclose(online["D"], brute["D"], rtol=1e-13)


def test_zero_queries_give_uniform_p_and_mean_value():
    """Q = 0: y = 0, E_B = 0, u = A log2 6 + B = 5.08 -> every code is 6."""
    rng = np.random.default_rng(15)
    N, d = 256, 64
    v = rng.standard_normal((N, d))
    ops = mxfp4.quantize(np.zeros((N, d))) + mxfp4.quantize(rng.standard_normal((N, d))) \
        + mxfp4.quantize(v, axis=-2)
    res = directp.forward_rows(*ops, np.arange(N), SCALE64)
    assert np.all(res["codes"] == 7) and np.all(res["E"] == 0)
    vhat = mxfp4.dequantize(*ops[4:6]).T
    assert np.allclose(res["O"], vhat.mean(axis=0)[None, :], rtol=0, atol=1e-14)


def test_constant_power_of_two_values_pass_through():
    rng = np.random.default_rng(16)
    N, d = 256, 64
    for k in (-3, 0, 5):
        ops = mxfp4.quantize(rng.standard_normal((N, d)) * 2) + mxfp4.quantize(rng.standard_normal((N, d))) \
            + mxfp4.quantize(np.full((N, d), 2.0 ** k), axis=-2)
        res = directp.forward_rows(*ops, np.arange(N), SCALE64)
        assert np.all(res["O"] == 2.0 ** k)


def test_unrounded_exp2_reduces_to_softmax_attention():
    """Without E2M1 rounding, p = 2**x = 6 * 2**(y - E_B) and the weights
    2**(E_B - M) make the output exactly softmax attention over Qhat, Khat, Vhat."""
    rng = np.random.default_rng(17)
    N, d = 384, 64
    _, ops = _quantized_head(rng, N, d, scale_q=2.0)
    res = directp.forward_rows(*ops, np.arange(N), SCALE64, mode="exp2_exact")
    qh = mxfp4.dequantize(*ops[0:2])
    kh = mxfp4.dequantize(*ops[2:4])
    vh = mxfp4.dequantize(*ops[4:6]).T
    ref = exact.attention(qh, kh, vh, SCALE64)
    assert np.allclose(res["O"], ref, rtol=0, atol=1e-12)


def test_dominant_key_selects_its_value():
    rng = np.random.default_rng(18)
    N, d, jstar = 256, 64, 77
    k = rng.standard_normal((N, d))
    k[jstar] = 4.0
    q = np.full((4, d), 4.0)
    v = rng.standard_normal((N, d))
    ops = mxfp4.quantize(q) + mxfp4.quantize(k) + mxfp4.quantize(v, axis=-2)
    res = directp.forward_rows(*ops, np.arange(4), SCALE64)
    vhat = mxfp4.dequantize(*ops[4:6]).T
    assert np.allclose(res["O"], vhat[jstar][None, :], rtol=0, atol=1e-15)
    # the dominant key's block sits more than 130 binades above every other block
    others = np.delete(res["E"], jstar // 32, axis=1)
    assert np.all(res["M"][:, None] - others > 130)


def test_extreme_row_range_stays_finite():
    rng = np.random.default_rng(19)
    N, d = 512, 128
    q = rng.standard_normal((N, d))
    k = rng.standard_normal((N, d))
    q[:, :3] *= 40.0
    k[:, :3] *= 40.0
    ops = mxfp4.quantize(q) + mxfp4.quantize(k) + mxfp4.quantize(rng.standard_normal((N, d)), axis=-2)
    res = directp.forward_rows(*ops, np.arange(0, N, 7), 1 / np.sqrt(d))
    span = res["E"].max(axis=1) - res["E"].min(axis=1)
    assert span.max() > 254          # beyond the E8M0 byte range
    assert np.all(np.isfinite(res["O"])) and np.all(res["D"] > 0)
    u = directp.p_scale_bytes(res["E"], res["M"])
    assert np.all(u[res["E"] - res["M"][:, None] < -127] == 0)


def test_plausibility_band_against_exact_attention(golden_dir):
    """MX/MX Direct-P fast on Gaussian D128 inputs lands near the paper's MX/MX
    control (Table all-formats); the band is the paper's error scale, not parity."""
    rng = np.random.default_rng(20)
    N, d = 1024, 128
    (q, k, v), ops = _quantized_head(rng, N, d)
    s = 1 / np.sqrt(d)
    res = directp.forward_rows(*ops, np.arange(N), s, want_codes=False)
    ref = exact.attention(q, k, v, s)
    cos, rel, _ = exact.error_metrics(res["O"], ref)
    p_cos, p_rel = _golden(golden_dir, "operator_error.txt", "mxmx_s1024")
    assert 0.90 <= cos <= 0.97 and 0.30 <= rel <= 0.42, (cos, rel)
    assert abs(cos - p_cos) < 0.02 and abs(rel - p_rel) < 0.04, (cos, rel)
    # the ideal converter is more accurate than the affine fit
    ideal = directp.forward_rows(*ops, np.arange(N), s, mode="exp2", want_codes=False)
    assert exact.error_metrics(ideal["O"], ref)[1] < rel


def test_raw_scores_exactness_guard():
    q6 = np.array([[1.0, 2.0 ** 40]])
    k6 = np.array([[1.0, 2.0 ** -10]])
    with pytest.raises(ValueError):
        directp.raw_scores(q6, k6)   # 1 + 2**30 needs 31 significant bits


# ---- native-exponential mixing (EX2 density) ----------------------------------------------

def test_ex2_key_mask_spacing():
    """k of the 16 pairs of a block, evenly spaced, both keys of a pair together."""
    for kx in directp.EX2_PAIRS:
        m = directp.ex2_key_mask(kx)
        assert m.sum() == 2 * kx
        assert np.array_equal(m[0::2], m[1::2])
        if kx:
            sel = np.flatnonzero(m[0::2])
            assert np.all(np.diff(sel) == 16 // kx) and sel[0] == 0
    with pytest.raises(ValueError):
        directp.ex2_key_mask(3)


@pytest.fixture(scope="module")
def gaussian_head_d128():
    rng = np.random.default_rng(20)
    N, d = 1024, 128
    (q, k, v), ops = _quantized_head(rng, N, d)
    return (q, k, v), ops, 1 / np.sqrt(d)


def test_all_ex2_pairs_is_the_ideal_converter(gaussian_head_d128):
    """ex2_pairs = 16 decides every code as Q_E2M1(2**x) (eq. ideal-code-path); the
    fp64 formula of that equation differs only where 2**x lies within fp32
    rounding of an E2M1 boundary."""
    _, ops, s = gaussian_head_d128
    rows = np.arange(256)
    mix = directp.forward_rows(*ops, rows, s, ex2_pairs=16)
    ideal = directp.forward_rows(*ops, rows, s, mode="exp2_exact")     # unrounded 2**x, fp64
    assert np.array_equal(mix["E"], ideal["E"])
    p = ideal["codes"]
    bounds = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
    near = np.min(np.abs(p[..., None] / bounds - 1.0), axis=-1) < 1e-6
    ref_codes = e2m1.round_index(p)
    assert np.array_equal(mix["codes"][~near], ref_codes[~near])
    # (the window holds, among others, every exactly-zero score of a block with
    # E_B = 3: 2**x is then 6/8 = 0.75, a tie, where the fp64 formula's rounded
    # log2 6 lands just below it)
    assert near.mean() < 1e-3


@pytest.mark.parametrize("kx", [1, 2, 4, 8])
def test_ex2_mixing_touches_only_selected_pairs(gaussian_head_d128, kx):
    """Unselected keys keep the affine codes bit for bit; selected keys carry the
    all-native codes."""
    _, ops, s = gaussian_head_d128
    rows = np.arange(0, 1024, 5)
    aff = directp.forward_rows(*ops, rows, s)["codes"]
    nat = directp.forward_rows(*ops, rows, s, ex2_pairs=16)["codes"]
    mix = directp.forward_rows(*ops, rows, s, ex2_pairs=kx)["codes"]
    keys = np.tile(directp.ex2_key_mask(kx), mix.shape[1] // 32)
    assert np.array_equal(mix[:, ~keys], aff[:, ~keys])
    assert np.array_equal(mix[:, keys], nat[:, keys])
    assert np.any(mix[:, keys] != aff[:, keys])


def test_ex2_density_raises_fidelity(gaussian_head_d128):
    """More native-exponential pairs move the operator toward the ideal converter:
    relative L2 against exact attention falls monotonically with the density,
    the direction of the paper's density sweep (Table b300-tuning), and the full
    density reaches the ideal converter's error."""
    (q, k, v), ops, s = gaussian_head_d128
    ref = exact.attention(q, k, v, s)
    rels = []
    for kx in directp.EX2_PAIRS:
        res = directp.forward_rows(*ops, np.arange(1024), s, ex2_pairs=kx, want_codes=False)
        rels.append(exact.error_metrics(res["O"], ref)[1])
    assert all(a > b for a, b in zip(rels, rels[1:])), rels
    ideal = directp.forward_rows(*ops, np.arange(1024), s, mode="exp2", want_codes=False)
    assert abs(rels[-1] - exact.error_metrics(ideal["O"], ref)[1]) < 1e-4


def test_ex2_block_argmax_gets_code_six(gaussian_head_d128):
    """At the block maximum x >= log2 6, so 2**x >= 6 saturates to code 6 on a
    selected key as it does under the affine map."""
    _, ops, s = gaussian_head_d128
    q6 = mxfp4.scaled_operand(*ops[0:2])[:64]
    k6 = mxfp4.scaled_operand(*ops[2:4])
    raw = directp.raw_scores(q6, k6)
    _, _, kk = directp.block_exponents_and_codes(raw, s, 1.5, 1.2, ex2_pairs=16)
    am = raw.reshape(64, -1, 32).argmax(axis=-1)
    assert np.all(np.take_along_axis(kk.reshape(64, -1, 32), am[..., None], -1) == 7)


# ---- causal form and the saved row normaliser ----------------------------------------------

def _scores_natural(ops, rows, s):
    q6 = mxfp4.scaled_operand(*ops[0:2])[rows]
    k6 = mxfp4.scaled_operand(*ops[2:4])
    return (q6 @ k6.T) * (s / 36.0)                          # z = s Qhat.Khat


@pytest.mark.parametrize("causal", [False, True])
def test_lse_of_unrounded_codes_is_the_textbook_logsumexp(causal):
    """With unrounded 2**x in place of the codes (mode exp2_exact) the represented
    operator is softmax itself, so LSE_i = M_i ln 2 + ln(D_i / 6) must equal
    log sum_j exp(z_ij) over the keys row i sees."""
    rng = np.random.default_rng(30)
    N, d = 256, 64
    _, ops = _quantized_head(rng, N, d, scale_q=3.0)
    rows = np.arange(N)
    res = directp.forward_rows(*ops, rows, SCALE64, mode="exp2_exact", causal=causal)
    z = _scores_natural(ops, rows, SCALE64)
    if causal:
        z = np.where(np.arange(N)[None, :] <= rows[:, None], z, -np.inf)
    zmax = z.max(axis=-1, keepdims=True)
    ref = zmax[:, 0] + np.log(np.exp(z - zmax).sum(axis=-1))
    assert np.allclose(res["LSE"], ref, rtol=0, atol=1e-12)


def test_causal_unrounded_reduces_to_masked_softmax_attention():
    rng = np.random.default_rng(31)
    N, d = 256, 64
    _, ops = _quantized_head(rng, N, d)
    rows = np.arange(N)
    res = directp.forward_rows(*ops, rows, SCALE64, mode="exp2_exact", causal=True)
    z = _scores_natural(ops, rows, SCALE64)
    z = np.where(np.arange(N)[None, :] <= rows[:, None], z, -np.inf)
    p = np.exp(z - z.max(axis=-1, keepdims=True))
    v = mxfp4.scaled_operand(*ops[4:6]).T / 6.0
    ref = (p @ v) / p.sum(axis=-1, keepdims=True)
    assert np.allclose(res["O"], ref, rtol=0, atol=1e-12)


def test_causal_codes_and_first_row():
    """Hidden keys take code 0; blocks the row sees whole keep the noncausal exponent
    and codes; row 0 sees key 0 alone, which gets code 6, so O_0 = Vhat_0 exactly."""
    rng = np.random.default_rng(32)
    N, d = 256, 64
    _, ops = _quantized_head(rng, N, d)
    rows = np.arange(N)
    full = directp.forward_rows(*ops, rows, SCALE64)
    cau = directp.forward_rows(*ops, rows, SCALE64, causal=True)
    vis = np.arange(N)[None, :] <= rows[:, None]
    assert np.all(cau["codes"][~vis] == 0)
    whole = np.repeat((np.arange(N // 32)[None, :] * 32 + 31) <= rows[:, None], 32, axis=-1)
    assert np.array_equal(cau["codes"][whole], full["codes"][whole])
    blocks_whole = (np.arange(N // 32)[None, :] * 32 + 31) <= rows[:, None]
    assert np.array_equal(cau["E"][blocks_whole], full["E"][blocks_whole])
    assert np.all(cau["E"][(np.arange(N // 32)[None, :] * 32) > rows[:, None]] == directp.NO_BLOCK)
    assert cau["codes"][0, 0] == 7
    v = mxfp4.scaled_operand(*ops[4:6]).T / 6.0
    assert np.array_equal(cau["O"][0], v[0])


def test_direct_p_lse_stays_near_the_exact_one():
    """The affine codes approximate 2**x, so the represented LSE stays near the exact
    log-sum-exp.  The block maximum always takes code 6, i.e. 2**floor(y) in place of
    2**y, so a row with one visible key (row 0) can sit up to ln 2 low; long rows
    average the code map's error out (a plausibility band, not parity)."""
    rng = np.random.default_rng(33)
    N, d = 512, 128
    _, ops = _quantized_head(rng, N, d)
    rows = np.arange(N)
    s = 1 / np.sqrt(d)
    res = directp.forward_rows(*ops, rows, s, causal=True)
    ref = directp.forward_rows(*ops, rows, s, mode="exp2_exact", causal=True)
    dl = res["LSE"] - ref["LSE"]
    assert np.all(dl > -np.log(2) - 1e-12) and np.all(dl < 0.25)
    assert np.max(np.abs(dl[256:])) < 0.25 and abs(np.mean(dl[256:])) < 0.1
