"""Pins of the MXFP4 input quantizer (oracle/mxfp4.py)."""
import os

import numpy as np
import pytest

from oracle import e2m1, mxfp4, prange


def _blocks(rng, n, kind):
    if kind == "gauss32":
        return rng.standard_normal((n, 32)).astype(np.float32).astype(np.float64)
    if kind == "bf16":
        import torch
        return torch.randn(n, 32, generator=torch.Generator().manual_seed(int(rng.integers(1 << 30)))) \
            .to(torch.bfloat16).to(torch.float64).numpy()
    if kind == "wide":
        x = rng.standard_normal((n, 32)) * np.exp2(rng.integers(-40, 40, (n, 32)))
        return x.astype(np.float32).astype(np.float64)
    raise ValueError(kind)


@pytest.mark.parametrize("kind", ["gauss32", "bf16", "wide"])
def test_scale_is_floor_or_ceil_power_of_two(kind):
    rng = np.random.default_rng(4)
    x = _blocks(rng, 2000, kind)
    _, scales = mxfp4.quantize(x)
    e = scales.astype(np.int64)[:, 0] - 127
    a = np.abs(x).max(axis=1)
    alpha = np.ldexp(1.0, e)
    floor_ok = (alpha <= a) & (a < 2 * alpha)
    ceil_ok = (alpha >= a) & (alpha / 2 < a)
    assert np.all(floor_ok | ceil_ok)


@pytest.mark.parametrize("kind", ["gauss32", "bf16", "wide"])
def test_delta_rule_is_exact_sse_comparison(kind):
    rng = np.random.default_rng(5)
    x = _blocks(rng, 150, kind)
    e, _ = mxfp4.choose_exponent(x)
    errs = mxfp4.squared_errors(x)
    n_floor = 0
    for i, (sse_f, sse_c) in enumerate(errs):
        e_f, e_c = mxfp4._block_exponents(np.abs(x[i]).max())
        if e_f == e_c:
            assert e[i] == e_c
            continue
        want = e_f if sse_f < sse_c else e_c
        n_floor += want == e_f
        assert e[i] == want, i
    assert n_floor > 0  # the floor candidate does get chosen


def test_chosen_error_not_worse_than_either_candidate():
    rng = np.random.default_rng(6)
    x = _blocks(rng, 100, "gauss32")
    codes, scales = mxfp4.quantize(x)
    q = e2m1.decode(e2m1.unpack_nibbles(codes))
    from fractions import Fraction
    for i, (sse_f, sse_c) in enumerate(mxfp4.squared_errors(x)):
        alpha = Fraction(2) ** (int(scales[i, 0]) - 127)
        got = sum((Fraction(float(a)) - alpha * Fraction(float(b)) / 6) ** 2 for a, b in zip(x[i], q[i]))
        assert got == min(sse_f, sse_c)


def test_idempotent_on_represented_values():
    rng = np.random.default_rng(7)
    x = _blocks(rng, 3000, "wide")
    xh = mxfp4.dequantize(*mxfp4.quantize(x))
    xhh = mxfp4.dequantize(*mxfp4.quantize(xh))
    assert np.array_equal(xh, xhh)


def test_exact_powers_and_table_values_round_trip():
    x = np.zeros((1, 32))
    x[0, :8] = e2m1.MAGNITUDES / 6.0 * 4.0      # block amplitude 4 (max 6*4/6 = 4)
    x[0, 8:16] = -e2m1.MAGNITUDES / 6.0 * 4.0
    codes, scales = mxfp4.quantize(x)
    assert scales[0, 0] == 127 + 2
    assert np.array_equal(mxfp4.dequantize(codes, scales), x)


def test_zero_negative_zero_and_nonfinite_blocks():
    x = np.zeros((3, 32))
    x[0, 5] = -0.0
    x[1, 3] = np.nan
    x[2, 7] = np.inf
    codes, scales = mxfp4.quantize(x)
    assert list(scales[:, 0]) == [0, 255, 255]
    unpacked = e2m1.unpack_nibbles(codes)
    assert unpacked[0, 5] == 8 and unpacked[0].sum() == 8
    assert np.all(unpacked[1:] == 0)


def test_tiny_and_huge_blocks_clamp_exponent():
    x = np.full((2, 32), 1.0)
    x[0] *= 2.0 ** -140          # below the E8M0 range: exponent clamps to -127
    x[1] *= 2.0 ** 127 * 1.5     # amplitude candidates 2^127 / 2^128: clamps to 127
    codes, scales = mxfp4.quantize(x)
    assert list(scales[:, 0]) == [0, 254]
    assert np.all(e2m1.unpack_nibbles(codes)[1] == 7)   # saturated at 6


def test_axis_layouts():
    rng = np.random.default_rng(8)
    v = rng.standard_normal((2, 64, 96)).astype(np.float32)
    c1, s1 = mxfp4.quantize(v, axis=-2)
    c2, s2 = mxfp4.quantize(np.swapaxes(v, -1, -2), axis=-1)
    assert c1.shape == (2, 96, 32) and s1.shape == (2, 96, 2)
    assert np.array_equal(c1, c2) and np.array_equal(s1, s2)
    # element (n, c) of V lives in row c, nibble n of the transposed codes
    vt = mxfp4.dequantize(c1, s1)
    assert vt[1, 7, 40] == mxfp4.dequantize(*mxfp4.quantize(v[1, 32:64, 7].reshape(1, 32)))[0, 40 - 32]


# --- Table p-range (Sec. "Problem 2") pins the amplitude rule ----------------

def _table(golden_dir):
    rows = {}
    with open(os.path.join(golden_dir, "table_p_range.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            t = line.split()
            rows[(int(t[0]), t[1])] = dict(zip(
                ["zero_scales", "zero_payload", "lost_mass", "p_rel_l2", "pv_cos", "pv_rel_l2"],
                [float(v) for v in t[2:]]))
    return rows


def _scores(S, seed=0, D=128):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((S, D))
    k = rng.standard_normal((S, D))
    v = rng.standard_normal((S, D))
    return q @ k.T / np.sqrt(D), v


def _close(got, want, rel):
    for key in ("zero_payload", "lost_mass", "p_rel_l2", "pv_rel_l2"):
        if abs(got[key] - want[key]) > rel * want[key]:
            return False
    return abs(got["pv_cos"] - want["pv_cos"]) < 0.002 and got["zero_scales"] == want["zero_scales"]


def test_table_p_range_mxfp4_row(golden_dir):
    z, v = _scores(1024)
    got = prange.diagnose(z, v, "mxfp4")
    assert _close(got, _table(golden_dir)[(1024, "mxfp4")], rel=0.05), got


def test_table_p_range_nvfp4_g448_row(golden_dir):
    z, v = _scores(1024)
    got = prange.diagnose(z, v, "nvfp4", G=448.0)
    assert _close(got, _table(golden_dir)[(1024, "nvfp4_g448")], rel=0.05), got


def test_table_p_range_nvfp4_g1_row(golden_dir):
    z, v = _scores(1024)
    got = prange.diagnose(z, v, "nvfp4", G=1.0)
    want = _table(golden_dir)[(1024, "nvfp4_g1")]
    for key in ("zero_scales", "zero_payload", "lost_mass", "p_rel_l2", "pv_rel_l2"):
        assert abs(got[key] - want[key]) < 0.05 * want[key], (key, got)


@pytest.mark.slow
def test_table_p_range_mxfp4_row_s4096(golden_dir):
    z, v = _scores(4096, seed=1)
    got = prange.diagnose(z[:1024], v, "mxfp4")
    assert _close(got, _table(golden_dir)[(4096, "mxfp4")], rel=0.05), got


@pytest.mark.parametrize("rule", ["ceil", "floor"])
def test_table_p_range_rejects_single_candidate_rules(golden_dir, monkeypatch, rule):
    """Planted mistake: always taking one candidate misses the paper's MXFP4 row."""
    def planted(blocks):
        a = np.abs(np.asarray(blocks, dtype=np.float64)).max(axis=-1)
        ok = a > 0
        e_f, e_c = mxfp4._block_exponents(np.where(ok, a, 1.0))
        return np.where(ok, e_c if rule == "ceil" else e_f, 0), ok
    monkeypatch.setattr(mxfp4, "choose_exponent", planted)
    z, v = _scores(1024)
    got = prange.diagnose(z, v, "mxfp4")
    assert not _close(got, _table(golden_dir)[(1024, "mxfp4")], rel=0.05), got
