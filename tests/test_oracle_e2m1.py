"""Pins of the E2M1 codec (oracle/e2m1.py) against the values the paper prints."""
import os

import numpy as np
import pytest

from oracle import e2m1


def _golden(golden_dir, key):
    with open(os.path.join(golden_dir, "e2m1.txt")) as f:
        for line in f:
            if line.startswith(key + " "):
                return [float(t) for t in line.split()[1:]]
    raise KeyError(key)


def test_magnitude_table_matches_paper(golden_dir):
    assert list(e2m1.MAGNITUDES) == _golden(golden_dir, "magnitudes")


def test_boundaries_are_paper_midpoints(golden_dir):
    bounds = _golden(golden_dir, "boundaries")
    mids = (e2m1.MAGNITUDES[1:] + e2m1.MAGNITUDES[:-1]) / 2
    assert list(mids) == bounds
    for j, t in enumerate(bounds):
        below, above = np.nextafter(t, -np.inf), np.nextafter(t, np.inf)
        assert e2m1.round_index(below) == j
        assert e2m1.round_index(above) == j + 1
        # exact midpoint: ties to the even index (mantissa bit 0)
        assert e2m1.round_index(t) == (j if j % 2 == 0 else j + 1)


def test_round_matches_boundary_count():
    # independent formulation: count the boundaries at or below r, with the tie
    # direction of each boundary decided by the parity of its upper neighbour
    rng = np.random.default_rng(1)
    r = np.concatenate([rng.uniform(0, 8, 20000), np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0, 7.0, 100.0])])
    bounds = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
    upper_even = (np.arange(1, 8) % 2) == 0
    crossed = np.where(upper_even, r[:, None] >= bounds, r[:, None] > bounds)
    assert np.array_equal(e2m1.round_index(r), crossed.sum(axis=1))


def test_saturation_and_exact_values():
    assert e2m1.round_value(6.0) == 6.0
    assert e2m1.round_value(1e30) == 6.0
    for k, m in enumerate(e2m1.MAGNITUDES):
        assert e2m1.round_index(m) == k


def test_signed_codes_round_trip():
    codes = np.arange(16, dtype=np.uint8)
    vals = e2m1.decode(codes)
    assert np.array_equal(e2m1.encode(vals)[vals != 0], codes[vals != 0])
    assert e2m1.encode(-0.0) == 8 and e2m1.encode(0.0) == 0
    assert e2m1.decode(np.uint8(0xF)) == -6.0


def test_nibble_order():
    packed = e2m1.pack_nibbles(np.array([1, 2, 3, 4], dtype=np.uint8))
    assert list(packed) == [0x21, 0x43]
    assert list(e2m1.unpack_nibbles(packed)) == [1, 2, 3, 4]


def test_rejects_negative_and_nan():
    with pytest.raises(ValueError):
        e2m1.round_index(-1.0)
    with pytest.raises(ValueError):
        e2m1.round_index(np.nan)


def test_round_matches_exhaustive_nearest_entry():
    """Brute force: distance to all eight magnitudes, ties to the even index."""
    rng = np.random.default_rng(9)
    r = np.concatenate([rng.uniform(0, 7, 50000), e2m1.MAGNITUDES,
                        (e2m1.MAGNITUDES[1:] + e2m1.MAGNITUDES[:-1]) / 2])
    dist = np.abs(r[:, None] - e2m1.MAGNITUDES[None, :])
    best = dist == dist.min(axis=1, keepdims=True)
    even = np.arange(8) % 2 == 0
    want = np.where(best.sum(axis=1) > 1, np.argmax(best & even, axis=1), np.argmax(best, axis=1))
    assert np.array_equal(e2m1.round_index(r), want)
