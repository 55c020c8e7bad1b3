"""Pins of the textbook attention oracle (oracle/exact.py): softmax attention of
eq. attention-intro / eq. exact-attention and the online recurrence over key
tiles of eq. online-recurrence.

The direct form is pinned by a pure-Python brute force (scalar loops over
``math.exp``, no NumPy arithmetic) on tiny inputs and by closed forms; the online
form is pinned against the direct form for tile widths that divide N, that leave
a ragged last tile, and that are wider than N, on logits large enough that a
missing rescale of the running maximum would overflow or lose the row.
"""
import math

import numpy as np
import pytest

from oracle import exact


def _brute_force(q, k, v, s):
    """O_i = sum_j exp(z_ij) v_j / sum_j exp(z_ij), z_ij = s <q_i, k_j>: scalar loops."""
    n_q, d = len(q), len(q[0])
    out = []
    for i in range(n_q):
        z = [s * sum(q[i][c] * k[j][c] for c in range(d)) for j in range(len(k))]
        zmax = max(z)
        w = [math.exp(zj - zmax) for zj in z]
        tot = math.fsum(w)
        out.append([math.fsum(w[j] * v[j][c] for j in range(len(k))) / tot for c in range(len(v[0]))])
    return np.array(out)


@pytest.mark.parametrize("seed,n_q,n_k,d", [(0, 3, 5, 4), (1, 4, 7, 3), (2, 1, 1, 2), (3, 6, 9, 8)])
def test_direct_form_equals_brute_force(seed, n_q, n_k, d):
    rng = np.random.default_rng(seed)
    q, k, v = rng.normal(size=(n_q, d)), rng.normal(size=(n_k, d)), rng.normal(size=(n_k, d + 1))
    s = 1.0 / math.sqrt(d)
    ref = _brute_force(q.tolist(), k.tolist(), v.tolist(), s)
    np.testing.assert_allclose(exact.attention(q, k, v, s), ref, rtol=1e-13, atol=1e-14)


def test_direct_form_closed_forms():
    rng = np.random.default_rng(4)
    k, v = rng.normal(size=(11, 4)), rng.normal(size=(11, 5))
    # Q = 0: every score is 0, the softmax is uniform and O is the mean of V
    np.testing.assert_allclose(exact.attention(np.zeros((3, 4)), k, v, 0.5), np.tile(v.mean(axis=0), (3, 1)),
                               rtol=1e-14, atol=1e-15)
    # one key far above the rest: O is that key's value row
    k2 = np.zeros((11, 4))
    k2[6, 0] = 1.0
    q2 = np.array([[2000.0, 0, 0, 0]])
    np.testing.assert_array_equal(exact.attention(q2, k2, v, 1.0), v[6:7])
    # two equal scores far above the rest: O is their average
    k2[2, 0] = 1.0
    np.testing.assert_allclose(exact.attention(q2, k2, v, 1.0), (v[2:3] + v[6:7]) / 2, rtol=1e-15)
    # a constant V row is returned unchanged
    np.testing.assert_allclose(exact.attention(rng.normal(size=(2, 4)), k, np.full((11, 5), 3.25), 1.0), 3.25,
                               rtol=1e-15)


@pytest.mark.parametrize("tile", [1, 16, 64, 100, 200, 512])
@pytest.mark.parametrize("logit_scale", [1.0, 40.0])
def test_online_recurrence_equals_direct_form(tile, logit_scale):
    """N = 200 keys: tile 16 and 64 leave ragged last tiles (8 keys), 100 divides N,
    200 is one tile and 512 is wider than N.  With logit scale 40 the row maxima
    move by hundreds between tiles (a dropped correction factor would be off by
    e^hundreds)."""
    rng = np.random.default_rng(5)
    B, H, Nq, N, d = 2, 3, 17, 200, 8
    q = rng.normal(size=(B, H, Nq, d)) * logit_scale
    k = rng.normal(size=(B, H, N, d))
    v = rng.normal(size=(B, H, N, d))
    s = 1.0 / math.sqrt(d)
    ref = exact.attention(q, k, v, s)
    got = exact.attention_online(q, k, v, s, tile=tile)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_online_recurrence_increasing_keys():
    """Keys sorted so that every tile raises the running maximum: the correction
    factor is applied at every tile boundary."""
    rng = np.random.default_rng(6)
    N, d = 96, 4
    k = rng.normal(size=(N, d))
    q = np.ones((2, d)) * 10.0
    k = k[np.argsort(k @ q[0])]
    v = rng.normal(size=(N, 3))
    np.testing.assert_allclose(exact.attention_online(q, k, v, 1.0, tile=8), exact.attention(q, k, v, 1.0),
                               rtol=1e-12, atol=1e-13)


def test_error_metrics_closed_forms():
    r = np.array([3.0, 4.0])
    assert exact.error_metrics(r, r) == pytest.approx((1.0, 0.0, 0.0))
    cos, rel, rmse = exact.error_metrics(np.array([3.0, 0.0]), r)
    assert cos == pytest.approx(3.0 / 5.0) and rel == pytest.approx(4.0 / 5.0)
    assert rmse == pytest.approx(math.sqrt(16.0 / 2))
    assert exact.error_metrics(-r, r)[0] == pytest.approx(-1.0)
