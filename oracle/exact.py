"""Textbook softmax attention in fp64 (test infrastructure; see oracle/__init__).

``O_i = sum_j exp(z_ij) V_j / sum_j exp(z_ij)`` with ``z = s Q K^T``
(eq. attention-intro and eq. exact-attention), and the FlashAttention online
recurrence over key tiles (eq. online-recurrence).  This is the accuracy
reference that the Direct-P approximation is measured against and the check for
the BF16 kernel; it is not the parity target of the FP4 path.
"""
import numpy as np


def attention(q, k, v, softmax_scale):
    """Exact attention for [..., N, d] inputs, fp64, max-subtracted for range."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    z = softmax_scale * (q @ np.swapaxes(k, -1, -2))
    z = z - z.max(axis=-1, keepdims=True)
    p = np.exp(z)
    return (p @ v) / p.sum(axis=-1, keepdims=True)


def attention_online(q, k, v, softmax_scale, tile=64):
    """Same result through the online recurrence over key tiles of width ``tile``."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    n = k.shape[-2]
    m = np.full(q.shape[:-1], -np.inf)
    ell = np.zeros(q.shape[:-1])
    o = np.zeros(q.shape[:-1] + (v.shape[-1],))
    for t0 in range(0, n, tile):
        z = softmax_scale * (q @ np.swapaxes(k[..., t0:t0 + tile, :], -1, -2))
        m_new = np.maximum(m, z.max(axis=-1))
        corr = np.exp(m - m_new)
        p = np.exp(z - m_new[..., None])
        ell = corr * ell + p.sum(axis=-1)
        o = corr[..., None] * o + p @ v[..., t0:t0 + tile, :]
        m = m_new
    return o / ell[..., None]


def error_metrics(approx, ref):
    """(cosine, relative L2, RMSE) of ``approx`` against ``ref`` (Sec. "Metrics")."""
    a = np.asarray(approx, dtype=np.float64).ravel()
    r = np.asarray(ref, dtype=np.float64).ravel()
    cos = float(a @ r / (np.linalg.norm(a) * np.linalg.norm(r)))
    rel = float(np.linalg.norm(a - r) / np.linalg.norm(r))
    rmse = float(np.sqrt(np.mean((a - r) ** 2)))
    return cos, rel, rmse
