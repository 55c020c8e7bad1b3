"""Seeded synthetic attention inputs shared by the CPU oracle and the HIP path.

This module holds random draws, casts and shapes only: none of the method's
arithmetic.  Both sides receive the same tensors from here; nothing else is
shared between them.

The paper's own operator inputs (a third-party tensor factory with a fixed seed,
and model activations) are not available, so these workloads stand in for them:
i.i.d. N(0, 1) Q, K, V with softmax scale 1/sqrt(d) reproduce the Gaussian
error statistics the paper reports for its synthetic grid, and two stress
variants add outlier channels and heavy tails in the spirit of the large model
logits that motivate the paper's range guard.

Recipe (all draws on the CPU with ``torch.Generator().manual_seed(seed)``, in the
order listed, as fp32 ``[B, H, N, d]``):

* ``gaussian``: Q, K, V = randn, randn, randn.
* ``outlier``: as ``gaussian``, then ``ch = randperm(d)[:ceil(0.02 d)]`` and
  ``Q[..., ch] *= 8``, ``K[..., ch] *= 8`` (same channels for every batch and
  head, so the outlier products add coherently).
* ``student_t``: for each of Q, K, V in turn: ``Z = randn``, then four more
  randn draws ``W = sum of squares``, ``T = Z / sqrt(W / 4)`` (Student-t with
  four degrees of freedom), scaled by ``1/sqrt(2)`` to unit variance.

Tensors are then cast to the workload dtype (round to nearest even for bf16).
Sampled query rows for large workloads are
``randperm(B*H*N, generator=manual_seed(seed + 1000))[:4096]`` over flattened
``(b*H + h)*N + i`` indices.

Size-limit cases (the longest sequence, the largest grid) take their operands
already in MXFP4 form, so that the oracle needs no quantizer pass over billions
of values: :func:`random_mxfp4_operands` draws every code byte uniformly (both
nibbles, all sixteen E2M1 codes, signed zero included) and every E8M0 scale byte
uniformly from a narrow band around 127, in the order Q codes, Q scales, K
codes, K scales, Vt codes, Vt scales.
"""
import math
from dataclasses import dataclass

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    N: int
    d: int
    dist: str          # "gaussian" | "outlier" | "student_t"
    dtype: str         # "fp32" | "bf16"
    seed: int
    all_rows: bool     # parity checked on every query row (else on sampled rows)

    @property
    def softmax_scale(self):
        return 1.0 / math.sqrt(self.d)

    @property
    def rows(self):
        return self.B * self.H * self.N

    @property
    def flops(self):
        """4 B H N^2 d: the paper's ops count BH 2S^2 (D_QK + D_VO) (eq. hao-flops)."""
        return 4.0 * self.B * self.H * self.N * self.N * self.d


WORKLOADS = {
    w.name: w
    for w in (
        Workload("tiny_b1h1_n128_d64", 1, 1, 128, 64, "gaussian", "fp32", 0, True),
        Workload("small_b1h8_n1024_d64", 1, 8, 1024, 64, "gaussian", "bf16", 1, True),
        Workload("outlier_b2h16_n4096_d128", 2, 16, 4096, 128, "outlier", "bf16", 2, False),
        Workload("student_t_b1h32_n8192_d128", 1, 32, 8192, 128, "student_t", "bf16", 3, False),
        Workload("long_b1h32_n16384_d128", 1, 32, 16384, 128, "gaussian", "bf16", 4, False),
    )
}

# The throughput point: the largest single-GPU workload.
BENCH_WORKLOAD = "long_b1h32_n16384_d128"
N_SAMPLED_ROWS = 4096


def _student_t(shape, g):
    z = torch.randn(shape, generator=g)
    w = torch.zeros(shape)
    for _ in range(4):
        w += torch.randn(shape, generator=g) ** 2
    return z / torch.sqrt(w / 4.0) / math.sqrt(2.0)


def generate(w, B=None, H=None, N=None):
    """(Q, K, V) CPU tensors of workload ``w`` (a Workload or its name).

    ``B``, ``H``, ``N`` override the shape (same recipe and seed) for reduced
    test cases.
    """
    if isinstance(w, str):
        w = WORKLOADS[w]
    shape = (B or w.B, H or w.H, N or w.N, w.d)
    g = torch.Generator().manual_seed(w.seed)
    if w.dist == "student_t":
        q = _student_t(shape, g)
        k = _student_t(shape, g)
        v = _student_t(shape, g)
    else:
        q = torch.randn(shape, generator=g)
        k = torch.randn(shape, generator=g)
        v = torch.randn(shape, generator=g)
    if w.dist == "outlier":
        n_out = math.ceil(0.02 * w.d)
        ch = torch.randperm(w.d, generator=g)[:n_out]
        q[..., ch] *= 8.0
        k[..., ch] *= 8.0
    elif w.dist not in ("gaussian", "student_t"):
        raise ValueError(w.dist)
    dt = {"fp32": torch.float32, "bf16": torch.bfloat16}[w.dtype]
    return q.to(dt), k.to(dt), v.to(dt)


def sampled_rows(w, n=N_SAMPLED_ROWS):
    """Flattened query-row indices on which large workloads are checked (ascending)."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    if w.all_rows:
        return np.arange(w.rows, dtype=np.int64)
    g = torch.Generator().manual_seed(w.seed + 1000)
    idx = torch.randperm(w.rows, generator=g)[:n].numpy().astype(np.int64)
    return np.sort(idx)


def as_f64(t):
    """fp64 NumPy copy of a CPU tensor (bf16 widens exactly)."""
    return t.detach().to(torch.float64).cpu().numpy()


def random_mxfp4_operands(B, H, N, d, seed, scale_lo=125, scale_hi=129, v_fp8=False):
    """Uniform random MXFP4 operand bytes in the layout of the forward's
    arguments: q/k codes [B, H, N, d/2] and scales [B, H, N, d/32], Vt codes
    [B, H, d, N/2] and scales [B, H, d, N/32] (uint8 CPU tensors).

    Scale bytes lie in [scale_lo, scale_hi]; with a band of width 4 every score
    of d <= 128 products is a multiple of 2^-6 below 2^17, so it is exact in fp32.
    ``v_fp8``: Vt codes are E4M3 bytes [B, H, d, N] instead, a uniform sign bit
    over a magnitude byte uniform in [0, 0x7e] (every finite E4M3 value; 0x7f
    is NaN).
    """
    g = torch.Generator().manual_seed(seed)

    def draw(shape, lo, hi):
        return torch.randint(lo, hi + 1, shape, generator=g, dtype=torch.uint8)

    ops = [draw((B, H, N, d // 2), 0, 255), draw((B, H, N, d // 32), scale_lo, scale_hi),
           draw((B, H, N, d // 2), 0, 255), draw((B, H, N, d // 32), scale_lo, scale_hi)]
    if v_fp8:
        ops.append(draw((B, H, d, N), 0, 0x7E) | (draw((B, H, d, N), 0, 1) << 7))
    else:
        ops.append(draw((B, H, d, N // 2), 0, 255))
    ops.append(draw((B, H, d, N // 32), scale_lo, scale_hi))
    return tuple(ops)
