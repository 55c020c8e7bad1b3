"""GPU check of the same-design BF16 baseline against exact fp64 attention
(eq. exact-attention) on the same bf16 inputs."""
import numpy as np
import pytest
import torch

import workloads
from oracle import exact
from parity import load_workload, rel_l2_cos

pytestmark = pytest.mark.gpu

# bf16 rounding of P (relative 2^-9 per element) bounds the error well below these
REL_MAX = 5e-3
COS_MIN = 0.99999


@pytest.fixture(scope="module")
def fa():
    import paper_2609_04105_amd as fa
    return fa


def _check(fa, host64, dev, rows, label):
    q, k, v = host64
    B, H, N, d = q.shape
    s = 1.0 / np.sqrt(d)
    qg, kg, vg = (t.to(torch.bfloat16) for t in dev)
    vt = fa.transpose_bf16(vg)
    assert torch.equal(vt, vg.transpose(-1, -2).contiguous())
    out = fa.forward_bf16(qg, kg, vt)
    torch.cuda.synchronize()
    got = out.reshape(-1, d)[torch.from_numpy(np.asarray(rows)).cuda()].cpu().numpy()
    q16, k16, v16 = (workloads.as_f64(t.cpu()) for t in (qg, kg, vg))
    ref = np.zeros((len(rows), d))
    heads = np.asarray(rows) // N
    for bh in np.unique(heads):
        b, h = divmod(int(bh), H)
        sel = np.nonzero(heads == bh)[0]
        ref[sel] = exact.attention(q16[b, h][np.asarray(rows)[sel] % N], k16[b, h], v16[b, h], s)
    rel, cos = rel_l2_cos(got, ref)
    print(f"[bf16 {label}] rel-L2 {rel:.3e} cos {cos:.8f}", flush=True)
    assert rel <= REL_MAX and cos >= COS_MIN


def test_bf16_small_all_rows(fa):
    host64, dev = load_workload("small_b1h8_n1024_d64")
    _check(fa, host64, dev, np.arange(8 * 1024), "small")


def test_bf16_tiny(fa):
    host64, dev = load_workload("tiny_b1h1_n128_d64")
    _check(fa, host64, dev, np.arange(128), "tiny")


@pytest.mark.parametrize("name", ["outlier_b2h16_n4096_d128", "long_b1h32_n16384_d128"])
def test_bf16_full_size_sampled(fa, name):
    host64, dev = load_workload(name)
    _check(fa, host64, dev, workloads.sampled_rows(name)[::4], name)


@pytest.mark.parametrize("d", [64, 128])
def test_bf16_tail_launch(fa, d):
    """B1 H24 N4096: the four-wave tail launch (384 eight-wave workgroups would
    leave a half-empty second round); every 97th row checked."""
    g = torch.Generator().manual_seed(10)
    q, k, v = (torch.randn(1, 24, 4096, d, generator=g).to(torch.bfloat16) for _ in range(3))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    _check(fa, host64, (q.cuda(), k.cuda(), v.cuda()), np.arange(0, 24 * 4096, 97), f"tail d{d}")
