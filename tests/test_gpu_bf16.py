"""GPU check of the same-design BF16 baseline against exact fp64 attention
(eq. exact-attention) on the same bf16 inputs, V taken as [B, H, N, d]."""
import numpy as np
import pytest
import torch

import workloads
from oracle import exact
from parity import load_workload, rel_l2_cos, row_rel_l2

pytestmark = pytest.mark.gpu

# bf16 rounding of P (relative 2^-9 per element, and the denominator sums the
# same rounded values) bounds the error well below these
REL_MAX = 5e-3
ROW_REL_MAX = 1e-2
COS_MIN = 0.99999


@pytest.fixture(scope="module")
def fa():
    import paper_2609_04105_amd as fa
    return fa


def _check(fa, host64, dev, rows, label, out_dtype=torch.float32):
    q, k, v = host64
    B, H, N, d = q.shape
    s = 1.0 / np.sqrt(d)
    qg, kg, vg = (t.to(torch.bfloat16) for t in dev)
    print(f"[bf16 {label}] B{B} H{H} N{N} d{d} rows={len(rows)}", flush=True)
    out = fa.forward_bf16(qg, kg, vg, out_dtype=out_dtype)
    torch.cuda.synchronize()
    got = out.reshape(-1, d)[torch.from_numpy(np.asarray(rows)).cuda()].float().cpu().numpy()
    q16, k16, v16 = (workloads.as_f64(t.cpu()) for t in (qg, kg, vg))
    ref = np.zeros((len(rows), d))
    heads = np.asarray(rows) // N
    for bh in np.unique(heads):
        b, h = divmod(int(bh), H)
        sel = np.nonzero(heads == bh)[0]
        ref[sel] = exact.attention(q16[b, h][np.asarray(rows)[sel] % N], k16[b, h], v16[b, h], s)
    rel, cos = rel_l2_cos(got, ref)
    worst = float(row_rel_l2(got, ref).max())
    print(f"[bf16 {label}] rel-L2 {rel:.3e} cos {cos:.8f} worst row rel-L2 {worst:.3e}", flush=True)
    assert rel <= REL_MAX and cos >= COS_MIN and worst <= ROW_REL_MAX, (rel, cos, worst)
    return out


def test_bf16_small_all_rows(fa):
    host64, dev = load_workload("small_b1h8_n1024_d64")
    _check(fa, host64, dev, np.arange(8 * 1024), "small")


def test_bf16_tiny(fa):
    host64, dev = load_workload("tiny_b1h1_n128_d64")
    _check(fa, host64, dev, np.arange(128), "tiny")


@pytest.mark.parametrize("N,d,H", [(128, 128, 1), (384, 128, 2), (640, 64, 2), (1152, 128, 3), (512, 128, 128),
                                   (256, 64, 256)])
def test_bf16_tiles_all_rows(fa, N, d, H):
    """One to eighteen 64-key tiles (a tail group of every length), four- and
    eight-wave workgroups, both head dimensions."""
    g = torch.Generator().manual_seed(N + d + H)
    q, k, v = (torch.randn(1, H, N, d, generator=g).to(torch.bfloat16) for _ in range(3))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    rows = np.arange(H * N) if H * N <= 8192 else np.arange(0, H * N, 7)
    _check(fa, host64, (q.cuda(), k.cuda(), v.cuda()), rows, f"tiles N{N} d{d} H{H}")


@pytest.mark.parametrize("name", ["outlier_b2h16_n4096_d128", "long_b1h32_n16384_d128"])
def test_bf16_full_size_sampled(fa, name):
    host64, dev = load_workload(name)
    _check(fa, host64, dev, workloads.sampled_rows(name)[::4], name)


@pytest.mark.parametrize("H,d", [(24, 64), (24, 128), (36, 64)])
def test_bf16_tail_launch(fa, H, d):
    """B1 N4096 grids of 384 and 576 eight-wave workgroups, rounds that do not
    divide the chip (one workgroup per CU at d = 128, two at d = 64); every 97th
    row checked."""
    g = torch.Generator().manual_seed(10)
    q, k, v = (torch.randn(1, H, 4096, d, generator=g).to(torch.bfloat16) for _ in range(3))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    _check(fa, host64, (q.cuda(), k.cuda(), v.cuda()), np.arange(0, H * 4096, 97), f"tail H{H} d{d}")


def test_bf16_large_logits_and_bf16_output(fa):
    """Scores spanning hundreds of binades within a row (the lazy reference
    rescales many times), and bf16 output equal to the rounded fp32 output."""
    g = torch.Generator().manual_seed(12)
    q = (torch.randn(1, 2, 1024, 128, generator=g) * 6).to(torch.bfloat16)
    k = (torch.randn(1, 2, 1024, 128, generator=g) * 6).to(torch.bfloat16)
    v = torch.randn(1, 2, 1024, 128, generator=g).to(torch.bfloat16)
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    dev = (q.cuda(), k.cuda(), v.cuda())
    o32 = _check(fa, host64, dev, np.arange(2048), "large logits")
    o16 = fa.forward_bf16(*dev, out_dtype=torch.bfloat16)
    assert torch.equal(o16, o32.to(torch.bfloat16))
    assert torch.isfinite(o32).all()


def test_bf16_deterministic_and_fully_overwritten(fa):
    g = torch.Generator().manual_seed(13)
    q, k, v = (torch.randn(1, 4, 512, 64, generator=g).to(torch.bfloat16).cuda() for _ in range(3))
    o1 = torch.full((1, 4, 512, 64), float("nan"), device="cuda")
    fa.forward_bf16(q, k, v, out=o1)
    o2 = torch.full_like(o1, float("nan"))
    fa.forward_bf16(q, k, v, out=o2)
    torch.cuda.synchronize()
    assert torch.isfinite(o1).all() and torch.equal(o1, o2)


def test_bf16_longest_sequence_sampled_rows(fa):
    """N = 2^22 keys, the longest sequence the entry point accepts: one head's K and V
    take 1 GiB each, so every in-head byte offset of the tile copies is near 2^30.
    Rows: the first and last of the sequence, of a query tile and of a workgroup,
    and random ones; inputs drawn on the GPU from a seeded generator."""
    N, d = 1 << 22, 128
    g = torch.Generator(device="cuda").manual_seed(24)
    q, k, v = (torch.randn((1, 1, N, d), device="cuda", generator=g).to(torch.bfloat16) for _ in range(3))
    rows = np.unique(np.concatenate([[0, 1, 255, 256, N // 2 + 31, N - 257, N - 256, N - 1],
                                     np.random.default_rng(24).integers(0, N, 8)]))
    print(f"[bf16 N=2^22] rows={len(rows)}", flush=True)
    out = fa.forward_bf16(q, k, v)
    torch.cuda.synchronize()
    got = out.reshape(-1, d)[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
    q64 = q[0, 0][torch.from_numpy(rows).cuda()].double().cpu().numpy()
    k64, v64 = (t[0, 0].double().cpu().numpy() for t in (k, v))
    ref = exact.attention(q64, k64, v64, 1.0 / np.sqrt(d))
    rel, cos = rel_l2_cos(got, ref)
    worst = float(row_rel_l2(got, ref).max())
    print(f"[bf16 N=2^22] rel-L2 {rel:.3e} cos {cos:.8f} worst row rel-L2 {worst:.3e}", flush=True)
    assert rel <= REL_MAX and cos >= COS_MIN and worst <= ROW_REL_MAX, (rel, cos, worst)


@pytest.mark.parametrize("B,H,N,d", [(1, 32, 2048, 128), (1, 31, 2048, 128), (1, 16, 2048, 64), (1, 15, 2048, 64),
                                     (3, 7, 1664, 128), (2, 5, 640, 64), (1, 1290, 256, 128), (1, 1, 128, 128)])
def test_bf16_launch_boundaries(fa, B, H, N, d):
    """Both sides of the launch rule (eight-wave workgroups from 256 of them at
    d = 128 and from 128 at d = 64, four-wave below and when N is not a multiple
    of 256), many heads, one tile; 40 seeded rows plus the first and last of the
    tensor and of a head."""
    g = torch.Generator().manual_seed(B * 1000003 + H * 1009 + N * 7 + d)
    q, k, v = (torch.randn(B, H, N, d, generator=g).to(torch.bfloat16) for _ in range(3))
    rows = np.random.default_rng(N + H).integers(0, B * H * N, 40)
    rows = np.unique(np.concatenate([rows, [0, N - 1, B * H * N - N, B * H * N - 1]]))
    heads = np.unique(rows // N)
    sel = torch.from_numpy(heads)
    # only the heads the rows touch go to the exact reference
    host64 = tuple(workloads.as_f64(t.reshape(B * H, 1, N, d)[sel].reshape(1, len(heads), N, d)) for t in (q, k, v))
    local = np.searchsorted(heads, rows // N) * N + rows % N
    s = 1.0 / np.sqrt(d)
    print(f"[bf16 sweep B{B} H{H} N{N} d{d}] rows={len(rows)}", flush=True)
    out = fa.forward_bf16(q.cuda(), k.cuda(), v.cuda())
    torch.cuda.synchronize()
    got = out.reshape(-1, d)[torch.from_numpy(rows).cuda()].float().cpu().numpy()
    ref = np.zeros((len(rows), d))
    for i, bh in enumerate(heads):
        idx = np.nonzero(rows // N == bh)[0]
        ref[idx] = exact.attention(host64[0][0, i][local[idx] % N], host64[1][0, i], host64[2][0, i], s)
    rel, cos = rel_l2_cos(got, ref)
    worst = float(row_rel_l2(got, ref).max())
    print(f"[bf16 sweep B{B} H{H} N{N} d{d}] rel-L2 {rel:.3e} cos {cos:.8f} worst row {worst:.3e}", flush=True)
    assert rel <= REL_MAX and cos >= COS_MIN and worst <= ROW_REL_MAX, (rel, cos, worst)
