"""Every forward route on shapes chosen at the launch rules' boundaries, against
the oracle on sampled rows (codes, block exponents, row reference and
denominator through the test entry point; O and LSE through the forward).

The shapes: exactly one full round of eight-wave workgroups; one workgroup past
a round and a last round of 64 (both take the four-wave tail launch on the
plain route, eight waves on the causal and FP8 routes); a last round of 224
(eight waves); more than five rounds; sequence lengths that are odd multiples
of 128 (four-wave launch), with batch > 1; the longest sequence below which
the grid leaves CUs idle; d = 64 grids of eight-wave workgroups (two per CU), the causal
route's among them; and the smallest problem.  Rows: the first and last
of the tensor and of a head, and seeded random ones.  Also the largest shapes of
the paper's D128 and D64 tables, which the benchmark times."""
import numpy as np
import pytest
import torch

import workloads
from test_gpu_forward import _run_and_check, _run_fp8, _run_guarded

pytestmark = pytest.mark.gpu

SHAPES = [  # B, H, N, d
    (1, 32, 2048, 128),    # 256 eight-wave workgroups: one full round
    (1, 257, 256, 128),    # 257: one past a round (tail rule)
    (5, 64, 256, 128),     # 320: last round 64 (tail rule)
    (2, 40, 1536, 128),    # 480: last round 224 (eight waves)
    (1, 1290, 256, 128),   # 1290: six rounds (eight waves)
    (3, 7, 1664, 128),     # N = 13 x 128: four-wave launch
    (2, 3, 4224, 64),      # N = 33 x 128, d = 64 (four waves per SIMD)
    (1, 3, 12288, 128),    # 144 workgroups: fewer than the CUs
    (1, 6, 8320, 64),      # N = 65 x 128
    (1, 16, 4096, 64),     # d = 64, 256 eight-wave workgroups: two per CU (causal: four-wave)
    (1, 768, 1024, 64),    # d = 64, 3072 eight-wave workgroups: the causal route takes them too
    (1, 1, 128, 128),      # one tile
]


def _inputs(B, H, N, d):
    g = torch.Generator().manual_seed(B * 1000003 + H * 1009 + N * 7 + d)
    q, k, v = (torch.randn(B, H, N, d, generator=g).to(torch.bfloat16) for _ in range(3))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    rows = np.random.default_rng(N + H).integers(0, B * H * N, 40)
    rows = np.unique(np.concatenate([rows, [0, N - 1, B * H * N - N, B * H * N - 1]]))
    return host64, (q.cuda(), k.cuda(), v.cuda()), rows


@pytest.mark.parametrize("B,H,N,d", SHAPES)
def test_every_route_at_launch_boundaries(B, H, N, d):
    import paper_2609_04105_amd as fa
    host64, dev, rows = _inputs(B, H, N, d)
    label = f"sweep B{B} H{H} N{N} d{d}"
    _run_and_check(fa, host64, dev, rows, label)
    _run_and_check(fa, host64, dev, rows, label + " causal", causal=True, lse=True)
    _run_and_check(fa, host64, dev, rows, label + " ex2 4", ex2_pairs=4)
    _run_guarded(fa, host64, dev, rows, label + " guard", 110, 16)
    _run_fp8(fa, host64, dev, rows, label + " fp8")


@pytest.mark.parametrize("H,N,d", [(24, 32768, 128), (64, 32768, 64)])
def test_paper_largest_shapes_sampled_rows(H, N, d):
    """The largest shapes of the paper's D128 and D64 tables (B1), in the launch the
    benchmark times (eight-wave workgroups at d = 128; 128-query workgroups at four
    waves per SIMD at d = 64): bf16 N(0,1) inputs drawn on the GPU, 24 rows from six
    heads (the first and last of the sequence among them) against the oracle."""
    import paper_2609_04105_amd as fa
    g = torch.Generator(device="cuda").manual_seed(N + H + d)
    q, k, v = (torch.randn((1, H, N, d), device="cuda", generator=g).to(torch.bfloat16) for _ in range(3))
    rng = np.random.default_rng(H + d)
    heads = np.unique(np.concatenate([[0, H - 1], rng.integers(0, H, 4)]))
    rows = np.unique(np.concatenate([h * N + np.concatenate([[0, N - 1], rng.integers(0, N, 3)]) for h in heads]))
    sel = torch.from_numpy(np.unique(heads)).cuda()
    # the oracle sees only the heads the rows touch, renumbered 0..len(heads)-1
    host64 = tuple(workloads.as_f64(t[:, sel].cpu()) for t in (q, k, v))
    remap = {int(h): i for i, h in enumerate(np.unique(heads))}
    local = np.array([remap[int(r // N)] * N + int(r % N) for r in rows])
    print(f"[paper shape B1 H{H} N{N} d{d}] rows={len(rows)} heads={len(heads)}", flush=True)
    out = fa.forward_mxfp4(*fa.quantize_qkv(q, k, v))
    torch.cuda.synchronize()
    got = out.reshape(-1, d)[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
    from parity import check_output, oracle_rows
    ref = oracle_rows(*host64, local, 1.0 / np.sqrt(d), want_codes=False)
    check_output(got, ref["O"], f"paper shape B1 H{H} N{N} d{d}")
