"""GPU parity of the MXFP4 quantizer: bit-exact codes and E8M0 bytes against the oracle."""
import numpy as np
import pytest
import torch

import workloads
from oracle import mxfp4

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fa():
    import paper_2609_04105_amd as fa
    return fa


def _check(fa, x_cpu, axis):
    cg, sg = fa.quantize_mxfp4(x_cpu.cuda(), axis=axis)
    co, so = mxfp4.quantize(workloads.as_f64(x_cpu), axis=axis)
    assert np.array_equal(sg.cpu().numpy(), so), "scale bytes differ"
    assert np.array_equal(cg.cpu().numpy(), co), "code bytes differ"


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("axis", [-1, -2])
def test_ragged_random(fa, dtype, axis):
    # 3 x 96 x 160: 1440 (axis -1) or 1440 (axis -2) blocks, not a multiple of the 256-thread launch
    g = torch.Generator().manual_seed(100)
    x = (torch.randn(3, 96, 160, generator=g) * torch.exp2(torch.randint(-6, 6, (3, 96, 160), generator=g))).to(dtype)
    _check(fa, x, axis)


@pytest.mark.parametrize("shape", [(3, 96, 192), (2, 256, 64), (1, 352, 128), (2, 512, 128)])
def test_staged_bf16_vt(fa, shape):
    """bf16 V^T with whole 64-column groups takes the staged kernel: ragged last
    groups of blocks (96 and 352 rows: 3 and 11 blocks per column, scale bytes
    stored one by one) and whole ones (8-byte scale stores), one to three column
    groups, values over 40 binades."""
    g = torch.Generator().manual_seed(shape[1] + 3 * shape[2])
    x = (torch.randn(*shape, generator=g) * torch.exp2(torch.randint(-20, 20, shape, generator=g))).to(torch.bfloat16)
    _check(fa, x, -2)


@pytest.mark.parametrize("axis", [-1, -2])
def test_adversarial_blocks(fa, axis):
    blocks = []
    mags = torch.tensor([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])
    blocks.append(torch.cat([mags, -mags, mags / 6 * 4, -mags / 3]))                # exact table values
    mids = torch.tensor([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0])
    blocks.append(torch.cat([mids, mids / 2, -mids / 4, mids * 2 / 3]))             # rounding ties
    blocks.append(torch.zeros(32))                                                  # zero block
    z = torch.zeros(32)
    z[3] = -0.0
    blocks.append(z)                                                                # signed zero
    blocks.append(torch.full((32,), 2.0 ** -140))                                   # below E8M0 range
    blocks.append(torch.full((32,), 3.0e38))                                        # near fp32 max
    w = torch.ones(32)
    w[0] = 2.0 ** 30
    blocks.append(w * torch.linspace(-1, 1, 32))                                    # wide dynamic range
    nan = torch.randn(32, generator=torch.Generator().manual_seed(1))
    nan[5] = float("nan")
    blocks.append(nan)
    inf = torch.randn(32, generator=torch.Generator().manual_seed(2))
    inf[9] = float("inf")
    blocks.append(inf)
    g = torch.Generator().manual_seed(3)
    for _ in range(23):
        blocks.append(torch.randn(32, generator=g) * float(2.0 ** torch.randint(-20, 20, (1,), generator=g)))
    x = torch.stack(blocks)                   # [32 blocks, 32]
    if axis == -2:
        x = x.T.contiguous()                  # blocks along rows
    _check(fa, x.to(torch.float32).reshape(1, *x.shape), axis)


def _adversarial_bf16_blocks():
    """32 blocks of 32 bf16 values: table values, rounding ties, zero and signed
    zero, subnormals, amplitudes clamped at either end of the E8M0 range,
    non-finite values and random blocks over 40 binades."""
    mags = torch.tensor([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])
    mids = torch.tensor([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0])
    blocks = [torch.cat([mags, -mags, mags / 6 * 4, -mags / 3]),
              torch.cat([mids, mids / 2, -mids / 4, mids * 2 / 3]),
              torch.cat([mids * 3 / 8, -mids * 5 / 16, mids / 12, mids * 7 / 24]),
              torch.zeros(32)]
    z = torch.zeros(32)
    z[3] = -0.0
    z[17] = -0.0
    blocks.append(z)
    blocks.append(torch.linspace(-1, 1, 32) * 2.0 ** -128)                 # subnormal bf16
    blocks.append(torch.full((32,), 2.0 ** -131) * torch.arange(32))          # amplitude below 2^-127
    blocks.append(torch.linspace(-1, 1, 32) * 3.0e38)                        # amplitude above 2^127
    w = torch.ones(32)
    w[0] = 2.0 ** 30
    blocks.append(w * torch.linspace(-1, 1, 32))
    nan = torch.randn(32, generator=torch.Generator().manual_seed(1))
    nan[5] = float("nan")
    blocks.append(nan)
    inf = torch.randn(32, generator=torch.Generator().manual_seed(2))
    inf[9] = -float("inf")
    blocks.append(inf)
    g = torch.Generator().manual_seed(3)
    while len(blocks) < 32:
        blocks.append(torch.randn(32, generator=g) * float(2.0 ** torch.randint(-20, 20, (1,), generator=g)))
    return torch.stack(blocks).to(torch.bfloat16)                            # [32 blocks, 32]


@pytest.mark.parametrize("axis,cols", [(-1, 32), (-2, 8), (-2, 64)])
def test_adversarial_blocks_bf16(fa, axis, cols):
    """The bf16 kernels: one block per row (axis -1), or four blocks of 32 rows
    down each column (axis -2): 8 columns take the per-thread kernel, 64 columns
    the kernel that stages its codes in LDS (the 32 blocks repeated with
    alternating signs)."""
    x = _adversarial_bf16_blocks()
    if axis == -1:
        x = x.reshape(1, 32, 32)
    else:                                      # block (g, c) = rows 32 g .. 32 g + 31 of column c
        reps = 4 * cols // 32
        x = torch.cat([x * (-1) ** k for k in range(reps)])
        x = x.reshape(4, cols, 32).permute(0, 2, 1).reshape(1, 128, cols).contiguous()
    _check(fa, x, axis)


@pytest.mark.parametrize("name", list(workloads.WORKLOADS))
def test_workload_operands(fa, name):
    """Bit-exact on the workloads: every block for small ones; for large ones the
    sampled query rows of Q and K and two full heads of V."""
    w = workloads.WORKLOADS[name]
    q, k, v = workloads.generate(w)
    qg, kg, vg = q.cuda(), k.cuda(), v.cuda()
    ops = fa.quantize_qkv(qg, kg, vg)
    host = [t.cpu().numpy() for t in ops]
    if w.all_rows:
        qc, qs = mxfp4.quantize(workloads.as_f64(q), axis=-1)
        kc, ks = mxfp4.quantize(workloads.as_f64(k), axis=-1)
        vc, vs = mxfp4.quantize(workloads.as_f64(v), axis=-2)
        for got, ref in zip(host, (qc, qs, kc, ks, vc, vs)):
            assert np.array_equal(got, ref)
        return
    rows = workloads.sampled_rows(w)
    b, h, i = rows // (w.H * w.N), (rows // w.N) % w.H, rows % w.N
    for x, cg, sg in ((q, host[0], host[1]), (k, host[2], host[3])):
        x64 = workloads.as_f64(x[torch.from_numpy(b), torch.from_numpy(h), torch.from_numpy(i)])
        c_ref, s_ref = mxfp4.quantize(x64, axis=-1)
        assert np.array_equal(cg[b, h, i], c_ref) and np.array_equal(sg[b, h, i], s_ref)
    for bh in (0, w.B * w.H - 1):
        bb, hh = divmod(bh, w.H)
        c_ref, s_ref = mxfp4.quantize(workloads.as_f64(v[bb, hh]), axis=-2)
        assert np.array_equal(host[4][bb, hh], c_ref) and np.array_equal(host[5][bb, hh], s_ref)


@pytest.mark.parametrize("axis", [-1, -2])
@pytest.mark.parametrize("rows", [128, 1024, 4096])
def test_anchor_order(fa, axis, rows):
    """fp4attn_quantize_mxfp4_anchored equals the plain quantizer applied to the
    rows in the oracle's anchor order (Sec. "Fix 3")."""
    from oracle import guard
    g = torch.Generator().manual_seed(rows + 7 * axis)
    x = torch.randn(2, rows, 64, generator=g).to(torch.bfloat16)
    perm = guard.anchor_permutation(rows)
    cg, sg = fa.quantize_mxfp4(x.cuda(), axis=axis, n_anchor=128)
    co, so = mxfp4.quantize(workloads.as_f64(x)[:, perm], axis=axis)
    assert np.array_equal(sg.cpu().numpy(), so) and np.array_equal(cg.cpu().numpy(), co)


def _check8(fa, x_cpu, axis):
    from oracle import fp8pv
    cg, sg = fa.quantize_mxfp8(x_cpu.cuda(), axis=axis)
    co, so = fp8pv.quantize(workloads.as_f64(x_cpu), axis=axis)
    assert np.array_equal(sg.cpu().numpy(), so), "MXFP8 scale bytes differ"
    assert np.array_equal(cg.cpu().numpy(), co), "MXFP8 code bytes differ"


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("axis", [-1, -2])
def test_mxfp8_ragged_random(fa, dtype, axis):
    g = torch.Generator().manual_seed(101)
    x = (torch.randn(3, 96, 160, generator=g) * torch.exp2(torch.randint(-20, 20, (3, 96, 160), generator=g))).to(dtype)
    _check8(fa, x, axis)


@pytest.mark.parametrize("axis", [-1, -2])
def test_mxfp8_adversarial_blocks(fa, axis):
    """Ties of the E4M3 grid, subnormal payloads, an exact 448 maximum, values just
    above it (the next power of two takes over), zeros, negative zero, NaN and
    infinities."""
    from oracle import fp8pv
    grid = torch.tensor(fp8pv.E4M3, dtype=torch.float64)
    mids = ((grid[1:] + grid[:-1]) / 2)[:32]
    blocks = [
        torch.cat([torch.tensor([448.0]), mids[:31]]),                       # ties, amplitude 2^0
        torch.cat([torch.tensor([448.0]), grid[1:32] * 0.75]),               # subnormal payloads
        torch.cat([torch.tensor([449.0]), -mids[:31]]),                      # just above 448
        torch.zeros(32),
        torch.cat([torch.tensor([-0.0, 1.0]), torch.zeros(30)]),
        torch.cat([torch.tensor([float("nan")]), torch.ones(31)]),
        torch.cat([torch.tensor([float("inf")]), torch.ones(31)]),
        torch.linspace(-1e-3, 1e-3, 32),
    ]
    x = torch.stack(blocks).to(torch.float32).reshape(1, 8, 32).repeat(1, 4, 1)   # [1, 32 rows, 32 cols]
    if axis == -2:
        x = x.transpose(-1, -2).contiguous()
    _check8(fa, x, axis)


@pytest.mark.parametrize("shape", [(3, 96, 192), (2, 256, 64), (1, 352, 128), (2, 512, 128)])
def test_mxfp8_staged_bf16(fa, shape):
    """bf16 V^T with whole 64-column groups takes the staged kernel: a ragged
    last group of blocks (96 rows) and full ones, values over 40 binades."""
    g = torch.Generator().manual_seed(shape[1] + shape[2])
    x = (torch.randn(*shape, generator=g) * torch.exp2(torch.randint(-20, 20, shape, generator=g))).to(torch.bfloat16)
    _check8(fa, x, -2)


def test_mxfp8_adversarial_blocks_bf16_staged(fa):
    """The adversarial blocks rounded to bf16, one per column of a 64-column
    matrix, through the staged V^T kernel."""
    from oracle import fp8pv
    grid = torch.tensor(fp8pv.E4M3, dtype=torch.float64)
    mids = ((grid[1:] + grid[:-1]) / 2)[:32]
    blocks = torch.stack([
        torch.cat([torch.tensor([448.0]), mids[:31]]),
        torch.cat([torch.tensor([448.0]), grid[1:32] * 0.75]),
        torch.cat([torch.tensor([480.0]), -mids[:31]]),                      # above 448 in bf16
        torch.zeros(32),
        torch.cat([torch.tensor([-0.0, 1.0]), torch.zeros(30)]),
        torch.cat([torch.tensor([float("nan")]), torch.ones(31)]),
        torch.cat([torch.tensor([float("inf")]), torch.ones(31)]),
        torch.linspace(-1e-3, 1e-3, 32),
    ]).to(torch.float32)
    x = blocks[torch.arange(64) % 8].transpose(0, 1).reshape(1, 32, 64).to(torch.bfloat16).contiguous()
    _check8(fa, x, -2)


def test_mxfp8_workload_v(fa):
    from oracle import fp8pv
    q, k, v = workloads.generate("outlier_b2h16_n4096_d128")
    cg, sg = fa.quantize_mxfp8(v.cuda(), axis=-2)
    co, so = fp8pv.quantize(workloads.as_f64(v), axis=-2)
    assert np.array_equal(sg.cpu().numpy(), so) and np.array_equal(cg.cpu().numpy(), co)


# (batch, rows, cols): both extents multiples of 32; cols a multiple of 64 or not
# (the staged V^T kernel or the per-thread one), groups of eight V^T blocks whole
# or ragged, one to three 64-column groups, single rows and single blocks
SWEEP_SHAPES = [(1, 32, 32), (1, 32, 64), (2, 64, 96), (3, 96, 128), (1, 160, 192), (2, 224, 64), (1, 256, 160),
                (4, 288, 128), (1, 512, 32), (2, 800, 64), (1, 1056, 128), (3, 32, 320)]


@pytest.mark.parametrize("shape", SWEEP_SHAPES)
def test_quantizer_shape_sweep(fa, shape):
    """MXFP4 (both axes, bf16 and fp32 inputs) and MXFP8 (bf16 and fp32) against the
    oracle, bit for bit, over values spanning 24 binades with a few zero and tiny
    blocks; with rows a multiple of 128 also the anchored form."""
    from oracle import fp8pv, guard
    B, R, C = shape
    g = torch.Generator().manual_seed(B * 1009 + R * 31 + C)
    x = torch.randn(B, R, C, generator=g) * torch.exp2(torch.randint(-12, 12, (B, R, C), generator=g).float())
    x[:, :, :32] *= (torch.rand(B, R, 1, generator=g) > 0.1).float()      # some zero blocks along a row
    x[:, 0, :] *= 2.0 ** -120                                             # a row of tiny values
    for dtype in (torch.bfloat16, torch.float32):
        xd = x.to(dtype)
        for axis in (-1, -2):
            _check(fa, xd, axis)
            _check8(fa, xd, axis)
        if R % 128 == 0:
            perm = guard.anchor_permutation(R)
            for axis in (-1, -2):
                cg, sg = fa.quantize_mxfp4(xd.cuda(), axis=axis, n_anchor=128)
                co, so = mxfp4.quantize(workloads.as_f64(xd)[:, perm], axis=axis)
                assert np.array_equal(sg.cpu().numpy(), so) and np.array_equal(cg.cpu().numpy(), co), (dtype, axis)
