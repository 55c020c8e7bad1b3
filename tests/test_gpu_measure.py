"""GPU checks of the measurement hooks: the FP4 matrix-unit stream whose rate
bench.py reports as the sustained ceiling beside the spec peak."""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("a_byte,b_byte,per_product", [(0x22, 0x22, 64.0), (0x22, 0x44, 128.0), (0x2A, 0x22, 0.0)])
def test_mfma_stream_sums_exactly(a_byte, b_byte, per_product):
    """The matrix-unit stream used as the measured ceiling computes what it claims:
    E2M1 1.0 (0x2 nibbles) times 1.0 or 2.0 (0x4) over K = 64 adds 64 or 128 to
    every accumulator element per product; 1.0 and -1.0 (0xA) in alternate
    nibbles of A cancel in pairs."""
    import paper_2609_04105_amd as fa
    blocks, iters = 3, 5
    a = torch.full((blocks * 256 * 64,), a_byte, dtype=torch.uint8, device="cuda")
    b = torch.full((blocks * 256 * 64,), b_byte, dtype=torch.uint8, device="cuda")
    out, flop = fa.debug_mfma_stream(a, b, blocks, iters)
    torch.cuda.synchronize()
    assert flop == blocks * 4 * iters * 4 * 2 * 32 * 32 * 64
    expect = 4 * 16 * per_product * iters   # 4 accumulators x 16 elements per lane
    assert torch.equal(out, torch.full_like(out, expect))
