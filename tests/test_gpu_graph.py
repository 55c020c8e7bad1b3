"""The forwards inside a captured HIP graph (torch.cuda.graph): the C-ABI
launches on the caller's stream, sets no memory and allocates nothing, so a
launch-bound caller can capture a sequence of calls once and replay it.
Every replay is checked bit for bit against the eager result, with eager work
and synchronisations between the replays."""
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fa():
    import paper_2609_04105_amd as fa
    return fa


@pytest.mark.parametrize("name", ["tiny_b1h1_n128_d64", "small_b1h8_n1024_d64"])
def test_forward_graph_replays_match_eager(fa, name):
    w = workloads.WORKLOADS[name]
    q, k, v = (t.cuda() for t in workloads.generate(w))
    q16, k16, v16 = (t.to(torch.bfloat16) for t in (q, k, v))
    ops = fa.quantize_qkv(q, k, v)
    lse = torch.empty((w.B, w.H, w.N), dtype=torch.float32, device="cuda")
    outs = [torch.empty((w.B, w.H, w.N, w.d), dtype=torch.float32, device="cuda") for _ in range(3)]
    out16 = torch.empty_like(outs[0])

    def calls():
        fa.forward_mxfp4(*ops, out=outs[0])
        fa.forward_mxfp4(*ops, out=outs[1], causal=True, lse=lse)
        fa.forward_mxfp4(*ops, out=outs[2], ex2_pairs=4)
        fa.forward_bf16(q16, k16, v16, out=out16)

    calls()
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs] + [out16.clone(), lse.clone()]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm the capture stream, as torch recommends
        calls()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        calls()
    for replay in range(4):
        for o in outs + [out16, lse]:
            o.fill_(float("nan"))          # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (got, want) in enumerate(zip(outs + [out16, lse], ref)):
            assert torch.equal(got, want), f"{name}: replay {replay}, output {i} differs from eager"
        calls()                            # eager calls between replays leave the same results
        torch.cuda.synchronize()
        assert torch.equal(outs[0], ref[0])
