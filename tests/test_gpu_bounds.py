"""Output bounds: every entry point writes exactly its outputs.  Each output is
handed over as the middle of a larger device buffer whose 4 KiB on either side
hold a fill pattern; after the call the pattern must be intact and the output
must equal what the call writes into a buffer of its own.  Shapes cover ragged
tails (N not a multiple of the workgroup's query tile), both head dimensions,
several heads and batches, and a launch whose last round is split into
smaller workgroups."""
import ctypes

import pytest
import torch

pytestmark = pytest.mark.gpu

PAD = 4096
FILL = 0xA5


@pytest.fixture(scope="module")
def fa():
    import paper_2609_04105_amd as fa
    return fa


class Guarded:
    """A ``shape``/``dtype`` tensor in the middle of a byte buffer with PAD
    pattern bytes before and after it."""

    def __init__(self, shape, dtype):
        n = torch.empty(shape, dtype=dtype).numel() * torch.empty((), dtype=dtype).element_size()
        self.buf = torch.full((PAD + n + PAD,), FILL, dtype=torch.uint8, device="cuda")
        self.t = self.buf[PAD:PAD + n].view(dtype).view(shape)

    def intact(self):
        return bool(torch.all(self.buf[:PAD] == FILL)) and bool(torch.all(self.buf[-PAD:] == FILL))


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


SHAPES = [(1, 3, 384, 128), (2, 5, 640, 64), (1, 1, 128, 64), (1, 24, 4096, 128), (1, 16, 4096, 64)]


@pytest.mark.parametrize("B,H,N,d", SHAPES)
def test_quantizers_write_only_their_outputs(fa, B, H, N, d):
    lib = fa.lib
    g = torch.Generator(device="cuda").manual_seed(B + H + N + d)
    x = torch.randn((B, H, N, d), device="cuda", generator=g).to(torch.bfloat16)
    f = fa.api._DTYPES[torch.bfloat16]
    cases = [  # (label, call, reference codes and scales, codes shape, scales shape)
        ("rows", lambda c, s: lib.fp4attn_quantize_mxfp4(_p(x), f, B * H, N, d, 1, _p(c), _p(s), None),
         fa.quantize_mxfp4(x, axis=-1), (B, H, N, d // 2), (B, H, N, d // 32)),
        ("columns", lambda c, s: lib.fp4attn_quantize_mxfp4(_p(x), f, B * H, N, d, 0, _p(c), _p(s), None),
         fa.quantize_mxfp4(x, axis=-2), (B, H, d, N // 2), (B, H, d, N // 32)),
        ("anchored rows", lambda c, s: lib.fp4attn_quantize_mxfp4_anchored(_p(x), f, B * H, N, d, 1, 128, _p(c),
                                                                          _p(s), None),
         fa.quantize_mxfp4(x, axis=-1, n_anchor=128), (B, H, N, d // 2), (B, H, N, d // 32)),
        ("anchored columns", lambda c, s: lib.fp4attn_quantize_mxfp4_anchored(_p(x), f, B * H, N, d, 0, 128, _p(c),
                                                                             _p(s), None),
         fa.quantize_mxfp4(x, axis=-2, n_anchor=128), (B, H, d, N // 2), (B, H, d, N // 32)),
        ("fp8 columns", lambda c, s: lib.fp4attn_quantize_mxfp8(_p(x), f, B * H, N, d, 0, _p(c), _p(s), None),
         fa.quantize_mxfp8(x, axis=-2), (B, H, d, N), (B, H, d, N // 32)),
    ]
    for label, call, (rc, rs), cshape, sshape in cases:
        print(f"[bounds quantize {label}] B{B} H{H} N{N} d{d}", flush=True)
        c, s = Guarded(cshape, torch.uint8), Guarded(sshape, torch.uint8)
        assert call(c.t, s.t) == 0
        torch.cuda.synchronize()
        assert c.intact() and s.intact(), f"{label}: bytes outside the outputs changed"
        assert torch.equal(c.t, rc) and torch.equal(s.t, rs), f"{label}: outputs differ from the plain call"


ROUTES = [("plain", {}), ("bf16 out", {"out_dtype": torch.bfloat16}), ("ex2", {"ex2_pairs": 4}),
          ("causal", {"causal": True, "lse": True}), ("lse", {"lse": True}), ("guard", {"guard": (110, 16)}),
          ("fp8", {"pv_fp8": True, "lse": True}), ("fp8 causal", {"pv_fp8": True, "causal": True})]


@pytest.mark.parametrize("B,H,N,d", SHAPES)
def test_forwards_write_only_their_outputs(fa, B, H, N, d):
    g = torch.Generator(device="cuda").manual_seed(7 * (B + H + N + d))
    q, k, v = (torch.randn((B, H, N, d), device="cuda", generator=g).to(torch.bfloat16) for _ in range(3))
    for label, opts in ROUTES:
        opts = dict(opts)
        print(f"[bounds forward {label}] B{B} H{H} N{N} d{d}", flush=True)
        ops = fa.quantize_qkv(q, k, v, anchored="guard" in opts, pv_fp8=opts.get("pv_fp8", False))
        out_dtype = opts.pop("out_dtype", torch.float32)
        want_lse = opts.pop("lse", False)
        o = Guarded((B, H, N, d), out_dtype)
        lse = Guarded((B, H, N), torch.float32) if want_lse else None
        fa.forward_mxfp4(*ops, out=o.t, lse=None if lse is None else lse.t, **opts)
        ref_lse = torch.empty((B, H, N), dtype=torch.float32, device="cuda") if want_lse else None
        ref = fa.forward_mxfp4(*ops, out_dtype=out_dtype, lse=ref_lse, **opts)
        torch.cuda.synchronize()
        assert o.intact(), f"{label}: bytes outside the output changed"
        assert torch.equal(o.t, ref), f"{label}: output differs from the plain call"
        if want_lse:
            assert lse.intact(), f"{label}: bytes outside lse changed"
            assert torch.equal(lse.t, ref_lse), f"{label}: lse differs from the plain call"

    print(f"[bounds forward bf16 kernel] B{B} H{H} N{N} d{d}", flush=True)
    for out_dtype in (torch.float32, torch.bfloat16):
        o = Guarded((B, H, N, d), out_dtype)
        fa.forward_bf16(q, k, v, out=o.t)
        ref = fa.forward_bf16(q, k, v, out_dtype=out_dtype)
        torch.cuda.synchronize()
        assert o.intact(), "BF16 kernel: bytes outside the output changed"
        assert torch.equal(o.t, ref), "BF16 kernel: output differs from the plain call"
