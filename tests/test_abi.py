"""CPU checks of the C-ABI boundary: the library loads, exports every entry
point declared in include/fp4attn.h, and rejects bad arguments before any HIP
call (no compute is launched here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fp4attn.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fp4attn_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2609_04105_amd as fa
    return fa.lib


def test_header_declares_the_boundary():
    names = _declared()
    assert {"fp4attn_quantize_mxfp4", "fp4attn_forward_mxfp4", "fp4attn_forward_bf16"} <= set(names)


def test_every_declared_symbol_is_exported(lib):
    raw = ctypes.CDLL(lib._name)
    for name in _declared():
        assert hasattr(raw, name), name


def test_binding_covers_every_symbol():
    from paper_2609_04105_amd import _lib
    assert set(_declared()) == set(_lib.SIGNATURES)


def test_status_strings(lib):
    assert lib.fp4attn_status_string(0) == b"ok"
    assert lib.fp4attn_status_string(2) == b"unsupported configuration"
    assert lib.fp4attn_status_string(99) == b"unknown status"
    assert lib.fp4attn_abi_version() >> 16 == 2


FAKE = [ctypes.c_void_p(4096 * (i + 1)) for i in range(8)]   # aligned, never dereferenced


def test_forward_validation(lib):
    f = lib.fp4attn_forward_mxfp4
    assert f(None, *FAKE[:5], 1, 1, 128, 64, 0.125, 1.5, 1.2, FAKE[6], 0, None) == 1
    assert b"q_codes" in lib.fp4attn_last_error()
    assert f(*FAKE[:6], 0, 1, 128, 64, 0.125, 1.5, 1.2, FAKE[6], 0, None) == 1
    assert f(*FAKE[:6], 1, 1, 100, 64, 0.125, 1.5, 1.2, FAKE[6], 0, None) == 1
    assert f(*FAKE[:6], 1, 1, 64, 64, 0.125, 1.5, 1.2, FAKE[6], 0, None) == 1
    assert f(*FAKE[:6], 1, 1, 128, 96, 0.125, 1.5, 1.2, FAKE[6], 0, None) == 2
    assert f(*FAKE[:6], 1, 1, 128, 64, float("nan"), 1.5, 1.2, FAKE[6], 0, None) == 1
    assert f(*FAKE[:6], 1, 1, 128, 64, 0.125, -1.0, 1.2, FAKE[6], 0, None) == 1
    assert f(*FAKE[:6], 1, 1, 128, 64, 0.125, 1.5, float("inf"), FAKE[6], 0, None) == 1
    assert f(*FAKE[:6], 1, 1, 128, 64, 0.125, 1.5, 1.2, FAKE[6], 3, None) == 1
    assert f(*FAKE[:6], 1, 1, 128, 64, 0.125, 1.5, 1.2, ctypes.c_void_p(4100), 0, None) == 1
    assert f(*FAKE[:6], 1 << 20, 1 << 10, 1 << 12, 64, 0.125, 1.5, 1.2, FAKE[6], 0, None) == 1
    # sizes whose products would overflow 64 bits are refused, not wrapped
    for B, H, N in ((1 << 62, 1 << 62, 128), (1, 1, 1 << 62), (1 << 40, 1, 1 << 40), (4097, 4097, 128)):
        assert f(*FAKE[:6], B, H, N, 64, 0.125, 1.5, 1.2, FAKE[6], 0, None) == 1, (B, H, N)
    # one head's operands must stay addressable with 32-bit offsets: N up to 2^22 keys
    assert f(*FAKE[:6], 1, 1, (1 << 22) + 128, 128, 0.125, 1.5, 1.2, FAKE[6], 0, None) == 2


def test_quantize_and_bf16_validation(lib):
    q = lib.fp4attn_quantize_mxfp4
    assert q(FAKE[0], 0, 1, 4, 48, 1, FAKE[1], FAKE[2], None) == 1     # cols not /32
    assert q(FAKE[0], 0, 1, 48, 4, 0, FAKE[1], FAKE[2], None) == 1     # rows not /32
    assert q(FAKE[0], 2, 1, 4, 64, 1, FAKE[1], FAKE[2], None) == 1     # dtype
    assert q(FAKE[0], 0, 1, 4, 64, 2, FAKE[1], FAKE[2], None) == 1     # axis
    assert q(FAKE[0], 0, 0, 4, 64, 1, FAKE[1], FAKE[2], None) == 1     # batch
    for batch, rows, cols in ((1 << 62, 1 << 62, 64), (1, 1 << 62, 1 << 62), (1 << 20, 1 << 20, 1 << 12)):
        assert q(FAKE[0], 0, batch, rows, cols, 1, FAKE[1], FAKE[2], None) == 1, (batch, rows, cols)
        assert q(FAKE[0], 0, batch, cols, rows, 0, FAKE[1], FAKE[2], None) == 1, (batch, rows, cols)
    q8 = lib.fp4attn_quantize_mxfp8
    assert q8(FAKE[0], 0, 1, 4, 48, 1, FAKE[1], FAKE[2], None) == 1    # cols not /32
    assert q8(None, 0, 1, 4, 64, 1, FAKE[1], FAKE[2], None) == 1
    qa = lib.fp4attn_quantize_mxfp4_anchored
    assert qa(FAKE[0], 0, 1, 256, 64, 1, 0, FAKE[1], FAKE[2], None) == 1     # n_anchor < 1
    assert qa(FAKE[0], 0, 1, 256, 64, 1, 96, FAKE[1], FAKE[2], None) == 1    # does not divide rows
    assert qa(FAKE[0], 0, 1, 256, 64, 2, 128, FAKE[1], FAKE[2], None) == 1   # axis
    b = lib.fp4attn_forward_bf16
    assert b(*FAKE[:3], 1, 1, 128, 80, 0.125, FAKE[4], 0, None) == 2
    assert b(None, *FAKE[1:3], 1, 1, 128, 64, 0.125, FAKE[4], 0, None) == 1
    d = lib.fp4attn_debug_directp_mxfp4
    assert d(*FAKE[:6], 1, 1, 128, 64, 0.125, None, FAKE[6], 0, FAKE[7], -1, *FAKE[:4], None, None) == 1  # n_rows < 0
    assert d(*FAKE[:6], 1, 1, 128, 64, 0.125, None, FAKE[6], 0, FAKE[7], 1, *FAKE[:4], ctypes.c_void_p(4096 + 8),
             None) == 1                                                 # misaligned wg_clock
    m = lib.fp4attn_debug_mfma_stream
    assert m(FAKE[0], FAKE[1], 0, 10, FAKE[2], None) == 1              # blocks < 1
    assert m(FAKE[0], FAKE[1], 65536, 10, FAKE[2], None) == 1          # blocks > 65535
    assert m(FAKE[0], FAKE[1], 4, 0, FAKE[2], None) == 1               # iters < 1
    assert m(None, FAKE[1], 4, 10, FAKE[2], None) == 1
    assert m(FAKE[0], FAKE[1], 4, 10, ctypes.c_void_p(4100), None) == 1  # misaligned out


def test_forward_options(lib):
    from paper_2609_04105_amd import _lib
    o = _lib.ForwardOptions()
    assert ctypes.sizeof(o) == 48
    lib.fp4attn_forward_options_init(ctypes.byref(o))
    assert (o.struct_size, o.affine_a, o.ex2_pairs) == (48, 1.5, 0) and abs(o.affine_b - 1.2) < 1e-6
    assert (o.guard, o.guard_margin, o.guard_shift, o.causal, o.pv_fp8, o.lse) == (0, 110, 16, 0, 0, None)
    e = lib.fp4attn_forward_mxfp4_ex
    for kx in (3, 5, 32, -1):
        o.ex2_pairs = kx
        assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 1
    o.ex2_pairs = 4
    o.struct_size = 12
    assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 1
    o.struct_size = 48
    o.guard = 1
    for M, L in ((110, 17), (-1, 0), (0, -1)):
        o.guard_margin, o.guard_shift = M, L
        assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 1
    o.guard_margin, o.guard_shift = 110, 16
    o.ex2_pairs = 2
    assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 2     # guard: 0, 4, 16 only
    o.guard, o.ex2_pairs = 2, 4
    assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 1
    o.guard = 0
    o.causal = 1
    o.ex2_pairs = 2
    assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 2     # causal: 0, 4, 16 only
    o.ex2_pairs, o.guard = 4, 1
    assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 2     # causal with guard
    o.guard, o.causal = 0, 3
    assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 1
    o.causal, o.lse = 0, 4096 + 4
    assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 1     # misaligned lse
    o.lse = None
    o.pv_fp8, o.ex2_pairs = 1, 4
    assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 2     # fp8 P/V with ex2
    o.ex2_pairs, o.guard = 0, 1
    assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 2     # fp8 P/V with guard
    o.guard, o.pv_fp8 = 0, 2
    assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 1
    o.pv_fp8, o.ex2_pairs = 0, 4
    o.affine_a = 0.0
    assert e(*FAKE[:6], 1, 1, 128, 64, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 1
    o.affine_a = 1.5
    assert e(*FAKE[:6], 1, 1, 128, 80, 0.125, ctypes.byref(o), FAKE[6], 0, None) == 2     # d = 80
    assert e(None, *FAKE[1:6], 1, 1, 128, 64, 0.125, None, FAKE[6], 0, None) == 1


def test_binding_requires_one_device_per_call():
    """The binding runs each call with the operands' device current; operands on
    two devices are refused before anything reaches the library."""
    import torch
    from paper_2609_04105_amd import api
    a, b = torch.zeros(2), torch.zeros(2, device="meta")
    assert api._same_device(a, a) == a.device
    with pytest.raises(ValueError, match="share a device"):
        api._same_device(a, a, b)
