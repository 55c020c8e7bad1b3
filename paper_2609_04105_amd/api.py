"""Torch-facing wrappers of the C-ABI (argument marshalling only).

Shapes follow include/fp4attn.h.  Inputs must be contiguous CUDA (HIP) tensors;
outputs are allocated with torch unless passed in.  Work is enqueued on the
current torch stream of the tensors' device.
"""
import ctypes
import math

import torch

from ._lib import FP4ATTN_BF16, FP4ATTN_F32, ForwardOptions, check, lib

_DTYPES = {torch.float32: FP4ATTN_F32, torch.bfloat16: FP4ATTN_BF16}


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def _stream(t):
    # the raw handle of torch's current stream on t's device (the same value as
    # torch.cuda.current_stream(device).cuda_stream, without building a Stream)
    return ctypes.c_void_p(torch._C._cuda_getCurrentRawStream(t.get_device()))


def _same_device(*tensors):
    """The one device every tensor of a call lives on (the library launches on the
    current HIP device, so each call runs with that device made current)."""
    dev = tensors[0].device
    for t in tensors[1:]:
        if t.device != dev:
            raise ValueError(f"tensors of one call must share a device: {dev} and {t.device}")
    return dev


def _launch(device, fn, *args):
    if device.index == torch.cuda.current_device():
        check(fn(*args))
        return
    with torch.cuda.device(device):
        check(fn(*args))


def _need(t, name, dtype=None, ndim=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype not in (dtype if isinstance(dtype, tuple) else (dtype,)):
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if ndim is not None and t.ndim != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got shape {tuple(t.shape)}")


def quantize_mxfp4(x, axis=-1, n_anchor=0):
    """MXFP4 codes and E8M0 scales of ``x`` [..., rows, cols] (fp32 or bf16).

    axis=-1: blocks of 32 along cols -> codes [..., rows, cols/2], scales [..., rows, cols/32].
    axis=-2: blocks along rows, stored transposed -> codes [..., cols, rows/2], scales [..., cols, rows/32].
    n_anchor > 0: the rows are taken in anchor order (fp4attn_quantize_mxfp4_anchored).
    """
    _need(x, "x", (torch.float32, torch.bfloat16))
    if x.dim() < 2:
        raise ValueError("x needs at least two dimensions")
    lead = tuple(x.shape[:-2])
    rows, cols = x.shape[-2:]
    batch = math.prod(lead) if lead else 1
    if axis in (-1, x.dim() - 1):
        c_axis, cshape, sshape = 1, lead + (rows, cols // 2), lead + (rows, cols // 32)
    elif axis in (-2, x.dim() - 2):
        c_axis, cshape, sshape = 0, lead + (cols, rows // 2), lead + (cols, rows // 32)
    else:
        raise ValueError("axis must be -1 or -2")
    codes = torch.empty(cshape, dtype=torch.uint8, device=x.device)
    scales = torch.empty(sshape, dtype=torch.uint8, device=x.device)
    if n_anchor:
        _launch(x.device, lib.fp4attn_quantize_mxfp4_anchored, _ptr(x), _DTYPES[x.dtype], batch, rows, cols, c_axis,
                n_anchor, _ptr(codes), _ptr(scales), _stream(x))
    else:
        _launch(x.device, lib.fp4attn_quantize_mxfp4, _ptr(x), _DTYPES[x.dtype], batch, rows, cols, c_axis,
                _ptr(codes), _ptr(scales), _stream(x))
    return codes, scales


def quantize_mxfp8(x, axis=-1):
    """MXFP8 (E4M3 + E8M0 per 32) codes and scales of ``x`` [..., rows, cols], one
    code byte per value; axis as :func:`quantize_mxfp4`."""
    _need(x, "x", (torch.float32, torch.bfloat16))
    if x.dim() < 2:
        raise ValueError("x needs at least two dimensions")
    lead = tuple(x.shape[:-2])
    rows, cols = x.shape[-2:]
    batch = math.prod(lead) if lead else 1
    if axis in (-1, x.dim() - 1):
        c_axis, cshape, sshape = 1, lead + (rows, cols), lead + (rows, cols // 32)
    elif axis in (-2, x.dim() - 2):
        c_axis, cshape, sshape = 0, lead + (cols, rows), lead + (cols, rows // 32)
    else:
        raise ValueError("axis must be -1 or -2")
    codes = torch.empty(cshape, dtype=torch.uint8, device=x.device)
    scales = torch.empty(sshape, dtype=torch.uint8, device=x.device)
    _launch(x.device, lib.fp4attn_quantize_mxfp8, _ptr(x), _DTYPES[x.dtype], batch, rows, cols, c_axis, _ptr(codes),
            _ptr(scales), _stream(x))
    return codes, scales


def quantize_qkv(q, k, v, anchored=False, pv_fp8=False):
    """Operands of the forward: MXFP4 Q, K along d; V along the sequence
    (transposed), MXFP4 or, with ``pv_fp8``, MXFP8.  ``anchored``: K and V in the
    anchor key order of the guarded forward (128 anchors)."""
    n_anchor = 128 if anchored else 0
    qc, qs = quantize_mxfp4(q, axis=-1)
    kc, ks = quantize_mxfp4(k, axis=-1, n_anchor=n_anchor)
    if pv_fp8:
        if anchored:
            raise ValueError("the FP8 P/V route has no anchored form")
        vc, vs = quantize_mxfp8(v, axis=-2)
    else:
        vc, vs = quantize_mxfp4(v, axis=-2, n_anchor=n_anchor)
    return qc, qs, kc, ks, vc, vs


def _fp4_shape(q_codes):
    _need(q_codes, "q_codes", torch.uint8, 4)
    B, H, N, half_d = q_codes.shape
    return B, H, N, 2 * half_d


def _check_operands(B, H, N, d, ops, pv_fp8=False):
    names = ("q_codes", "q_scales", "k_codes", "k_scales", "vt_codes", "vt_scales")
    shapes = ((B, H, N, d // 2), (B, H, N, d // 32), (B, H, N, d // 2), (B, H, N, d // 32),
              (B, H, d, N if pv_fp8 else N // 2), (B, H, d, N // 32))
    for t, name, shape in zip(ops, names, shapes):
        _need(t, name, torch.uint8, 4)
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {shape}")


def _out(out, B, H, N, d, out_dtype, device):
    if out is None:
        return torch.empty((B, H, N, d), dtype=out_dtype, device=device)
    _need(out, "out", (torch.float32, torch.bfloat16), 4)
    if tuple(out.shape) != (B, H, N, d):
        raise ValueError(f"out has shape {tuple(out.shape)}, expected {(B, H, N, d)}")
    return out


def forward_options(affine_a=1.5, affine_b=1.2, ex2_pairs=0, guard=None, causal=False, lse=None, pv_fp8=False):
    """An fp4attn_forward_options struct: the library's defaults, then the given
    fields; ``guard`` = (margin, shift) turns the sampled guard on; ``lse`` is a
    contiguous fp32 GPU tensor [B, H, N] or None."""
    o = ForwardOptions()
    lib.fp4attn_forward_options_init(ctypes.byref(o))
    o.affine_a, o.affine_b, o.ex2_pairs = affine_a, affine_b, ex2_pairs
    if guard is not None:
        o.guard, (o.guard_margin, o.guard_shift) = 1, guard
    o.causal = 1 if causal else 0
    o.pv_fp8 = 1 if pv_fp8 else 0
    if lse is not None:
        _need(lse, "lse", torch.float32, 3)
        o.lse = lse.data_ptr()
    return o


def forward_mxfp4(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, softmax_scale=None,
                  affine_a=1.5, affine_b=1.2, out=None, out_dtype=torch.float32, ex2_pairs=None, guard=None,
                  causal=False, lse=None, pv_fp8=False):
    """Direct-P full-MXFP4 attention forward; returns O [B, H, N, d].

    ``ex2_pairs`` (0, 1, 2, 4, 8 or 16 of the 16 key pairs of each 32-key
    block take the native exponential), ``guard`` = (margin, shift) (the
    sampled guard; K and V from ``quantize_qkv(..., anchored=True)``),
    ``causal``, ``lse`` (an fp32 [B, H, N] tensor that receives the row
    normaliser) or ``pv_fp8`` (FP8 P and V; V from ``quantize_qkv(..., pv_fp8=True)``)
    select the extended entry point; otherwise the plain forward runs.
    """
    B, H, N, d = _fp4_shape(q_codes)
    ops = (q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales)
    _check_operands(B, H, N, d, ops, pv_fp8)
    out = _out(out, B, H, N, d, out_dtype, q_codes.device)
    dev = _same_device(*ops, out, *(() if lse is None else (lse,)))
    s = 1.0 / math.sqrt(d) if softmax_scale is None else softmax_scale
    if ex2_pairs is None and guard is None and not causal and lse is None and not pv_fp8:
        _launch(dev, lib.fp4attn_forward_mxfp4, *(_ptr(t) for t in ops), B, H, N, d, s, affine_a, affine_b, _ptr(out),
                _DTYPES[out.dtype], _stream(out))
    else:
        if lse is not None and tuple(lse.shape) != (B, H, N):
            raise ValueError(f"lse has shape {tuple(lse.shape)}, expected {(B, H, N)}")
        o = forward_options(affine_a, affine_b, ex2_pairs or 0, guard, causal, lse, pv_fp8)
        _launch(dev, lib.fp4attn_forward_mxfp4_ex, *(_ptr(t) for t in ops), B, H, N, d, s, ctypes.byref(o),
                _ptr(out), _DTYPES[out.dtype], _stream(out))
    return out


def attention_mxfp4(q, k, v, softmax_scale=None, causal=False, lse=None, ex2_pairs=None, guard=None,
                    pv_fp8=False, out=None, out_dtype=torch.float32):
    """Quantize ``q``, ``k``, ``v`` ([B, H, N, d], bf16 or fp32) and run the Direct-P
    forward in one call: MXFP4 Q and K; V in MXFP4 or, with ``pv_fp8``, MXFP8; K and
    V in anchor order when ``guard`` is given.  The quantized operands are not kept
    (use :func:`quantize_qkv` and :func:`forward_mxfp4` to reuse them)."""
    ops = quantize_qkv(q, k, v, anchored=guard is not None, pv_fp8=pv_fp8)
    return forward_mxfp4(*ops, softmax_scale=softmax_scale, out=out, out_dtype=out_dtype, ex2_pairs=ex2_pairs,
                         guard=guard, causal=causal, lse=lse, pv_fp8=pv_fp8)


def debug_directp_mxfp4(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, row_ids, softmax_scale=None,
                        affine_a=1.5, affine_b=1.2, out_dtype=torch.float32, wg_clock=False, ex2_pairs=0,
                        guard=None, causal=False, lse=False, pv_fp8=False):
    """Forward plus the Direct-P state of the (strictly ascending) flattened ``row_ids``.

    Returns a dict: out, p_codes [R, N/2] uint8 ([R, N] E4M3 bytes with
    ``pv_fp8``), block_exp [R, N/32] int16, row_m [R] int32, row_d [R] fp32,
    with ``lse`` also lse [B, H, N], and with ``wg_clock`` also wg_clock
    [B*H*N/128, 2] int64 (per workgroup: shader-clock cycles, 100 MHz ticks;
    rows past the launch's workgroup count stay zero).
    """
    B, H, N, d = _fp4_shape(q_codes)
    ops = (q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales)
    _check_operands(B, H, N, d, ops, pv_fp8)
    _need(row_ids, "row_ids", torch.int64, 1)
    R = row_ids.numel()   # 0: no dump, the launch is the plain forward kernel
    dev = _same_device(*ops, row_ids)
    out = torch.empty((B, H, N, d), dtype=out_dtype, device=dev)
    res = {
        "out": out,
        "p_codes": torch.empty((R, N if pv_fp8 else N // 2), dtype=torch.uint8, device=dev),
        "block_exp": torch.empty((R, N // 32), dtype=torch.int16, device=dev),
        "row_m": torch.empty((R,), dtype=torch.int32, device=dev),
        "row_d": torch.empty((R,), dtype=torch.float32, device=dev),
    }
    if wg_clock:
        res["wg_clock"] = torch.zeros((B * H * N // 128, 2), dtype=torch.int64, device=dev)
    if lse:
        res["lse"] = torch.empty((B, H, N), dtype=torch.float32, device=dev)
    s = 1.0 / math.sqrt(d) if softmax_scale is None else softmax_scale
    o = forward_options(affine_a, affine_b, ex2_pairs, guard, causal, res.get("lse"), pv_fp8)
    _launch(dev, lib.fp4attn_debug_directp_mxfp4, *(_ptr(t) for t in ops), B, H, N, d, s, ctypes.byref(o),
            _ptr(out), _DTYPES[out_dtype], _ptr(row_ids) if R else None, R, _ptr(res["p_codes"]),
            _ptr(res["block_exp"]), _ptr(res["row_m"]), _ptr(res["row_d"]),
            _ptr(res["wg_clock"]) if wg_clock else None, _stream(out))
    return res


def debug_mfma_stream(a_codes, b_codes, blocks, iters):
    """Sustained FP4 matrix-unit stream on given operands (fp4attn_debug_mfma_stream):
    ``blocks`` x 256 threads, each with 64 bytes of ``a_codes`` and of ``b_codes``
    (uint8, at least blocks * 256 * 64 bytes each); returns the per-thread
    accumulator sums [blocks * 256] fp32 and the flop count of the launch."""
    need = blocks * 256 * 64
    for t, name in ((a_codes, "a_codes"), (b_codes, "b_codes")):
        _need(t, name, torch.uint8)
        if t.numel() < need:
            raise ValueError(f"{name} holds {t.numel()} bytes, the launch reads {need}")
    dev = _same_device(a_codes, b_codes)
    out = torch.empty(blocks * 256, dtype=torch.float32, device=dev)
    _launch(dev, lib.fp4attn_debug_mfma_stream, _ptr(a_codes), _ptr(b_codes), blocks, iters, _ptr(out), _stream(out))
    return out, blocks * 4 * iters * 4 * 2.0 * 32 * 32 * 64


def forward_bf16(q, k, v, softmax_scale=None, out=None, out_dtype=torch.float32):
    """Same-design BF16 attention forward; q, k, v [B, H, N, d] bf16."""
    _need(q, "q", torch.bfloat16, 4)
    _need(k, "k", torch.bfloat16, 4)
    _need(v, "v", torch.bfloat16, 4)
    B, H, N, d = q.shape
    if tuple(k.shape) != (B, H, N, d) or tuple(v.shape) != (B, H, N, d):
        raise ValueError("q, k and v must all be [B, H, N, d]")
    out = _out(out, B, H, N, d, out_dtype, q.device)
    dev = _same_device(q, k, v, out)
    s = 1.0 / math.sqrt(d) if softmax_scale is None else softmax_scale
    _launch(dev, lib.fp4attn_forward_bf16, _ptr(q), _ptr(k), _ptr(v), B, H, N, d, s, _ptr(out), _DTYPES[out.dtype],
            _stream(out))
    return out
