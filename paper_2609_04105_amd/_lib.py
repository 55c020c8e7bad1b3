"""ctypes loader for libfp4attn.so and the signatures of its C-ABI entry points."""
import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfp4attn.so")

FP4ATTN_OK = 0
FP4ATTN_F32 = 0
FP4ATTN_BF16 = 1

_c_p = ctypes.c_void_p
_i64 = ctypes.c_int64
_int = ctypes.c_int
_f32 = ctypes.c_float


class ForwardOptions(ctypes.Structure):
    """fp4attn_forward_options (include/fp4attn.h)."""
    _fields_ = [("struct_size", ctypes.c_uint32), ("affine_a", ctypes.c_float), ("affine_b", ctypes.c_float),
                ("ex2_pairs", ctypes.c_int32), ("guard", ctypes.c_int32), ("guard_margin", ctypes.c_int32),
                ("guard_shift", ctypes.c_int32), ("causal", ctypes.c_int32), ("pv_fp8", ctypes.c_int32),
                ("lse", ctypes.c_void_p)]


# name -> argtypes; entry points not in RESTYPES return a status int
SIGNATURES = {
    "fp4attn_quantize_mxfp4": [_c_p, _int, _i64, _i64, _i64, _int, _c_p, _c_p, _c_p],
    "fp4attn_quantize_mxfp8": [_c_p, _int, _i64, _i64, _i64, _int, _c_p, _c_p, _c_p],
    "fp4attn_quantize_mxfp4_anchored": [_c_p, _int, _i64, _i64, _i64, _int, _i64, _c_p, _c_p, _c_p],
    "fp4attn_forward_mxfp4": [_c_p] * 6 + [_i64] * 4 + [_f32] * 3 + [_c_p, _int, _c_p],
    "fp4attn_forward_bf16": [_c_p] * 3 + [_i64] * 4 + [_f32, _c_p, _int, _c_p],
    "fp4attn_forward_options_init": [ctypes.POINTER(ForwardOptions)],
    "fp4attn_forward_mxfp4_ex": [_c_p] * 6 + [_i64] * 4 + [_f32, ctypes.POINTER(ForwardOptions), _c_p, _int, _c_p],
    "fp4attn_debug_directp_mxfp4": [_c_p] * 6 + [_i64] * 4 + [_f32, ctypes.POINTER(ForwardOptions)]
    + [_c_p, _int, _c_p, _i64] + [_c_p] * 5 + [_c_p],
    "fp4attn_debug_mfma_stream": [_c_p, _c_p, _int, _int, _c_p, _c_p],
    "fp4attn_status_string": [_int],
    "fp4attn_last_error": [],
    "fp4attn_abi_version": [],
}
RESTYPES = {"fp4attn_status_string": ctypes.c_char_p, "fp4attn_last_error": ctypes.c_char_p,
            "fp4attn_abi_version": ctypes.c_int, "fp4attn_forward_options_init": None}


class Fp4AttnError(RuntimeError):
    def __init__(self, status, detail):
        self.status = status
        super().__init__(f"fp4attn status {status}: {detail}")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python paper_2609_04105_amd/build.py` "
            "(or __graft_entry__.build()); there is no fallback path")
    handle = ctypes.CDLL(LIB_PATH)
    for name, args in SIGNATURES.items():
        fn = getattr(handle, name)
        fn.argtypes = args
        fn.restype = RESTYPES.get(name, ctypes.c_int)
    return handle


lib = _load()


def check(status):
    """Raise Fp4AttnError unless ``status`` is FP4ATTN_OK."""
    if status != FP4ATTN_OK:
        detail = lib.fp4attn_last_error().decode() or lib.fp4attn_status_string(status).decode()
        raise Fp4AttnError(status, detail)


def abi_version():
    v = lib.fp4attn_abi_version()
    return v >> 16, v & 0xFFFF
