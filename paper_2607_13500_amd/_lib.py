"""ctypes handle on libaltr.so (the gfx950 HIP library) with argument types.

torch is imported first on purpose: the library's HIP runtime dependency
(libamdhip64.so.7) then resolves to the runtime torch already loaded, so device
pointers and streams from torch are valid in the library.
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (must precede loading the library, see above)

from . import build as _build

LIB_PATH = _build.LIB


class Params(ctypes.Structure):
    """Mirror of tr_params in include/tr.h."""
    _fields_ = [
        ("D", ctypes.c_int32),
        ("Dc", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("max_images", ctypes.c_int32),
        ("max_tokens", ctypes.c_int64),
        ("max_N", ctypes.c_int32),
        ("flags", ctypes.c_int32),
        ("lam", ctypes.c_double),
        ("keep_ratio", ctypes.c_double),
    ]


TR_OK, TR_EINVAL, TR_ENOMEM, TR_EUNSUPPORTED, TR_EDEVICE = range(5)
TR_FP32, TR_BF16 = 0, 1
TR_FLAG_STRIDE_REAL = 1
TR_FLAG_SHANNON = 2
TR_FLAG_CHECK_FINITE = 4
TR_NOALLOC_MAX_TOKENS = 524288
TR_NOALLOC_MAX_IMAGES = 256

_lib = None


def load(build_if_missing: bool = True) -> ctypes.CDLL:
    """Load libaltr.so; build it with hipcc first only when no built copy exists."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        if not build_if_missing:
            raise RuntimeError("libaltr.so is not built (run paper_2607_13500_amd/build.py)")
        _build.build()
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    P = ctypes.POINTER
    lib.tr_create.argtypes = [P(Params), P(vp)]
    lib.tr_create.restype = i32
    lib.tr_reduce.argtypes = [vp, vp, vp, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.tr_reduce.restype = i32
    lib.tr_score.argtypes = [vp, vp, vp, vp, i64, vp, vp, vp, vp]
    lib.tr_score.restype = i32
    lib.tr_nonfinite_rows.argtypes = [vp, vp, i32, vp]
    lib.tr_nonfinite_rows.restype = i32
    lib.tr_select.argtypes = [vp, vp, vp, i32, vp, vp, vp, vp, vp]
    lib.tr_select.restype = i32
    lib.tr_gemm_bf16.argtypes = [vp, vp, i64, vp, i64, vp, i64, vp, i64, i32, i32, i32, vp]
    lib.tr_gemm_bf16.restype = i32
    lib.tr_mlp_out_cos.argtypes = [vp, vp, i64, vp, i64, vp, vp, i32, i32, vp, vp]
    lib.tr_mlp_out_cos.restype = i32
    lib.tr_reduce_given_s.argtypes = [vp, vp, vp, i32, vp, vp, vp, vp, vp, vp, vp]
    lib.tr_reduce_given_s.restype = i32
    lib.tr_reduce_project.argtypes = [vp, vp, vp, vp, i32, vp, vp, vp, i64, i32, vp, vp, vp, vp]
    lib.tr_reduce_project.restype = i32
    lib.tr_read_bandwidth.argtypes = [vp, vp, i32, vp, i32, vp]
    lib.tr_read_bandwidth.restype = i32
    lib.tr_reduce_noalloc.argtypes = [P(Params), vp, vp, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.tr_reduce_noalloc.restype = i32
    lib.tr_check_reduce.argtypes = [P(Params), vp, vp, vp, i32, vp, vp, vp, vp, vp, vp, vp]
    lib.tr_check_reduce.restype = i32
    lib.tr_plan.argtypes = [P(Params), i32, vp, vp, vp, vp, vp, vp]
    lib.tr_plan.restype = i32
    lib.tr_capacity_N.argtypes = []
    lib.tr_capacity_N.restype = i32
    lib.tr_timing_enable.argtypes = [vp, i32]
    lib.tr_timing_enable.restype = i32
    lib.tr_timing_read.argtypes = [vp, P(ctypes.c_double), P(i64)]
    lib.tr_timing_read.restype = i32
    lib.tr_destroy.argtypes = [vp]
    lib.tr_destroy.restype = None
    lib.tr_strerror.argtypes = [i32]
    lib.tr_strerror.restype = ctypes.c_char_p
    lib.tr_last_error.argtypes = []
    lib.tr_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib
