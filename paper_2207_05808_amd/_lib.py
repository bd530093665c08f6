"""ctypes binding of libmaddness.so (the C ABI declared in include/maddness.h).

Argument marshalling only: every step of the path runs in the HIP kernels of
the library.  torch supplies device memory and the current stream.  There is
no fallback of any kind; if the library is missing or fails to load, every
call raises.

torch is imported before the library is loaded so that the process holds a
single HIP runtime (torch's), which the library then binds to by soname.
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (must precede loading libmaddness.so, see module doc)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmaddness.so")

OK, EINVAL, EHIP, EUNSUPPORTED, ENOMEM = 0, 1, 2, 3, 4

_lib = None


class MaddnessError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn}: status {status} ({msg})")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with paper_2207_05808_amd.build.build() "
                "(or __graft_entry__.build()); there is no fallback path")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        L.maddness_version.argtypes = []
        L.maddness_status_string.argtypes = [ctypes.c_int]
        L.maddness_status_string.restype = ctypes.c_char_p
        L.maddness_encode.argtypes = [vp, i64, i32, i64, vp, vp, i32, vp, vp]
        L.maddness_lut_accumulate.argtypes = [vp, i64, i32, vp, vp, vp, i32, vp, vp, vp]
        L.maddness_lut_accumulate_f32.argtypes = [vp, i64, i32, vp, i32, vp, vp]
        L.maddness_matmul.argtypes = [vp, i64, i32, i64, vp, vp, i32, vp, vp, vp, i32, vp, vp, vp, vp]
        L.maddness_matmul_f32.argtypes = [vp, i64, i32, i64, vp, vp, i32, vp, i32, vp, vp, vp]
        L.maddness_matmul_act.argtypes = [vp, i64, i32, i64, vp, vp, i32, vp, vp, vp, i32, vp, i32, vp, vp, vp]
        L.maddness_matmul_act_f32.argtypes = [vp, i64, i32, i64, vp, vp, i32, vp, i32, vp, i32, vp, vp, vp]
        L.maddness_lut_accumulate_avg.argtypes = [vp, i64, i32, vp, vp, vp, i32, vp, vp, vp]
        L.maddness_build_lut_shared.argtypes = [vp, vp, i32, i32, i32, vp, vp, vp, vp]
        L.maddness_build_lut.argtypes = [vp, vp, i32, i32, i32, vp, vp, vp, vp]
        L.maddness_build_lut_f32.argtypes = [vp, vp, i32, i32, i32, vp, vp]
        L.maddness_quantize_lut.argtypes = [vp, i32, i32, i32, vp, vp, vp, vp]
        L.maddness_encoder_gram.argtypes = [vp, i64, i32, vp, vp]
        L.maddness_encoder_scatter.argtypes = [vp, i64, i32, vp, i32, vp, vp, i64, vp]
        L.maddness_encoder_scatter_workspace_bytes.argtypes = [i64, i32]
        L.maddness_encoder_scatter_workspace_bytes.restype = i64
        L.maddness_fit_lut_workspace_bytes.argtypes = [i64, i32]
        L.maddness_fit_lut_workspace_bytes.restype = i64
        L.maddness_fit_lut_ridge.argtypes = [vp, i64, i32, vp, i32, vp, ctypes.c_double, vp, vp, i64, vp]
        L.maddness_matmul_noalloc.argtypes = [vp, i64, i32, i64, vp, vp, i32, vp, vp, vp, i32, vp, vp, vp, vp]
        L.maddness_matmul_noalloc.restype = ctypes.c_int
        L.maddness_matmul_index_bytes.argtypes = [vp, i64, i32, i64, i32, i32, i32, i32]
        L.maddness_matmul_index_bytes.restype = i64
        L.maddness_fit_lut_gd_workspace_bytes.argtypes = [i64, i32, i32]
        L.maddness_fit_lut_gd_workspace_bytes.restype = i64
        L.maddness_fit_lut_gd.argtypes = [vp, i64, i32, vp, i32, vp, i32, vp, ctypes.c_double, ctypes.c_double, i32,
                                          vp, vp, i64, vp]
        for f in ("maddness_version", "maddness_encode", "maddness_lut_accumulate",
                  "maddness_lut_accumulate_f32", "maddness_matmul", "maddness_matmul_f32",
                  "maddness_matmul_act", "maddness_matmul_act_f32", "maddness_build_lut",
                  "maddness_build_lut_f32", "maddness_lut_accumulate_avg", "maddness_build_lut_shared",
                  "maddness_quantize_lut", "maddness_encoder_gram", "maddness_encoder_scatter",
                  "maddness_fit_lut_ridge", "maddness_fit_lut_gd"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def check(fn: str, status: int) -> None:
    if status != OK:
        raise MaddnessError(fn, status, lib().maddness_status_string(status).decode())
