"""MI355X (gfx950) inference path of the MADDNESS-style approximate matrix
product studied in McCarter & Dronen, "Look-ups are not (yet) all you need for
deep learning inference": tree encoding plus lookup-accumulate over 8-bit
block floating point (or fp32) tables, as hand-written HIP kernels behind the
C ABI of include/maddness.h.

The entry points load lazily, so ``paper_2207_05808_amd.workloads`` (the
seeded input generator) imports without torch or the HIP library.
"""
_BINDING = ("encode", "lut_accumulate", "lut_accumulate_f32", "matmul", "matmul_f32", "matmul_act",
            "matmul_act_f32", "lut_accumulate_avg", "build_lut_shared",
            "build_lut", "build_lut_f32", "quantize_lut", "encoder_gram", "encoder_scatter", "fit_lut_ridge", "fit_lut_gd",
            "fit_lut_workspace_bytes", "fit_lut_gd_workspace_bytes", "matmul_index_bytes", "matmul_noalloc",
            "version", "prepare_matmul", "prepare_matmul_f32", "PreparedCall")

__all__ = list(_BINDING) + ["MaddnessError"]


def __getattr__(name):
    if name in _BINDING:
        from . import binding
        return getattr(binding, name)
    if name == "MaddnessError":
        from ._lib import MaddnessError
        return MaddnessError
    raise AttributeError(name)
