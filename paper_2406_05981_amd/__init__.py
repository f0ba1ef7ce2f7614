"""MI355X (gfx950) shift-add linear layer of ShiftAddLLM (Sec. 4.1).

The computation lives in ``libshiftadd.so`` (HIP kernels behind the C ABI of
``include/shiftadd.h``); :mod:`paper_2406_05981_amd.shiftadd` is its binding.
Attribute access on this package loads the binding, which raises if the
library has not been built (``python -m paper_2406_05981_amd.build``).
"""
__all__ = [
    "sa_packed_bytes", "sa_packed_offset", "sa_pack_weights", "sa_unpack_weights",
    "sa_build_lut", "sa_shiftadd_gemm", "sa_plan_gemm", "sa_shiftadd_gemm_colwise",
    "sa_plan_gemm_colwise", "sa_quantize_bcq", "sa_read_probe", "sa_status_string",
    "sa_version", "quantize_bcq", "shiftadd_gemm_colwise", "sa_shiftadd_gemm_blockwise",
    "sa_plan_gemm_blockwise", "shiftadd_gemm_blockwise", "sa_shiftadd_gemm_terms",
    "sa_quantize_bcq_terms", "quantize_bcq_terms", "sa_gram_f16", "sa_inverse_cholesky_diag",
    "sa_importance_criterion", "sa_fit_per_bit", "sa_allocate_bits", "bit_criterion",
    "pack_weights", "shiftadd_gemm", "SaError", "sa_shiftadd_gemm_kslice",
    "sa_kslice_workspace_bytes", "sa_shiftadd_gemm_f16",
]


def __getattr__(name):
    if name in __all__:
        from . import shiftadd
        return getattr(shiftadd, name)
    raise AttributeError(name)
