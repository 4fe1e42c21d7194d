"""IsoQuant stage-1 quantize/dequantize for AMD Instinct MI355X (gfx950).

The computation runs in libisoquant.so (HIP kernels behind a C ABI, see
include/isoquant.h); this package is its Python binding.
"""
from .isoquant import (ISOQ_BLOCK8, ISOQ_F16, ISOQ_F32, ISOQ_FAST, ISOQ_FULL, ISOQ_PLANAR2D, IsoqError,
                       LIB_PATH, Params, isoq_codebook_lloyd, isoq_dequantize,
                       isoq_export_params_per_set, isoq_kv_append, isoq_kv_scores,
                       isoq_packed_bytes, isoq_record_bytes, Sketch, isoq_sketch_init, isoq_sketch_destroy,
                       isoq_sketch_export, isoq_quantize_qjl, isoq_kv_scores_qjl, isoq_kv_append_qjl,
                       isoq_params_destroy,
                       isoq_params_export, isoq_params_info, isoq_params_init, isoq_quantize,
                       isoq_raw_params_per_set, isoq_rotation_draws, isoq_roundtrip,
                       isoq_status_string)

__all__ = [
    "ISOQ_BLOCK8", "ISOQ_F16", "ISOQ_F32", "ISOQ_FAST", "ISOQ_FULL", "ISOQ_PLANAR2D", "IsoqError", "LIB_PATH",
    "Params", "isoq_codebook_lloyd", "isoq_dequantize", "isoq_export_params_per_set", "isoq_kv_append",
    "isoq_kv_scores", "Sketch", "isoq_sketch_init", "isoq_sketch_destroy", "isoq_sketch_export",
    "isoq_quantize_qjl", "isoq_kv_scores_qjl", "isoq_kv_append_qjl",
    "isoq_packed_bytes", "isoq_record_bytes", "isoq_params_destroy", "isoq_params_export", "isoq_params_info",
    "isoq_params_init", "isoq_quantize", "isoq_raw_params_per_set", "isoq_rotation_draws",
    "isoq_roundtrip", "isoq_status_string",
]
