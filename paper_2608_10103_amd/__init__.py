"""Dense C = A * B on one AMD Instinct MI355X (gfx950): FP16->FP32, INT8->INT32
and signed INT4->INT32, on hand-written MFMA kernels behind a C ABI
(include/mpgemm.h, libmpgemm.so). This package is the Python binding."""
from .gemm import (GEMM, EXPORTED_SYMBOLS, LIB_PATH, HipError, gemm_bt, gemm_f16_f32, gemm_s4_s32, gemm_scaled,
                   gemm_s8_s32, lib, new_workspace, num_variants, raw_call, s4_run_to_e2m3, s4_run_to_fp6,
                   select_splits, select_variant, sk_schedule, variant_name, variant_supports,
                   workspace_size)

__all__ = ["GEMM", "EXPORTED_SYMBOLS", "LIB_PATH", "HipError", "gemm_bt", "gemm_f16_f32", "gemm_s8_s32", "gemm_scaled",
           "gemm_s4_s32", "lib", "new_workspace", "num_variants", "raw_call", "s4_run_to_e2m3", "s4_run_to_fp6",
           "select_splits", "select_variant", "sk_schedule", "variant_name", "variant_supports", "workspace_size"]
