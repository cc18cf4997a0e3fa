"""Helpers for the GPU tests: move seeded numpy operands to the GPU, run one
entry point through the C ABI, and compare with the oracle."""
import numpy as np
import torch

import oracle
import paper_2608_10103_amd as mp

TORCH_IN = {"f16": torch.float16, "s8": torch.int8, "s4": torch.uint8}
F16_TOL = 1e-3  # max |C_gpu - C_exact| / sum_k |a||b|


def dev(x: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda")


def gpu_gemm(dtype, A, B, variant=None, stream=None, splits=None, workspace=None):
    """Run the dtype's entry point (or a given variant, optionally with an
    explicit split-K count) on numpy operands; returns C as numpy (float32 or
    int32). An explicit variant or split gets the workspace it needs
    (allocated through PyTorch) unless one is given."""
    Ad, Bd = dev(A), dev(B)
    if workspace is None and (variant is not None or splits is not None):
        workspace = "auto"
    C = mp.GEMM[dtype](Ad, Bd, variant=variant, stream=stream, splits=splits, workspace=workspace)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def oracle_gemm(dtype, A, B, rows=None):
    """(C_ref, D) where D is the FP16 error scale (None for integers)."""
    if dtype == "f16":
        return oracle.gemm_f16(A, B, rows=rows)
    if dtype == "s8":
        return oracle.gemm_s8(A, B, rows=rows), None
    return oracle.gemm_s4(A, B, rows=rows), None


def assert_parity(dtype, C_gpu, C_ref, D, what=""):
    """Bit-exact for the integer paths, normalised error <= 1e-3 for FP16."""
    if dtype == "f16":
        assert C_gpu.dtype == np.float32
        err = oracle.normalized_error(C_gpu, C_ref, D)
        assert err <= F16_TOL, f"{what}: normalised error {err:.3e} > {F16_TOL}"
        return err
    assert C_gpu.dtype == np.int32
    assert np.all(np.abs(C_ref) < 2**31), f"{what}: oracle result leaves int32"
    bad = np.argwhere(C_gpu.astype(np.int64) != C_ref)
    assert bad.size == 0, (f"{what}: {len(bad)} mismatches, first at {tuple(bad[0])}: "
                           f"gpu {C_gpu[tuple(bad[0])]} oracle {C_ref[tuple(bad[0])]}")
    return 0.0


# Output formats of the scaled entry point: (stored fraction bits, minimum
# normal exponent).
_FORMATS = {"f32": (23, -126), "f16": (10, -14), "bf16": (7, -126)}
TORCH_OUT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def ulp_of(x, out):
    """Spacing of the output format at |x|: 2^(e - fraction bits) for |x| in
    [2^e, 2^(e+1)), the subnormal spacing below the smallest normal. The
    binade comes from frexp (exact), not from a rounded log2."""
    frac, emin = _FORMATS[out]
    ax = np.maximum(np.abs(np.asarray(x, dtype=np.float64)), 2.0 ** emin)
    _, e = np.frexp(ax)  # ax = m 2^e, 0.5 <= m < 1: the binade starts at 2^(e - 1)
    return np.ldexp(1.0, e.astype(np.int64) - 1 - frac)


def assert_scaled(got, exact, D, out, what=""):
    """Scaled outputs. Integer inputs: the exact sum is rounded to binary32,
    multiplied by sa then sb in binary32 (three roundings, relative error
    below 3 * 2^-24, i.e. under 3 binary32 ulp of the exact value), then
    rounded to the output type: |got - exact| <= 3 ulp for binary32 output,
    <= 1 ulp for binary16 / bfloat16 (half an ulp from the last rounding plus
    the binary32 error, far below the other half). FP16 inputs add the sum's
    bound 1e-3 * D (D already scaled) and 2^-21 |exact| for the binary32
    scaling."""
    g = got.float().cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    tol = ulp_of(exact, out) * (3.0 if out == "f32" else 1.0)
    if D is not None:
        tol = tol + F16_TOL * D + 2.0 ** -21 * np.abs(exact)
    err = np.abs(g - exact)
    bad = err > tol
    assert not np.any(bad), (f"{what}: {int(bad.sum())} elements off, worst at "
                             f"{np.unravel_index(np.argmax(err - tol), err.shape)}")
