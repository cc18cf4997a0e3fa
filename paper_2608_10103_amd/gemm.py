"""Python binding for libmpgemm.so (the C ABI in include/mpgemm.h).

Argument marshalling only: shape/dtype/device checks, then a ctypes call into
the HIP library, which validates again and enqueues its own kernels on the
given stream. PyTorch supplies device memory and streams; no torch operator
runs on the GPU path. If the library is not built this module raises instead
of computing anything another way.

Scratch memory: the plain entry points use none. Calls that need some (an
explicit split K, the INT4 variants fed by an FP6 pre-pass, zero points) take
a workspace: a zero-filled uint8 CUDA tensor (new_workspace), or
workspace="auto" to have this module allocate one through PyTorch for the
call. The library itself never allocates.

Operand conventions (see include/mpgemm.h):
  A  (M, K)    row-major          float16 / int8, or uint8 (M, K/2) for INT4
  B  (N, K)    = K x N column-major, same dtypes (uint8 (N, K/2) for INT4)
  C  (M, N)    row-major          float32 (FP16 path) or int32
"""
from __future__ import annotations

import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmpgemm.so")
DTYPE_CODE = {"f16": 0, "s8": 1, "s4": 2}
_IN_DTYPE = {"f16": torch.float16, "s8": torch.int8, "s4": torch.uint8}
_OUT_DTYPE = {"f16": torch.float32, "s8": torch.int32, "s4": torch.int32}
_lib = None


class HipError(RuntimeError):
    """A non-zero hipError_t returned by the library."""

    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: hipError_t {code}")
        self.code = code


def lib() -> ctypes.CDLL:
    """The loaded HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() "
                           "or python -m paper_2608_10103_amd.build")
    L = ctypes.CDLL(LIB_PATH)
    I, P = ctypes.c_int, ctypes.c_void_p
    for name in ("gemm_f16_f32", "gemm_s8_s32", "gemm_s4_s32"):
        fn = getattr(L, name)
        fn.argtypes = [I, I, I, P, P, P, P]
        fn.restype = I
    L.mpgemm_num_variants.argtypes = [I]
    L.mpgemm_num_variants.restype = I
    L.mpgemm_variant_name.argtypes = [I, I]
    L.mpgemm_variant_name.restype = ctypes.c_char_p
    L.mpgemm_select_variant.argtypes = [I, I, I, I, P, P, P]
    L.mpgemm_select_variant.restype = I
    L.mpgemm_select_variant_ws.argtypes = [I, I, I, I, P, P, P]
    L.mpgemm_select_variant_ws.restype = I
    L.mpgemm_variant_supports.argtypes = [I, I, I, I, I, P, P, P]
    L.mpgemm_variant_supports.restype = I
    L.mpgemm_run_variant.argtypes = [I, I, I, I, I, P, P, P, P]
    L.mpgemm_run_variant.restype = I
    L.mpgemm_select_splits.argtypes = [I, I, I, I, I]
    L.mpgemm_select_splits.restype = I
    IP = ctypes.POINTER(ctypes.c_int)
    L.mpgemm_sk_schedule.argtypes = [I, I, I, I, I, IP, IP, IP]
    L.mpgemm_sk_schedule.restype = I
    L.gemm_scaled.argtypes = [I, I, I, I, P, P, P, P, P]
    L.gemm_scaled.restype = I
    S = ctypes.c_size_t
    L.mpgemm_gemm_ws.argtypes = [I, I, I, I, P, P, P, P, P, S, P]
    L.mpgemm_gemm_ws.restype = I
    L.mpgemm_gemm_noalloc.argtypes = [I, I, I, I, P, P, P, P, P]
    L.mpgemm_gemm_noalloc.restype = I
    L.mpgemm_run_variant_ws.argtypes = [I, I, I, I, I, I, P, P, P, P, P, S, P]
    L.mpgemm_run_variant_ws.restype = I
    L.mpgemm_workspace_size.argtypes = [I, I, I, I, I, I, P, ctypes.POINTER(S)]
    L.mpgemm_workspace_size.restype = I
    L.mpgemm_s4_run_to_fp6.argtypes = [P, P]
    L.mpgemm_s4_run_to_fp6.restype = None
    L.mpgemm_s4_run_to_e2m3.argtypes = [P, P]
    L.mpgemm_s4_run_to_e2m3.restype = None
    L.mpgemm_gemm_bt.argtypes = [I, I, I, I, P, P, P, P]
    L.mpgemm_gemm_bt.restype = I
    _lib = L
    return L


EXPORTED_SYMBOLS = ("gemm_f16_f32", "gemm_s8_s32", "gemm_s4_s32", "gemm_scaled", "mpgemm_gemm_ws",
                    "mpgemm_gemm_noalloc",
                    "mpgemm_workspace_size", "mpgemm_num_variants", "mpgemm_variant_name",
                    "mpgemm_select_variant", "mpgemm_select_variant_ws", "mpgemm_variant_supports",
                    "mpgemm_run_variant",
                    "mpgemm_select_splits", "mpgemm_run_variant_ws", "mpgemm_s4_run_to_fp6",
                    "mpgemm_s4_run_to_e2m3", "mpgemm_gemm_bt", "mpgemm_sk_schedule")


def _stream_ptr(stream, device) -> int:
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return int(stream.cuda_stream)


def _shapes(dtype: str, A: torch.Tensor, B: torch.Tensor):
    want = _IN_DTYPE[dtype]
    for name, t in (("A", A), ("B", B)):
        if not isinstance(t, torch.Tensor) or t.dtype != want or t.dim() != 2:
            raise TypeError(f"{name} must be a 2-D {want} tensor")
        if not t.is_cuda:
            raise ValueError(f"{name} must be on a GPU")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if A.device != B.device:
        raise ValueError("A and B must be on the same device")
    M, KA = A.shape
    N, KB = B.shape
    if KA != KB:
        raise ValueError(f"K mismatch: A has {KA}, B has {KB} per row")
    K = 2 * KA if dtype == "s4" else KA
    return M, N, K


def _out(dtype, M, N, A, C):
    if C is None:
        return torch.empty((M, N), dtype=_OUT_DTYPE[dtype], device=A.device)
    if C.dtype != _OUT_DTYPE[dtype] or tuple(C.shape) != (M, N) or not C.is_contiguous():
        raise ValueError(f"C must be a contiguous ({M}, {N}) {_OUT_DTYPE[dtype]} tensor")
    if C.device != A.device:
        raise ValueError("C must be on the operands' device")
    return C


def workspace_size(dtype: str, M: int, N: int, K: int, variant=None, splits=None, epi=None) -> int:
    """Bytes of workspace a call would use (mpgemm_workspace_size): the
    automatic choice (variant None, splits None) or an explicit one; epi an
    Epilogue or None. Raises HipError for arguments the call would refuse."""
    out = ctypes.c_size_t(0)
    code = lib().mpgemm_workspace_size(DTYPE_CODE[dtype], -1 if variant is None else variant, splits or 0,
                                       M, N, K, None if epi is None else ctypes.addressof(epi),
                                       ctypes.byref(out))
    if code != 0:
        raise HipError(code, f"workspace size of {dtype} {M}x{N}x{K}")
    return int(out.value)


def new_workspace(nbytes: int, device) -> torch.Tensor:
    """A zero-filled workspace (uint8 CUDA tensor) of at least nbytes; PyTorch's
    allocations are 256-byte aligned, as the library requires."""
    return torch.zeros(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def _workspace(workspace, dtype, M, N, K, variant, splits, epi, device, stream):
    """(pointer, bytes, tensor) of a workspace argument: None, "auto" (allocated
    here through PyTorch, zero-filled, its memory kept from reuse until the
    call's stream has done with it) or a uint8 CUDA tensor."""
    if workspace is None:
        return None, 0, None
    if isinstance(workspace, str):
        if workspace != "auto":
            raise ValueError('workspace must be None, "auto" or a uint8 CUDA tensor')
        n = workspace_size(dtype, M, N, K, variant, splits, epi)
        if n == 0:
            return None, 0, None
        workspace = new_workspace(n, device)
        if stream is not None:
            workspace.record_stream(stream)
    if (not isinstance(workspace, torch.Tensor) or workspace.dtype != torch.uint8 or not workspace.is_cuda
            or not workspace.is_contiguous() or workspace.device != device):
        raise ValueError(f"workspace must be a contiguous uint8 tensor on {device}")
    return workspace.data_ptr(), workspace.numel(), workspace


def _call(dtype: str, A, B, C, stream, variant, splits=None, workspace=None):
    M, N, K = _shapes(dtype, A, B)
    C = _out(dtype, M, N, A, C)
    s = _stream_ptr(stream, A.device)
    if splits is not None and variant is None:
        raise ValueError("splits needs an explicit variant")
    wp, wn, _keep = _workspace(workspace, dtype, M, N, K, variant, splits, None, A.device, stream)
    with torch.cuda.device(A.device):
        if wn == 0 and splits is None:
            if variant is None:
                fn = getattr(lib(), {"f16": "gemm_f16_f32", "s8": "gemm_s8_s32",
                                     "s4": "gemm_s4_s32"}[dtype])
                code = fn(M, N, K, A.data_ptr(), B.data_ptr(), C.data_ptr(), s)
            else:
                code = lib().mpgemm_run_variant(DTYPE_CODE[dtype], variant, M, N, K, A.data_ptr(),
                                                B.data_ptr(), C.data_ptr(), s)
        elif variant is None:
            code = lib().mpgemm_gemm_ws(DTYPE_CODE[dtype], M, N, K, A.data_ptr(), B.data_ptr(), C.data_ptr(),
                                        None, wp, wn, s)
        else:
            code = lib().mpgemm_run_variant_ws(DTYPE_CODE[dtype], variant, splits or 0, M, N, K, A.data_ptr(),
                                               B.data_ptr(), C.data_ptr(), None, wp, wn, s)
    if code != 0:
        raise HipError(code, f"{dtype} GEMM {M}x{N}x{K}")
    return C


def gemm_f16_f32(A, B, C=None, stream=None, variant=None, splits=None, workspace=None):
    """C = A @ B with FP16 A (M, K), FP16 B (N, K) = K x N column-major; FP32 C."""
    return _call("f16", A, B, C, stream, variant, splits, workspace)


def gemm_s8_s32(A, B, C=None, stream=None, variant=None, splits=None, workspace=None):
    """C = A @ B with INT8 A (M, K), INT8 B (N, K); INT32 C."""
    return _call("s8", A, B, C, stream, variant, splits, workspace)


def gemm_s4_s32(A, B, C=None, stream=None, variant=None, splits=None, workspace=None):
    """C = A @ B with packed INT4 A (M, K/2) and B (N, K/2) uint8 (low nibble =
    even k); INT32 C."""
    return _call("s4", A, B, C, stream, variant, splits, workspace)


GEMM = {"f16": gemm_f16_f32, "s8": gemm_s8_s32, "s4": gemm_s4_s32}


def gemm_bt(dtype: str, A, B_kn, C=None, stream=None):
    """C = A * B with B given K x N row-major (N-contiguous) (mpgemm_gemm_bt):
    FP16 or INT8 A (M, K) and B_kn (K, N) of the dtype's input type, or INT4 A
    (M, K/2) packed along K and B_kn (K, N/2) packed along N (uint8, low
    nibble = even column)."""
    if dtype not in ("f16", "s8", "s4"):
        raise ValueError("transposed B: f16, s8 or s4")
    want = _IN_DTYPE[dtype]
    for name, t in (("A", A), ("B", B_kn)):
        if not isinstance(t, torch.Tensor) or t.dtype != want or t.dim() != 2:
            raise TypeError(f"{name} must be a 2-D {want} tensor")
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous GPU tensor")
    if A.device != B_kn.device:
        raise ValueError("A and B must be on the same device")
    M, K = A.shape
    KB, N = B_kn.shape
    if dtype == "s4":
        K, N = 2 * K, 2 * N
    if K != KB:
        raise ValueError(f"K mismatch: A has {K}, B has {KB} rows")
    C = _out(dtype, M, N, A, C)
    s = _stream_ptr(stream, A.device)
    with torch.cuda.device(A.device):
        code = lib().mpgemm_gemm_bt(DTYPE_CODE[dtype], M, N, K, A.data_ptr(), B_kn.data_ptr(),
                                    C.data_ptr(), s)
    if code != 0:
        raise HipError(code, f"transposed-B {dtype} GEMM {M}x{N}x{K}")
    return C


class Epilogue(ctypes.Structure):
    """mpgemm_epilogue of include/mpgemm.h (device pointers, output type)."""
    _fields_ = [("scale_a", ctypes.c_void_p), ("scale_b", ctypes.c_void_p),
                ("zero_a", ctypes.c_void_p), ("zero_b", ctypes.c_void_p), ("out_type", ctypes.c_int)]


OUT_TYPE = {torch.float32: 1, torch.float16: 2, torch.bfloat16: 3}


def _vec(x, n, dtype, name, device):
    if x is None:
        return None
    if x.dtype != dtype or x.dim() != 1 or x.numel() != n or not x.is_contiguous() or x.device != device:
        raise ValueError(f"{name} must be a contiguous ({n},) {dtype} tensor on {device}")
    return x.data_ptr()


def gemm_scaled(dtype: str, A, B, scale_a=None, scale_b=None, zero_a=None, zero_b=None,
                out_dtype=torch.float16, C=None, stream=None, variant=None, splits=None, workspace=None):
    """C = round(scale_a[i] * scale_b[j] * sum_k (A(i,k) - zero_a[i]) (B(k,j) - zero_b[j]))
    in out_dtype (float32, float16 or bfloat16); operands as for GEMM[dtype];
    scales float32 (M,) / (N,), zero points int32 (M,) / (N,) (integer inputs
    only; they need a workspace), any of them None. Runs in the GEMM kernels'
    epilogue."""
    M, N, K = _shapes(dtype, A, B)
    if out_dtype not in OUT_TYPE:
        raise ValueError("out_dtype must be float32, float16 or bfloat16")
    dev = A.device
    epi = Epilogue(_vec(scale_a, M, torch.float32, "scale_a", dev), _vec(scale_b, N, torch.float32, "scale_b", dev),
                   _vec(zero_a, M, torch.int32, "zero_a", dev), _vec(zero_b, N, torch.int32, "zero_b", dev),
                   OUT_TYPE[out_dtype])
    if C is None:
        C = torch.empty((M, N), dtype=out_dtype, device=dev)
    elif C.dtype != out_dtype or tuple(C.shape) != (M, N) or not C.is_contiguous() or C.device != dev:
        raise ValueError(f"C must be a contiguous ({M}, {N}) {out_dtype} tensor on {dev}")
    if splits is not None and variant is None:
        raise ValueError("splits needs an explicit variant")
    wp, wn, _keep = _workspace(workspace, dtype, M, N, K, variant, splits, epi, dev, stream)
    s = _stream_ptr(stream, dev)
    with torch.cuda.device(dev):
        if variant is None and wn == 0:
            code = lib().gemm_scaled(DTYPE_CODE[dtype], M, N, K, A.data_ptr(), B.data_ptr(), C.data_ptr(),
                                     ctypes.addressof(epi), s)
        elif variant is None:
            code = lib().mpgemm_gemm_ws(DTYPE_CODE[dtype], M, N, K, A.data_ptr(), B.data_ptr(), C.data_ptr(),
                                        ctypes.addressof(epi), wp, wn, s)
        else:
            code = lib().mpgemm_run_variant_ws(DTYPE_CODE[dtype], variant, splits or 0, M, N, K,
                                               A.data_ptr(), B.data_ptr(), C.data_ptr(),
                                               ctypes.addressof(epi), wp, wn, s)
    if code != 0:
        raise HipError(code, f"scaled {dtype} GEMM {M}x{N}x{K}")
    return C


def raw_call(dtype: str, M: int, N: int, K: int, a_ptr: int, b_ptr: int, c_ptr: int,
             stream_ptr: int = 0, variant: int | None = None) -> int:
    """Call an entry point with raw integers/pointers; returns the hipError_t."""
    L = lib()
    if variant is None:
        fn = getattr(L, {"f16": "gemm_f16_f32", "s8": "gemm_s8_s32", "s4": "gemm_s4_s32"}[dtype])
        return fn(M, N, K, a_ptr, b_ptr, c_ptr, stream_ptr)
    return L.mpgemm_run_variant(DTYPE_CODE[dtype], variant, M, N, K, a_ptr, b_ptr, c_ptr,
                                stream_ptr)


def select_splits(dtype: str, variant: int, M: int, N: int, K: int) -> int:
    """Split-K count the entry points use for this variant (1 = none)."""
    return lib().mpgemm_select_splits(DTYPE_CODE[dtype], variant, M, N, K)


def sk_schedule(dtype: str, variant: int, M: int, N: int, K: int) -> tuple[int, int, int]:
    """Stream-K schedule of a variant for this problem on the current device:
    (whole tiles first, K-parts of each remaining tile (1: off), grid)."""
    dp, parts, grid = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    code = lib().mpgemm_sk_schedule(DTYPE_CODE[dtype], variant, M, N, K, ctypes.byref(dp),
                                    ctypes.byref(parts), ctypes.byref(grid))
    if code != 0:
        raise HipError(code, f"stream-K schedule of {dtype} variant {variant} for {M}x{N}x{K}")
    return dp.value, parts.value, grid.value


def num_variants(dtype: str) -> int:
    return lib().mpgemm_num_variants(DTYPE_CODE[dtype])


def variant_name(dtype: str, variant: int) -> str:
    return lib().mpgemm_variant_name(DTYPE_CODE[dtype], variant).decode()


def select_variant(dtype: str, M: int, N: int, K: int, a_ptr: int = 0, b_ptr: int = 0,
                   c_ptr: int = 16, with_ws: bool = False) -> int:
    """Variant the entry point would run (with_ws: mpgemm_gemm_ws with a large
    enough workspace); pointers only matter for alignment, the defaults are
    16-byte aligned stand-ins, never dereferenced."""
    if a_ptr == 0:
        a_ptr = 1 << 20
    if b_ptr == 0:
        b_ptr = 1 << 40
    if c_ptr == 16:
        c_ptr = 1 << 44
    fn = lib().mpgemm_select_variant_ws if with_ws else lib().mpgemm_select_variant
    return fn(DTYPE_CODE[dtype], M, N, K, a_ptr, b_ptr, c_ptr)


def variant_supports(dtype: str, variant: int, M: int, N: int, K: int, a_ptr: int = 1 << 20,
                     b_ptr: int = 1 << 40, c_ptr: int = 1 << 44) -> bool:
    return lib().mpgemm_variant_supports(DTYPE_CODE[dtype], variant, M, N, K, a_ptr, b_ptr,
                                         c_ptr) == 1


def s4_run_to_e2m3(run: bytes) -> list:
    """Host-side INT4 -> biased FP6 E2M3 conversion of one 16-byte run (the
    conversion the INT4 kernel applies inside the GEMM): the six 32-bit words
    of the 192-bit string of 32 six-bit codes (code = nibble ^ 8)."""
    if len(run) != 16:
        raise ValueError("a run is 16 bytes")
    src = (ctypes.c_uint8 * 16)(*run)
    out = (ctypes.c_uint32 * 6)()
    lib().mpgemm_s4_run_to_e2m3(ctypes.addressof(src), ctypes.addressof(out))
    return list(out)


def s4_run_to_fp6(run: bytes) -> list:
    """Host-side INT4 -> FP6 E3M2 conversion of one 16-byte run (32 nibbles):
    the six 32-bit words of the 192-bit code string; field f = 8d + 4h + i
    (bits [6f, 6f + 6)) holds the code of nibble h (0 low, 1 high) of byte i
    of 4-byte word d. The same function the FP6 kernels apply on the device."""
    if len(run) != 16:
        raise ValueError("a run is 16 bytes")
    src = (ctypes.c_uint8 * 16)(*run)
    out = (ctypes.c_uint32 * 6)()
    lib().mpgemm_s4_run_to_fp6(ctypes.addressof(src), ctypes.addressof(out))
    return list(out)
