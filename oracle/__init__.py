"""CPU oracle for C = A * B (FP16->FP32, INT8->INT32, INT4->INT32).

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package. It never imports the
GPU library, and the GPU library never imports it: the two share no code.

The arithmetic lives in ``oracle.c`` (plain C, POSIX threads), which writes out
the definition C[i][j] = sum_k A(i,k) B(k,j) with A row-major and B
column-major (the paper's ".row.col" MMA operand order, Listing
"lst:int4-primitives"), in binary64 for FP16 inputs and in exact int64 for the
integer paths. This module only loads that library and marshals numpy arrays.

The functions here pin nothing by themselves; ``tests/test_oracle.py`` pins them
against closed forms, brute force on tiny shapes and numpy's matmul.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

_ERRORS = {1: "invalid argument", 2: "non-finite input", 3: "out of memory",
           4: "thread creation failed"}


def default_threads() -> int:
    """Threads the oracle uses by default: the CPUs this process may run on,
    capped at 16 (the CPU share of a one-GPU machine)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _rows_arg(rows, M):
    if rows is None:
        return None, M
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int32))
    return r, int(r.size)


def _check(code):
    if code != 0:
        raise ValueError(f"oracle: {_ERRORS.get(code, code)}")


class Oracle:
    """One loaded copy of the oracle library (the built liboracle.so by
    default; the tests also load deliberately broken builds of oracle.c to
    show the pins catch such mistakes)."""

    def __init__(self, path: str = _LIB_PATH):
        lib = ctypes.CDLL(path)
        L, P, I = ctypes.c_long, ctypes.c_void_p, ctypes.c_int
        lib.oracle_gemm_f16.argtypes = [L, L, L, P, P, P, P, P, L, I]
        lib.oracle_gemm_s8.argtypes = [L, L, L, P, P, P, P, L, I]
        lib.oracle_gemm_s4.argtypes = [L, L, L, P, P, P, P, L, I]
        for fn in (lib.oracle_gemm_f16, lib.oracle_gemm_s8, lib.oracle_gemm_s4):
            fn.restype = I
        lib.oracle_half_to_double.argtypes = [ctypes.c_uint16]
        lib.oracle_half_to_double.restype = ctypes.c_double
        lib.oracle_s4_value.argtypes = [P, L]
        lib.oracle_s4_value.restype = I
        self.lib = lib
        self.path = path

    def gemm_f16(self, A: np.ndarray, B: np.ndarray, rows=None, threads: int | None = None):
        """FP16 oracle. A: (M, K) float16; B: (N, K) float16 (K x N column-major).

        Returns (C, D), both float64 of shape (R, N): C the binary64 sum of exact
        products in k order, D = sum_k |A(i,k)| |B(k,j)|. R = len(rows) if given.
        """
        A = np.ascontiguousarray(A, dtype=np.float16)
        B = np.ascontiguousarray(B, dtype=np.float16)
        M, K = A.shape
        N, Kb = B.shape
        if Kb != K:
            raise ValueError("K mismatch")
        r, R = _rows_arg(rows, M)
        C = np.empty((R, N), dtype=np.float64)
        D = np.empty((R, N), dtype=np.float64)
        _check(self.lib.oracle_gemm_f16(M, N, K, _ptr(A.view(np.uint16)), _ptr(B.view(np.uint16)),
                                        _ptr(C), _ptr(D), None if r is None else _ptr(r), R,
                                        threads or default_threads()))
        return C, D

    def gemm_s8(self, A: np.ndarray, B: np.ndarray, rows=None, threads: int | None = None):
        """INT8 oracle. A: (M, K) int8; B: (N, K) int8. Returns int64 (R, N)."""
        A = np.ascontiguousarray(A, dtype=np.int8)
        B = np.ascontiguousarray(B, dtype=np.int8)
        M, K = A.shape
        N, Kb = B.shape
        if Kb != K:
            raise ValueError("K mismatch")
        r, R = _rows_arg(rows, M)
        C = np.empty((R, N), dtype=np.int64)
        _check(self.lib.oracle_gemm_s8(M, N, K, _ptr(A), _ptr(B), _ptr(C),
                                       None if r is None else _ptr(r), R,
                                       threads or default_threads()))
        return C

    def gemm_s4(self, A: np.ndarray, B: np.ndarray, K: int | None = None, rows=None,
                threads: int | None = None):
        """INT4 oracle. A: (M, K/2) packed uint8; B: (N, K/2) packed uint8 (low
        nibble = even k). Returns int64 (R, N)."""
        A = np.ascontiguousarray(A, dtype=np.uint8)
        B = np.ascontiguousarray(B, dtype=np.uint8)
        M, KB = A.shape
        N, KBb = B.shape
        if KBb != KB:
            raise ValueError("K mismatch")
        if K is None:
            K = 2 * KB
        if K != 2 * KB:
            raise ValueError("packed width must be K/2")
        r, R = _rows_arg(rows, M)
        C = np.empty((R, N), dtype=np.int64)
        _check(self.lib.oracle_gemm_s4(M, N, K, _ptr(A), _ptr(B), _ptr(C),
                                       None if r is None else _ptr(r), R,
                                       threads or default_threads()))
        return C

    def half_to_double(self, bits) -> np.ndarray:
        """The oracle's own binary16 decode applied to each uint16 pattern."""
        b = np.asarray(bits, dtype=np.uint16).ravel()
        f = self.lib.oracle_half_to_double
        return np.array([f(int(x)) for x in b], dtype=np.float64)

    def s4_decode_bytes(self, values) -> np.ndarray:
        """The oracle's own nibble decode of each byte: (n, 2) array of
        (value at even k, value at odd k)."""
        f = self.lib.oracle_s4_value
        out = []
        for v in np.asarray(values, dtype=np.uint8).ravel():
            buf = np.array([v], dtype=np.uint8)
            out.append((f(_ptr(buf), 0), f(_ptr(buf), 1)))
        return np.array(out, dtype=np.int64)

    def s4_unpack(self, packed: np.ndarray) -> np.ndarray:
        """Decode a packed (..., K/2) INT4 array to int8 (..., K) with the
        oracle's nibble decode (through a 256-entry table it builds)."""
        table = self.s4_decode_bytes(np.arange(256))
        p = np.asarray(packed, dtype=np.uint8)
        out = np.empty(p.shape[:-1] + (2 * p.shape[-1],), dtype=np.int8)
        out[..., 0::2] = table[p, 0]
        out[..., 1::2] = table[p, 1]
        return out


_default = None


def get() -> Oracle:
    """The oracle built from oracle.c (built on first use if missing)."""
    global _default
    if _default is None:
        if not os.path.exists(_LIB_PATH):
            from oracle.build import build
            build()
        _default = Oracle(_LIB_PATH)
    return _default


def gemm_f16(A, B, rows=None, threads=None):
    return get().gemm_f16(A, B, rows=rows, threads=threads)


def gemm_s8(A, B, rows=None, threads=None):
    return get().gemm_s8(A, B, rows=rows, threads=threads)


def gemm_s4(A, B, K=None, rows=None, threads=None):
    return get().gemm_s4(A, B, K=K, rows=rows, threads=threads)


def half_to_double(bits):
    return get().half_to_double(bits)


def s4_decode_bytes(values):
    return get().s4_decode_bytes(values)


def s4_unpack(packed):
    return get().s4_unpack(packed)


def normalized_error(C_gpu: np.ndarray, C_ref: np.ndarray, D: np.ndarray) -> float:
    """max over elements of |C_gpu - C_ref| / D, with D = sum |a||b|.

    Where D == 0 the exact result is 0 and any nonzero GPU value counts as an
    infinite error; any non-finite GPU value also counts as infinite.
    """
    g = np.asarray(C_gpu, dtype=np.float64)
    if not np.all(np.isfinite(g)):
        return float("inf")
    err = np.abs(g - C_ref)
    zero = D == 0
    if np.any(err[zero] != 0):
        return float("inf")
    if np.all(zero):
        return 0.0
    return float(np.max(err[~zero] / D[~zero]))


# ----------------------------------------------------------------- scaled outputs
#
# The paper's kernels return raw sums with no dequantisation or scaling (Scope
# and Generality). The library's scaled entry point adds that step; its
# definition, written out here from scratch:
#   C[i][j] = round_out( sa[i] * sb[j] * sum_k (A(i,k) - za[i]) * (B(k,j) - zb[j]) )
# Integer inputs: the inner sum over decoded values is exact (int64 matmul of
# the zero-point-shifted operands), the scaling is done in binary64, and the
# result is rounded once, to nearest even, into the output format.

def round_bf16(x) -> np.ndarray:
    """Round binary64 values to the nearest bfloat16 value (1 sign, 8 exponent
    bits with bias 127, 7 stored fraction bits), ties to even, returned as
    binary64. Written from the format: a finite nonzero x = m * 2^e with
    0.5 <= |m| < 1 keeps 8 significant bits, m * 2^8 rounded to an integer
    (numpy's rint rounds halves to even); below the smallest normal (2^-126)
    the spacing stays 2^-133; beyond the largest finite value the result is
    infinite."""
    x = np.asarray(x, dtype=np.float64)
    out = np.array(x, copy=True)
    fin = np.isfinite(x) & (x != 0)
    m, e = np.frexp(x[fin])
    e = np.maximum(e, -125)  # subnormal range: fixed spacing 2^(-125-8)
    out[fin] = np.ldexp(np.rint(np.ldexp(x[fin], 8 - e)), e - 8)
    big = np.abs(out) > float.fromhex("0x1.fep127")
    out[big] = np.copysign(np.inf, out[big])
    return out


def round_out(x, out: str) -> np.ndarray:
    """Round binary64 values to the output type ('f32', 'f16', 'bf16'), ties to
    even, as binary64 (numpy's casts round binary64 to binary32/binary16 to
    nearest even)."""
    x = np.asarray(x, dtype=np.float64)
    if out == "f32":
        return x.astype(np.float32).astype(np.float64)
    if out == "f16":
        return x.astype(np.float16).astype(np.float64)
    if out == "bf16":
        return round_bf16(x)
    raise ValueError(out)


def _decoded(dtype, X):
    """Integer operand as int64 values, one per element (rows of K)."""
    if dtype == "s8":
        return np.asarray(X, dtype=np.int8).astype(np.int64)
    return s4_unpack(np.asarray(X, dtype=np.uint8)).astype(np.int64)


def gemm_scaled(dtype, A, B, out, sa=None, sb=None, za=None, zb=None):
    """(C_rounded, exact, D): the rounded scaled output, the binary64 value
    before rounding, and for FP16 inputs the error scale |sa||sb| sum |a||b|
    (None for integers). A is (M, K) row-major, B (N, K) = K x N column-major,
    in the storage formats of gemm_f16 / gemm_s8 / gemm_s4."""
    if dtype == "f16":
        if za is not None or zb is not None:
            raise ValueError("zero points apply to integer inputs only")
        C, D = gemm_f16(A, B)
    else:
        a, b = _decoded(dtype, A), _decoded(dtype, B)
        if za is not None:
            a = a - np.asarray(za, dtype=np.int64)[:, None]
        if zb is not None:
            b = b - np.asarray(zb, dtype=np.int64)[:, None]
        C = (a @ b.T).astype(np.float64)  # exact: |values| < 2^53
        D = None
    M, N = C.shape
    s_a = np.ones(M) if sa is None else np.asarray(sa, dtype=np.float64)
    s_b = np.ones(N) if sb is None else np.asarray(sb, dtype=np.float64)
    exact = C * s_a[:, None] * s_b[None, :]
    if D is not None:
        D = D * np.abs(s_a)[:, None] * np.abs(s_b)[None, :]
    return round_out(exact, out), exact, D
