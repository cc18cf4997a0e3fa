"""The entry point for callers that cannot allocate (mpgemm_gemm_noalloc),
through the C ABI, against the workspace entry point it mirrors
(mpgemm_gemm_ws with a caller workspace) and the CPU oracle: two calls in a
row, the second on a smaller problem, with no synchronisation between them;
split-K and stream-K shapes (the scratch holds the partial tiles and the
counters, cleared by the call) and zero points (the scratch holds the row
sums)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2608_10103_amd as mp
import seeded_inputs as si
from tests.gpu_util import assert_parity, assert_scaled, dev, oracle_gemm

pytestmark = pytest.mark.gpu

CODE = {"f16": 0, "s8": 1, "s4": 2}
OUT = {"f16": torch.float32, "s8": torch.int32, "s4": torch.int32}


def _noalloc(dtype, Ad, Bd, C, M, N, K, epi=None):
    return mp.lib().mpgemm_gemm_noalloc(CODE[dtype], M, N, K, Ad.data_ptr(), Bd.data_ptr(), C.data_ptr(),
                                        None if epi is None else ctypes.addressof(epi),
                                        torch.cuda.current_stream().cuda_stream)


def _with_ws(dtype, Ad, Bd, C, M, N, K, epi=None):
    n = mp.workspace_size(dtype, M, N, K, epi=epi)
    ws = mp.new_workspace(n, "cuda")
    code = mp.lib().mpgemm_gemm_ws(CODE[dtype], M, N, K, Ad.data_ptr(), Bd.data_ptr(), C.data_ptr(),
                                   None if epi is None else ctypes.addressof(epi), ws.data_ptr(), ws.numel(),
                                   torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return code


@pytest.mark.parametrize("dtype,shapes", [
    ("f16", [(64, 1000, 8192), (32, 500, 4096)]),      # 128 x 128 tiles split 4 ways, then a smaller split
    ("s8", [(128, 2048, 8192), (40, 1100, 2048)]),      # narrow tiles split 4 ways, then 2
    ("s4", [(100, 2000, 8192), (64, 1000, 4096)]),
])
def test_noalloc_matches_the_workspace_entry_point(dtype, shapes):
    ops, outs = [], []
    for i, (M, N, K) in enumerate(shapes):
        v = mp.select_variant(dtype, M, N, K)
        assert mp.select_splits(dtype, v, M, N, K) > 1, (dtype, M, N, K)  # the case uses the scratch
        A, B = si.gen_operands(dtype, M, N, K, seed=4100 + i)
        Ad, Bd = dev(A), dev(B)
        C = torch.full((M, N), -7, dtype=OUT[dtype], device="cuda")
        assert _noalloc(dtype, Ad, Bd, C, M, N, K) == 0
        ops.append((A, B, Ad, Bd, M, N, K))
        outs.append(C)
    torch.cuda.synchronize()
    for (A, B, Ad, Bd, M, N, K), C in zip(ops, outs):
        ref = torch.full((M, N), -9, dtype=OUT[dtype], device="cuda")
        assert _with_ws(dtype, Ad, Bd, ref, M, N, K) == 0
        assert torch.equal(C, ref), (dtype, M, N, K)  # same kernel, same split, same order
        assert_parity(dtype, C.cpu().numpy(), *oracle_gemm(dtype, A, B), f"noalloc {dtype} {M}x{N}x{K}")


@pytest.mark.parametrize("dtype", ["f16", "s8"])
def test_noalloc_stream_k(dtype):
    """Stream-K shapes (the scratch holds the split tiles' partials and the
    tile counters): two calls in a row, the second smaller with another
    schedule, against mpgemm_gemm_ws and the oracle."""
    shapes = [(2100, 2000, 6400), (2220, 1950, 4096)] if dtype == "f16" else [(2100, 2000, 12800), (2220, 1950, 8192)]
    ops, outs = [], []
    for i, (M, N, K) in enumerate(shapes):
        v = mp.select_variant(dtype, M, N, K, with_ws=True)
        assert mp.variant_name(dtype, v).endswith("_sk") and mp.sk_schedule(dtype, v, M, N, K)[1] > 1
        assert mp.workspace_size(dtype, M, N, K) <= 32 << 20
        A, B = si.gen_operands(dtype, M, N, K, seed=4300 + i)
        Ad, Bd = dev(A), dev(B)
        C = torch.full((M, N), -7, dtype=OUT[dtype], device="cuda")
        assert _noalloc(dtype, Ad, Bd, C, M, N, K) == 0
        ops.append((A, B, Ad, Bd, M, N, K))
        outs.append(C)
    torch.cuda.synchronize()
    for (A, B, Ad, Bd, M, N, K), C in zip(ops, outs):
        ref = torch.full((M, N), -9, dtype=OUT[dtype], device="cuda")
        assert _with_ws(dtype, Ad, Bd, ref, M, N, K) == 0
        assert torch.equal(C, ref), (dtype, M, N, K)
        rows = np.array(sorted(set(range(0, M, 7)) | {M - 1}))
        assert_parity(dtype, C.cpu().numpy()[rows], *oracle_gemm(dtype, A, B, rows=rows),
                      f"noalloc stream-K {dtype} {M}x{N}x{K}")


def test_noalloc_zero_points():
    """Scaled INT8 and INT4 outputs with zero points (row sums in the scratch),
    two calls in a row, the second smaller."""
    E = mp.gemm.Epilogue
    for dtype in ("s8", "s4"):
        outs = []
        for i, (M, N, K) in enumerate([(300, 520, 1024), (100, 130, 512)]):
            A, B = si.gen_operands(dtype, M, N, K, seed=4200 + i)
            rng = np.random.default_rng(i)
            sa = rng.uniform(2.0 ** -12, 2.0 ** -10, M).astype(np.float32)
            za = rng.integers(-3, 4, M).astype(np.int32)
            zb = rng.integers(-3, 4, N).astype(np.int32)
            t = [dev(x) for x in (A, B, sa, za, zb)]
            epi = E(t[2].data_ptr(), None, t[3].data_ptr(), t[4].data_ptr(), 1)
            C = torch.empty((M, N), dtype=torch.float32, device="cuda")
            assert _noalloc(dtype, t[0], t[1], C, M, N, K, epi) == 0
            outs.append((A, B, sa, za, zb, t, epi, C, M, N, K))
        torch.cuda.synchronize()
        for A, B, sa, za, zb, t, epi, C, M, N, K in outs:
            ref = torch.empty((M, N), dtype=torch.float32, device="cuda")
            assert _with_ws(dtype, t[0], t[1], ref, M, N, K, epi) == 0
            assert torch.equal(C, ref)
            _, exact, _ = oracle.gemm_scaled(dtype, A, B, "f32", sa, None, za, zb)
            assert_scaled(C, exact, None, "f32", f"noalloc zero points {dtype}")


def test_noalloc_plain_and_errors():
    """A square problem needs no scratch; argument errors as the workspace
    entry point; empty problems are no-ops."""
    A, B = si.gen_operands("s8", 512, 512, 512, seed=4300)
    Ad, Bd = dev(A), dev(B)
    C = torch.empty((512, 512), dtype=torch.int32, device="cuda")
    assert _noalloc("s8", Ad, Bd, C, 512, 512, 512) == 0
    torch.cuda.synchronize()
    assert_parity("s8", C.cpu().numpy(), *oracle_gemm("s8", A, B), "noalloc square")
    L = mp.lib()
    assert L.mpgemm_gemm_noalloc(1, -1, 512, 512, Ad.data_ptr(), Bd.data_ptr(), C.data_ptr(), None, None) == 1
    assert L.mpgemm_gemm_noalloc(7, 512, 512, 512, Ad.data_ptr(), Bd.data_ptr(), C.data_ptr(), None, None) == 1
    assert L.mpgemm_gemm_noalloc(1, 0, 512, 512, 0, 0, 0, None, None) == 0
