"""GPU parity: the HIP library through its C ABI against the CPU oracle.

Workloads: the five named configurations (FP16 512 uniform seed 0; INT8 2048
seed 1; INT4 4096 seed 2; FP16 8192 normal seed 3 on 256 sampled rows plus the
first and last; the 15-point precision x size sweep, seeds 10..24), every
compiled kernel variant on shapes spanning several tiles, closed forms and
edge cases. Integer results must match bit for bit; FP16 within a normalised
error of 1e-3.
"""
import ctypes
import re

import numpy as np
import pytest
import torch

import oracle
import paper_2608_10103_amd as mp
import seeded_inputs as si
from tests.gpu_util import F16_TOL, assert_parity, dev, gpu_gemm, oracle_gemm

pytestmark = pytest.mark.gpu

DTYPES = ("f16", "s8", "s4")
INVALID = 1  # hipErrorInvalidValue


def _log(msg):
    print(msg, flush=True)


# ---------------------------------------------------------------- named configurations


def test_f16_512_first_launch():
    """FP16 512^3, U[-1,1] seed 0, full oracle, the very first launch."""
    A, B = si.gen_operands("f16", 512, 512, 512, seed=0, dist="uniform")
    C = gpu_gemm("f16", A, B)
    ref, D = oracle_gemm("f16", A, B)
    err = assert_parity("f16", C, ref, D, "f16 512")
    _log(f"f16 512 normalised error {err:.3e}")


def test_s8_2048():
    A, B = si.gen_operands("s8", 2048, 2048, 2048, seed=1)
    assert_parity("s8", gpu_gemm("s8", A, B), *oracle_gemm("s8", A, B), "s8 2048")


def test_s4_4096():
    A, B = si.gen_operands("s4", 4096, 4096, 4096, seed=2)
    assert_parity("s4", gpu_gemm("s4", A, B), *oracle_gemm("s4", A, B), "s4 4096")


def test_f16_8192_sampled_rows():
    n = 8192
    A, B = si.gen_operands("f16", n, n, n, seed=3, dist="normal")
    C = gpu_gemm("f16", A, B)
    rows = si.sample_rows(si.F16_8192_ROW_SEED, n, si.F16_8192_ROW_COUNT, force=(0, n - 1))
    ref, D = oracle_gemm("f16", A, B, rows=rows)
    err = assert_parity("f16", C[rows], ref, D, "f16 8192 rows")
    _log(f"f16 8192 ({len(rows)} rows) normalised error {err:.3e}")


def test_f16_8192_all_ones_and_identity():
    n = 8192
    ones = torch.ones((n, n), dtype=torch.float16, device="cuda")
    C = mp.gemm_f16_f32(ones, ones)
    torch.cuda.synchronize()
    assert bool((C == float(n)).all())
    del C
    # identity: A = I, so C = B read as a K x N matrix (B stored (N, K) -> C = B^T)
    _, B = si.gen_operands("f16", 1, n, n, seed=3, dist="normal")
    eye = torch.eye(n, dtype=torch.float16, device="cuda")
    C = mp.gemm_f16_f32(eye, dev(B)).cpu().numpy()
    want = B.T.astype(np.float32)
    sub = np.abs(B.T.astype(np.float64)) < 2.0 ** -14  # binary16 subnormals (and zeros)
    assert np.array_equal(C[~sub], want[~sub])
    ok = (C[sub] == want[sub]) | (C[sub] == 0)
    assert ok.all()
    kept = int(np.sum((C[sub] == want[sub]) & (want[sub] != 0)))
    _log(f"identity 8192: {int(sub.sum())} subnormal/zero inputs, {kept} nonzero subnormals kept exactly")


SWEEP = si.sweep_points()


@pytest.mark.parametrize("dtype,n,seed", SWEEP, ids=[f"{d}-{n}" for d, n, _ in SWEEP])
def test_sweep_point(dtype, n, seed):
    """Precision x size sweep. INT8/INT4 in full at every size; FP16 in full up
    to 4096 and on the sampled-row protocol at 8192."""
    A, B = si.gen_operands(dtype, n, n, n, seed=seed)
    C = gpu_gemm(dtype, A, B)
    rows = None
    if dtype == "f16" and n == 8192:
        rows = si.sample_rows(seed + 1000, n, 256, force=(0, n - 1))
    ref, D = oracle_gemm(dtype, A, B, rows=rows)
    got = C if rows is None else C[rows]
    err = assert_parity(dtype, got, ref, D, f"{dtype} {n}")
    _log(f"sweep {dtype} {n} seed {seed}: ok (err {err:.2e}), variant "
         f"{mp.variant_name(dtype, mp.select_variant(dtype, n, n, n))}")


# ---------------------------------------------------------------- every variant


def _variant_shapes(dtype, v):
    """Shapes a variant supports that span several tiles and K-slices."""
    name = mp.variant_name(dtype, v)
    if name.startswith("generic"):
        return [(97, 65, 130), (33, 31, 66)]
    if name.startswith("skinny"):
        # at most `rows` rows on the small side (either side); whole 64-byte
        # K-steps split over 8 waves: fewer steps than waves, step counts off
        # the 4-step prefetch group, long K; ragged large side
        rows, per_wg = (int(x) for x in re.match(r"skinny(\d+)x(\d+)_", name).groups())
        e = {"f16": 32, "s8": 64, "s4": 128}[dtype]  # elements per 64-byte step
        return [(rows, 3 * per_wg + 5, 9 * e), (1, per_wg, e), (rows - 3, 700, 40 * e),
                (2 * per_wg + 7, rows, 17 * e), (300, 1, 5 * e), (rows // 2 + 1, 64, 3 * e)]
    if name.startswith("wide"):
        # 256 x 256 tiles, 128-byte K-slices (one slice, an odd count, many);
        # ragged edges (panels partly or wholly past M or N); FP16 and INT8
        if dtype == "s4":
            return []
        e = {"f16": 64, "s8": 128}[dtype]
        return [(256, 256, e), (512, 768, 3 * e), (768, 256, 5 * e), (512, 512, 33 * e), (256, 1024, 2 * e),
                (257, 513, 2 * e), (1, 255, e), (300, 77, 3 * e), (600, 700, 5 * e), (129, 1000, 4 * e)]
    if name.startswith("e2m3"):
        # INT4 with the conversion inside the GEMM: K a multiple of 256 (two
        # slices per loop iteration: 1, 5 and 8 iterations), ragged M and N
        return [(256, 256, 256), (512, 768, 1280), (300, 77, 512), (1, 255, 256), (257, 513, 768),
                (33, 65, 2048), (768, 256, 256)]
    bm, bn = (int(x) for x in re.match(r"(?:fp6)?[a-z]+(\d+)x(\d+)_", name).groups())
    if name.startswith("fp6"):
        # INT4 on the FP6 cores: any even K (zero-padded to whole stages)
        k = int(name.split("_k")[1].split("_")[0])
        return [(2 * bm, 3 * bn, 5 * k), (bm, bn, k), (2 * bm + 17, bn + 5, 3 * k + 34),
                (1, bn - 1, 2), (bm + 31, 1, 2 * k + 6), (33, 65, 4 * k - 2)]
    kb = int(name.split("_k")[1].split("_")[0])
    elems_per_kb = {"f16": kb // 2, "s8": kb, "s4": 2 * kb}[dtype]
    return [(2 * bm, 3 * bn, 5 * elems_per_kb), (bm, bn, elems_per_kb), (3 * bm, bn, 2 * elems_per_kb),
            # more K-slices than a 4- or 5-deep ring holds, not a multiple of 3
            (bm, 2 * bn, 7 * elems_per_kb),
            # more than twice what an 8-deep ring holds, ragged edges
            (bm + 3, 2 * bn - 1, 19 * elems_per_kb),
            # ragged M and N: predicated edge tiles
            (2 * bm + 17, bn + 5, 3 * elems_per_kb), (1, bn - 1, elems_per_kb), (bm + 31, 1, 2 * elems_per_kb)]


@pytest.mark.parametrize("dtype", DTYPES)
def test_every_variant(dtype):
    for v in range(mp.num_variants(dtype)):
        for (M, N, K) in _variant_shapes(dtype, v):
            assert mp.variant_supports(dtype, v, M, N, K)
            A, B = si.gen_operands(dtype, M, N, K, seed=1000 + v)
            C = gpu_gemm(dtype, A, B, variant=v)
            assert_parity(dtype, C, *oracle_gemm(dtype, A, B),
                          f"{dtype} variant {mp.variant_name(dtype, v)} {M}x{N}x{K}")
        _log(f"{dtype} variant {mp.variant_name(dtype, v)}: ok")


# ---------------------------------------------------------------- closed forms


@pytest.mark.parametrize("dtype", DTYPES)
def test_all_ones_closed_form(dtype):
    for n in (512, 4096):
        kw = n // 2 if dtype == "s4" else n
        fill = {"f16": 1.0, "s8": 1, "s4": 0x11}[dtype]
        t = torch.full((n, kw), fill, dtype={"f16": torch.float16, "s8": torch.int8,
                                            "s4": torch.uint8}[dtype], device="cuda")
        C = mp.GEMM[dtype](t, t)
        torch.cuda.synchronize()
        assert bool((C == n).all()), f"{dtype} all-ones {n}"


def test_integer_extremes():
    K = 8192
    m = torch.full((256, K), -128, dtype=torch.int8, device="cuda")
    C = mp.gemm_s8_s32(m, m)
    assert bool((C == 16384 * K).all())  # 2^27, the int32 headroom case
    p = torch.full((256, K), 127, dtype=torch.int8, device="cuda")
    assert bool((mp.gemm_s8_s32(m, p) == -16256 * K).all())
    e4 = torch.full((256, K // 2), 0x88, dtype=torch.uint8, device="cuda")  # all -8
    assert bool((mp.gemm_s4_s32(e4, e4) == 64 * K).all())
    s4 = torch.full((256, K // 2), 0x77, dtype=torch.uint8, device="cuda")  # all 7
    assert bool((mp.gemm_s4_s32(e4, s4) == -56 * K).all())
    torch.cuda.synchronize()


@pytest.mark.parametrize("dtype", ["s8", "s4"])
def test_permutation(dtype):
    """A = P (a permutation matrix): row i of C is column perm[i] of B."""
    K = N = 1024
    perm = np.random.default_rng(7).permutation(K)
    P = np.zeros((K, K), np.int8)
    P[np.arange(K), perm] = 1
    _, B = si.gen_operands(dtype, 1, N, K, seed=5)
    A = P if dtype == "s8" else si.pack_s4(P)
    C = gpu_gemm(dtype, A, B)
    Bl = B.astype(np.int64) if dtype == "s8" else oracle.s4_unpack(B).astype(np.int64)
    assert np.array_equal(C.astype(np.int64), Bl.T[perm])


def test_s4_every_nibble_through_the_api():
    """A = I (packed) and B cycling through all 256 byte values: C = B, so every
    nibble decode of the B side shows up in C; then the roles swapped."""
    K = 512
    I = si.pack_s4(np.eye(K, dtype=np.int8))
    Bb = (np.arange(256 * (K // 2)) % 256).astype(np.uint8).reshape(256, K // 2)
    Bb = np.ascontiguousarray(np.roll(Bb, 3, axis=1))
    want = np.empty((256, K), np.int64)
    lo, hi = (Bb & 0xF).astype(np.int64), (Bb >> 4).astype(np.int64)
    want[:, 0::2] = np.where(lo >= 8, lo - 16, lo)
    want[:, 1::2] = np.where(hi >= 8, hi - 16, hi)
    C = gpu_gemm("s4", I, Bb)  # (K, 256): C[k, j] = B(k, j)
    assert np.array_equal(C.astype(np.int64), want.T)
    C2 = gpu_gemm("s4", Bb, I)  # (256, K): C[i, k] = A(i, k)
    assert np.array_equal(C2.astype(np.int64), want)


@pytest.mark.parametrize("n", [512, 4096])
def test_f16_small_integers_bit_exact(n):
    """Integer-valued FP16 inputs with |v| <= 8: every partial sum is an integer
    below 2^24, so FP32 accumulation is exact in any order."""
    w = si.splitmix64(77, 0, 2 * n * n)
    vals = (si.words_to_int8(w).astype(np.int16) // 16).astype(np.float16)  # [-8, 7]
    A, B = vals[:n * n].reshape(n, n), vals[n * n:].reshape(n, n)
    C = gpu_gemm("f16", A, B)
    ref = A.astype(np.int64) @ B.astype(np.int64).T
    assert np.array_equal(C.astype(np.int64), ref)


# ---------------------------------------------------------------- edge cases


EDGE = [1, 2, 3, 31, 33, 100]


@pytest.mark.parametrize("dtype", DTYPES)
def test_edge_shapes(dtype):
    for M in EDGE:
        for N in EDGE:
            for K in (1, 2, 3, 31, 33, 100):
                if dtype == "s4" and K % 2:
                    continue
                A, B = si.gen_operands(dtype, M, N, K, seed=M * 10007 + N * 101 + K)
                C = gpu_gemm(dtype, A, B)
                assert_parity(dtype, C, *oracle_gemm(dtype, A, B), f"{dtype} {M}x{N}x{K}")


@pytest.mark.parametrize("dtype", DTYPES)
def test_ragged_large(dtype):
    """K off the slice grid goes to the bounds-checked kernel; ragged M and N
    with whole slices stay on the tiled kernels with predicated edges."""
    M, N, K = 1000, 777, 1030
    A, B = si.gen_operands(dtype, M, N, K, seed=4242)
    assert mp.select_variant(dtype, M, N, K) == 0
    assert_parity(dtype, gpu_gemm(dtype, A, B), *oracle_gemm(dtype, A, B), f"{dtype} ragged")
    for (M, N, K) in [(1000, 777, 1024), (4097, 300, 512), (16, 4096, 1024), (3000, 5, 256)]:
        A, B = si.gen_operands(dtype, M, N, K, seed=M + N + K)
        v = mp.select_variant(dtype, M, N, K)
        assert v > 0, (M, N, K)
        assert_parity(dtype, gpu_gemm(dtype, A, B), *oracle_gemm(dtype, A, B),
                      f"{dtype} {M}x{N}x{K} {mp.variant_name(dtype, v)}")


@pytest.mark.parametrize("dtype", DTYPES)
def test_k_zero_writes_zeros(dtype):
    M, N = 70, 40
    C = torch.full((M, N), 7, dtype=torch.float32 if dtype == "f16" else torch.int32,
                   device="cuda")
    kw = 0
    A = torch.empty((M, kw), dtype={"f16": torch.float16, "s8": torch.int8,
                                    "s4": torch.uint8}[dtype], device="cuda")
    B = torch.empty((N, kw), dtype=A.dtype, device="cuda")
    mp.GEMM[dtype](A, B, C=C)
    torch.cuda.synchronize()
    assert bool((C == 0).all())


def test_empty_m_or_n_is_noop():
    assert mp.raw_call("s8", 0, 5, 8, 0, 0, 0) == 0
    assert mp.raw_call("f16", 5, 0, 8, 0, 0, 0) == 0


@pytest.mark.parametrize("dtype", DTYPES)
def test_unaligned_operands(dtype):
    """Operands offset from 16-byte alignment (element-aligned) take the
    bounds-checked kernel and stay exact."""
    M, N, K = 256, 256, 256
    A, B = si.gen_operands(dtype, M, N, K, seed=99)
    esz = 2 if dtype == "f16" else 1
    kw = A.shape[1]
    raw = torch.empty(M * kw * esz + 64, dtype=torch.uint8, device="cuda")
    rawb = torch.empty(N * kw * esz + 64, dtype=torch.uint8, device="cuda")
    off = esz  # one element past a 16-byte boundary
    raw[off:off + A.nbytes].copy_(torch.from_numpy(A.view(np.uint8).ravel()).cuda())
    rawb[off:off + B.nbytes].copy_(torch.from_numpy(B.view(np.uint8).ravel()).cuda())
    C = torch.empty((M, N), dtype=torch.float32 if dtype == "f16" else torch.int32, device="cuda")
    a_ptr, b_ptr = raw.data_ptr() + off, rawb.data_ptr() + off
    assert mp.lib().mpgemm_select_variant(mp.gemm.DTYPE_CODE[dtype], M, N, K, a_ptr, b_ptr,
                                          C.data_ptr()) == 0
    code = mp.raw_call(dtype, M, N, K, a_ptr, b_ptr, C.data_ptr(),
                       torch.cuda.current_stream().cuda_stream)
    assert code == 0
    torch.cuda.synchronize()
    assert_parity(dtype, C.cpu().numpy(), *oracle_gemm(dtype, A, B), f"{dtype} unaligned")


def test_argument_errors():
    a = torch.zeros((64, 64), dtype=torch.int8, device="cuda")
    c = torch.zeros((64, 64), dtype=torch.int32, device="cuda")
    pa, pc = a.data_ptr(), c.data_ptr()
    INVALID = 1  # hipErrorInvalidValue
    assert mp.raw_call("s8", -1, 64, 64, pa, pa, pc) == INVALID
    assert mp.raw_call("s8", 64, 64, -2, pa, pa, pc) == INVALID
    assert mp.raw_call("s4", 64, 64, 63, pa, pa, pc) == INVALID  # odd K
    assert mp.raw_call("s8", 64, 64, 64, 0, pa, pc) == INVALID
    assert mp.raw_call("s8", 64, 64, 64, pa, pa, 0) == INVALID
    assert mp.raw_call("s8", 64, 64, 64, pa, pa, pa) == INVALID  # C overlaps A
    assert mp.raw_call("s8", 64, 64, 64, pa, pa, pc + 2) == INVALID  # C misaligned
    h = torch.zeros((64, 64), dtype=torch.float16, device="cuda")
    assert mp.raw_call("f16", 64, 64, 64, h.data_ptr() + 1, h.data_ptr(), pc) == INVALID
    assert mp.raw_call("s8", 64, 64, 64, pa, pa, pc, variant=99) == INVALID
    # a tiled variant refuses shapes off its tile grid
    assert mp.raw_call("s8", 100, 256, 256, pa, pa, pc, variant=1) == INVALID
    torch.cuda.synchronize()


# ---------------------------------------------------------------- determinism and streams


@pytest.mark.parametrize("dtype", DTYPES)
def test_repeat_launches_identical(dtype):
    n = 2048
    A, B = si.gen_operands(dtype, n, n, n, seed=31)
    Ad, Bd = dev(A), dev(B)
    first = mp.GEMM[dtype](Ad, Bd)
    for _ in range(4):
        again = mp.GEMM[dtype](Ad, Bd)
        torch.cuda.synchronize()
        assert torch.equal(first, again)


def test_two_streams():
    n = 1024
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    A, B = si.gen_operands("s8", n, n, n, seed=41)
    A2, B2 = si.gen_operands("s4", n, n, n, seed=42)
    Ad, Bd, A2d, B2d = dev(A), dev(B), dev(A2), dev(B2)
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        C1 = mp.gemm_s8_s32(Ad, Bd, stream=s1)
    with torch.cuda.stream(s2):
        C2 = mp.gemm_s4_s32(A2d, B2d, stream=s2)
    s1.synchronize()
    s2.synchronize()
    assert_parity("s8", C1.cpu().numpy(), *oracle_gemm("s8", A, B), "stream 1")
    assert_parity("s4", C2.cpu().numpy(), *oracle_gemm("s4", A2, B2), "stream 2")


# ---------------------------------------------------------------- INT4 on the FP6 matrix cores


def _fp6_variants():
    """Variants fed by the FP6 E3M2 conversion pre-pass (need a workspace)."""
    return [v for v in range(mp.num_variants("s4")) if mp.variant_name("s4", v).startswith("fp6")]


def _e2m3_variants():
    """Variants converting to biased FP6 E2M3 inside the GEMM (no workspace)."""
    return [v for v in range(mp.num_variants("s4")) if mp.variant_name("s4", v).startswith("e2m3")]


def _chunk_sums_hit_low_bits(a_vals, b_vals, bias, floor_bits):
    """CPU check that a test pattern can expose an accumulator narrower than
    FP32's 24 bits: the exact running sums the MFMA's FP32 accumulator holds
    after each 64-k chunk (k-chunks of 64 consecutive k, as the kernels feed
    them), in units of one product of biased values u = v + bias, include one
    of magnitude >= 2^floor_bits units whose lowest bit is set. Also returns
    whether every running sum stays below 2^24 units (the exact range)."""
    u = (np.asarray(a_vals, np.int64) + bias) * (np.asarray(b_vals, np.int64) + bias)
    run = np.cumsum(u.reshape(-1, 64).sum(axis=1))
    hit = (np.abs(run) >= 2 ** floor_bits) & (run % 2 == 1)
    return bool(hit.any()), int(run.max()) < 2 ** 24


def _pack_rows(vals):
    return si.pack_s4(np.asarray(vals, np.int8))


def _adversarial_s4(K, rows_a, rows_b, seed):
    """Three patterns per K (A rows, B rows as INT4 values), each with the
    oracle's result:
      ones-odd: A all 7, B all 7 except one k per 64-k chunk set to 6 (every
        chunk adds the odd 63 * 49 + 42 = 3129);
      mirror: the same with B negated (-7, one -6 per chunk);
      step: A = 7 (first half of K) then -7 alternating with 7 for k odd; B = 7
        (first half) then seeded values in [-8, 7]: the running sum climbs
        towards the top of the exact range, then odd terms of both signs
        arrive."""
    half = K // 2
    a1 = np.full(K, 7, np.int8)
    b1 = np.full(K, 7, np.int8)
    b1[5::64] = 6
    rng = np.random.default_rng(seed)
    a3 = np.full(K, 7, np.int8)
    a3[half:] = np.where(np.arange(K - half) % 2 == 0, -7, 7)
    b3 = np.full(K, 7, np.int8)
    b3[half:] = rng.integers(-8, 8, K - half)
    out = []
    for name, av, bv in (("ones-odd", a1, b1), ("mirror", a1, -b1), ("step", a3, b3)):
        out.append((name, av, bv, _pack_rows(np.tile(av, (rows_a, 1))), _pack_rows(np.tile(bv, (rows_b, 1)))))
    return out


@pytest.mark.parametrize("K", [8192, 1 << 17, 1 << 18])
def test_fp6_prepass_exact_at_large_sums(K):
    """The FP6 E3M2 pre-pass kernels accumulate exact integers in FP32: the
    adversarial patterns drive the running sums to 2^20..2^23.6 with odd low
    bits (checked on the CPU first), on every such variant, on a whole
    256 x 256 tile and a ragged 33 x 65 one, bit-exact against the oracle."""
    cases = _adversarial_s4(K, 256, 256, seed=K)
    for name, av, bv, A, B in cases:
        if K >= 1 << 17:
            hit, fits = _chunk_sums_hit_low_bits(av, bv, 0, 20)
            assert fits
            assert hit, f"{name} K={K}: no odd running sum above 2^20"
        ref = oracle.gemm_s4(A, B)
        ref_r = ref[:33, :65]
        for v in _fp6_variants():
            vn = mp.variant_name("s4", v)
            _log(f"fp6 pre-pass {vn} K={K} {name}")
            C = gpu_gemm("s4", A, B, variant=v)
            assert np.array_equal(C.astype(np.int64), ref), (vn, name, K)
            C = gpu_gemm("s4", A[:33], B[:65], variant=v)
            assert np.array_equal(C.astype(np.int64), ref_r), (vn, name, K, "ragged")


@pytest.mark.parametrize("K", [8192, 1 << 15, 1 << 16])
def test_e2m3_exact_at_large_sums(K):
    """The INT4 kernel with the conversion inside the GEMM holds biased sums
    sum (a + 8)(b + 8) / 64 in FP32: the same patterns drive them to
    2^22..2^23.8 units of 1/64 with odd low bits (checked on the CPU), on
    every such variant, whole tiles and ragged ones, and through gemm_s4_s32,
    bit-exact against the oracle."""
    cases = _adversarial_s4(K, 256, 512, seed=K + 1)
    for name, av, bv, A, B in cases:
        if K == 1 << 16:
            hit, fits = _chunk_sums_hit_low_bits(av, bv, 8, 22)
            assert fits, f"{name}: biased sum leaves the exact range"
            # in the biased domain the mirror's products are small (u_b = 1, 2)
            assert hit or name == "mirror", f"{name} K={K}: no odd running sum above 2^22"
        ref = oracle.gemm_s4(A, B)
        for v in _e2m3_variants():
            vn = mp.variant_name("s4", v)
            _log(f"e2m3 {vn} K={K} {name}")
            C = gpu_gemm("s4", A, B, variant=v)
            assert np.array_equal(C.astype(np.int64), ref), (vn, name, K)
            C = gpu_gemm("s4", A[:33], B[:65], variant=v)
            assert np.array_equal(C.astype(np.int64), ref[:33, :65]), (vn, name, K, "ragged")
        C = gpu_gemm("s4", A, B)  # the entry point's own choice
        assert np.array_equal(C.astype(np.int64), ref), (name, K, "entry point")


def test_s4_4096_adversarial_through_the_entry_point():
    """gemm_s4_s32 at 4096^3 on the adversarial patterns (the INT4 sweep's
    configuration size), bit-exact."""
    n = 4096
    v = mp.select_variant("s4", n, n, n)
    assert mp.variant_name("s4", v).startswith("e2m3")
    for name, av, bv, A, B in _adversarial_s4(n, n, n, seed=44):
        C = gpu_gemm("s4", A, B)
        rows = np.array([0, 1, 2047, n - 1])
        ref = oracle.gemm_s4(A, B, rows=rows)
        assert np.array_equal(C[rows].astype(np.int64), ref), name
        assert np.all(C == C[0, 0]), name  # identical rows of A and of B: one value


def test_fp6_prepass_one_workspace_in_one_stream():
    """Back-to-back FP6 pre-pass calls of growing and shrinking size on one
    stream, no synchronisation between them, all sharing one caller
    workspace sized for the largest (calls in order on a stream may share
    one)."""
    v = max(_fp6_variants(), key=lambda x: mp.variant_name("s4", x).startswith("fp6pipe128"))
    shapes = [(512, 384, 512), (2048, 1536, 1024), (256, 128, 4096), (1024, 1024, 2050)]
    ws = mp.new_workspace(max(mp.workspace_size("s4", *sh, variant=v) for sh in shapes), "cuda")
    cases = []
    for i, (M, N, K) in enumerate(shapes):
        A, B = si.gen_operands("s4", M, N, K, seed=300 + i)
        cases.append((A, B, mp.gemm_s4_s32(dev(A), dev(B), variant=v, workspace=ws)))
    torch.cuda.synchronize()
    for A, B, C in cases:
        assert np.array_equal(C.cpu().numpy().astype(np.int64), oracle.gemm_s4(A, B))


def test_fp6_two_streams():
    """Two FP6 pre-pass INT4 GEMMs in flight on two streams at once, each with
    its own workspace; and two in-GEMM-conversion ones (no workspace)."""
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    A1, B1 = si.gen_operands("s4", 2048, 2048, 2048, seed=51)
    A2, B2 = si.gen_operands("s4", 1024, 768, 4096, seed=52)
    d = [dev(x) for x in (A1, B1, A2, B2)]
    for v in (_fp6_variants()[0], _e2m3_variants()[0]):
        w1 = mp.new_workspace(mp.workspace_size("s4", 2048, 2048, 2048, variant=v), "cuda")
        w2 = mp.new_workspace(mp.workspace_size("s4", 1024, 768, 4096, variant=v), "cuda")
        torch.cuda.synchronize()
        with torch.cuda.stream(s1):
            C1 = mp.gemm_s4_s32(d[0], d[1], stream=s1, variant=v, workspace=w1)
        with torch.cuda.stream(s2):
            C2 = mp.gemm_s4_s32(d[2], d[3], stream=s2, variant=v, workspace=w2)
        s1.synchronize()
        s2.synchronize()
        assert np.array_equal(C1.cpu().numpy().astype(np.int64), oracle.gemm_s4(A1, B1))
        assert np.array_equal(C2.cpu().numpy().astype(np.int64), oracle.gemm_s4(A2, B2))


def test_s4_4096_in_a_hip_graph():
    """gemm_s4_s32 at 4096^3 recorded into a HIP graph (it allocates, frees
    and synchronises nothing) and replayed three times, with eager work and
    synchronisation between the replays; every replay bit-exact."""
    n = 4096
    A, B = si.gen_operands("s4", n, n, n, seed=2)
    Ad, Bd = dev(A), dev(B)
    C = torch.empty((n, n), dtype=torch.int32, device="cuda")
    eager = mp.gemm_s4_s32(Ad, Bd)
    torch.cuda.synchronize()
    rows = np.array([0, 1, 1234, n - 1])
    assert np.array_equal(eager.cpu().numpy()[rows].astype(np.int64), oracle.gemm_s4(A, B, rows=rows))
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        mp.gemm_s4_s32(Ad, Bd, C=C, stream=s)
    for r in range(3):
        C.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(C, eager), f"replay {r}"
        junk = mp.gemm_s4_s32(Bd, Ad)  # eager work between the replays
        torch.cuda.synchronize()
        del junk


# ---------------------------------------------------------------- split-K and LLM-inference shapes


def _pipelined_variants(dtype):
    """The variants that split K (the stream-K ones do not)."""
    return [v for v in range(mp.num_variants(dtype))
            if mp.variant_name(dtype, v).startswith(("pipe", "spread")) and not mp.variant_name(dtype, v).endswith("_sk")]


@pytest.mark.parametrize("dtype", DTYPES)
def test_splitk_every_pipelined_variant(dtype):
    """Every split-capable variant with 2, 3 and 4 K-ranges on ragged shapes
    spanning several tiles (caller workspaces): bit-exact integers, FP16
    within the bound."""
    for v in _pipelined_variants(dtype):
        name = mp.variant_name(dtype, v)
        bm, bn = (int(x) for x in re.match(r"[a-z]+(\d+)x(\d+)_", name).groups())
        kb = int(name.split("_k")[1].split("_")[0])
        e = {"f16": kb // 2, "s8": kb, "s4": 2 * kb}[dtype]
        for splits, (M, N, K) in [(2, (bm + 17, 2 * bn - 3, 4 * e)), (3, (2 * bm, bn + 1, 6 * e)),
                                  (4, (1, bn, 8 * e)), (4, (bm - 5, 3 * bn, 4 * e))]:
            A, B = si.gen_operands(dtype, M, N, K, seed=700 + v + splits)
            C = gpu_gemm(dtype, A, B, variant=v, splits=splits)
            assert_parity(dtype, C, *oracle_gemm(dtype, A, B), f"{dtype} {name} splits {splits} {M}x{N}x{K}")
        _log(f"{dtype} split-K {name}: ok")


@pytest.mark.parametrize("dtype", DTYPES)
def test_llm_inference_shapes(dtype):
    """Skinny GEMMs of LLM inference (M tokens x N outputs x K inputs) through
    the entry point (no workspace: never split) and through mpgemm_gemm_ws
    with a workspace (split where the choice splits), whatever kernel it
    picks."""
    for (M, N, K) in [(1, 4096, 4096), (16, 4096, 4096), (64, 8192, 4096), (128, 4096, 8192),
                      (256, 4096, 4096), (16, 14336, 4096), (7, 1000, 2048),
                      # the narrow tiles, mirrored when N is the small side
                      (48, 4096, 2048), (2048, 48, 2048), (4096, 128, 1024), (200, 2048, 1024),
                      # the narrow tiles with the eight-slice ring (FP16, INT8), ragged sides
                      (9, 8192, 8192), (16, 8192, 4096), (8192, 16, 4096), (8192, 100, 8192),
                      # 257 .. 512 rows: narrow tiles in place of 128 x 128
                      (384, 2048, 4096), (4096, 500, 4096), (320, 4096, 2048),
                      # under half the CUs with 128 x 128 tiles: narrow tiles, ragged
                      (1100, 1300, 2048), (700, 700, 4096),
                      # 272 tiles of 128 x 128: stream-K with a workspace
                      (2100, 2000, 6400)]:
        A, B = si.gen_operands(dtype, M, N, K, seed=M + N + K)
        ref = oracle_gemm(dtype, A, B)
        v = mp.select_variant(dtype, M, N, K)
        assert_parity(dtype, gpu_gemm(dtype, A, B), *ref, f"{dtype} {M}x{N}x{K} {mp.variant_name(dtype, v)}")
        assert_parity(dtype, gpu_gemm(dtype, A, B, workspace="auto"), *ref,
                      f"{dtype} {M}x{N}x{K} {mp.variant_name(dtype, v)} splits {mp.select_splits(dtype, v, M, N, K)}")
    _log(f"{dtype} LLM shapes: ok")


def _random_shapes(seed, n):
    """Seeded shapes across the automatic choice's regions: the streaming
    kernel (1..7 rows), narrow and eight-slice narrow tiles (8..1024 rows),
    tiles leaving CUs idle (up to 1408 square-ish), 128 x 128 and 256 x 256,
    either side small, ragged sides, K off the big multiples (but on the
    128-byte grid of every precision, a multiple of 256 elements)."""
    rng = np.random.default_rng(seed)
    small = [1, 3, 7, 8, 12, 16, 33, 64, 100, 128, 200, 257, 320, 500, 640, 777, 1000, 1100, 1300]
    large = [1024, 1500, 2048, 3000, 4096, 5000, 8192]
    out = []
    for _ in range(n):
        a = int(rng.choice(small))
        b = int(rng.choice(large)) if a <= 1024 else int(rng.integers(a, 1409))
        K = 256 * int(rng.integers(1, 33))
        out.append((a, b, K) if rng.random() < 0.6 else (b, a, K))
    return out


@pytest.mark.parametrize("dtype", DTYPES)
def test_automatic_choice_random_shapes(dtype):
    """Whatever kernel the entry point picks, with and without a workspace,
    on seeded shapes across every region of the choice: sampled rows against
    the oracle (first, last and four seeded rows)."""
    # plus a ragged INT4 shape past 144 tiles of 256 x 256 (the 8-wave FP6
    # kernel with a workspace, the 128 x 128 one without)
    for i, (M, N, K) in enumerate(_random_shapes(4242 + DTYPES.index(dtype), 16) + [(3200, 6528, 1024)]):
        A, B = si.gen_operands(dtype, M, N, K, seed=5000 + i)
        rng = np.random.default_rng(i)
        rows = np.unique(np.concatenate([[0, M - 1], rng.integers(0, M, 4)]))
        ref = oracle_gemm(dtype, A, B, rows=rows)
        v = mp.select_variant(dtype, M, N, K)
        vw = mp.select_variant(dtype, M, N, K, with_ws=True)
        _log(f"random {dtype} {M}x{N}x{K}: {mp.variant_name(dtype, v)} / ws {mp.variant_name(dtype, vw)}")
        assert_parity(dtype, gpu_gemm(dtype, A, B)[rows], *ref, f"{dtype} {M}x{N}x{K} {mp.variant_name(dtype, v)}")
        assert_parity(dtype, gpu_gemm(dtype, A, B, workspace="auto")[rows], *ref,
                      f"{dtype} {M}x{N}x{K} ws {mp.variant_name(dtype, vw)}")


@pytest.mark.parametrize("dtype", DTYPES)
def test_splitk_deterministic_and_concurrent(dtype):
    """Split results do not depend on which workgroup finishes last (five
    launches on one reused workspace bit-identical: each call leaves its
    counters zero), and two split-K GEMMs on two streams at once, each with
    its own workspace."""
    v = [x for x in _pipelined_variants(dtype) if mp.variant_name(dtype, x) == "spread128x128_w2x2_k64_s4"][0]
    A, B = si.gen_operands(dtype, 512, 640, 2048, seed=91)
    Ad, Bd = dev(A), dev(B)
    ws = mp.new_workspace(mp.workspace_size(dtype, 512, 640, 2048, variant=v, splits=8), "cuda")
    first = mp.GEMM[dtype](Ad, Bd, variant=v, splits=8, workspace=ws)
    for _ in range(4):
        assert torch.equal(first, mp.GEMM[dtype](Ad, Bd, variant=v, splits=8, workspace=ws))
    torch.cuda.synchronize()
    assert_parity(dtype, first.cpu().numpy(), *oracle_gemm(dtype, A, B), f"{dtype} split 8")
    A2, B2 = si.gen_operands(dtype, 384, 256, 4096, seed=92)
    A2d, B2d = dev(A2), dev(B2)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    w1 = mp.new_workspace(mp.workspace_size(dtype, 512, 640, 2048, variant=v, splits=4), "cuda")
    w2 = mp.new_workspace(mp.workspace_size(dtype, 384, 256, 4096, variant=v, splits=16), "cuda")
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        C1 = mp.GEMM[dtype](Ad, Bd, variant=v, splits=4, stream=s1, workspace=w1)
    with torch.cuda.stream(s2):
        C2 = mp.GEMM[dtype](A2d, B2d, variant=v, splits=16, stream=s2, workspace=w2)
    s1.synchronize()
    s2.synchronize()
    assert_parity(dtype, C1.cpu().numpy(), *oracle_gemm(dtype, A, B), f"{dtype} stream 1")
    assert_parity(dtype, C2.cpu().numpy(), *oracle_gemm(dtype, A2, B2), f"{dtype} stream 2")


def test_splitk_argument_errors():
    v = [x for x in _pipelined_variants("s8") if mp.variant_name("s8", x) == "spread128x128_w2x2_k64_s4"][0]
    t = torch.zeros((256, 1024), dtype=torch.int8, device="cuda")
    L = mp.lib()
    c = torch.zeros((256, 256), dtype=torch.int32, device="cuda")
    ws = mp.new_workspace(mp.workspace_size("s8", 256, 256, 1024, variant=v, splits=16), "cuda")
    run = lambda var, sp, K, w=ws.data_ptr(), n=ws.numel(): L.mpgemm_run_variant_ws(
        1, var, sp, 256, 256, K, t.data_ptr(), t.data_ptr(), c.data_ptr(), None, w, n, 0)
    assert run(v, -1, 1024) == INVALID
    assert run(v, 17, 1024) == INVALID
    assert run(v, 3, 1024) == INVALID  # 16 slices do not split in 3
    assert run(0, 2, 1024) == INVALID  # the bounds-checked kernel does not split
    assert run(v, 16, 1024, None, 0) == INVALID  # a split needs a workspace
    assert run(v, 16, 1024, ws.data_ptr(), 4096) == INVALID  # too small for it
    assert run(v, 16, 1024) == 0
    torch.cuda.synchronize()


# ---------------------------------------------------------------- stream-K


def _named(dtype, name):
    return [v for v in range(mp.num_variants(dtype)) if mp.variant_name(dtype, v) == name][0]


SK_WIDE, SK_PIPE, SK_SPREAD = ("wide256x256_w2x2_k128_m16_sk", "pipe256x256_w2x4_k128_s2_sk",
                               "spread128x128_w2x2_k128_s4_sk")
SK_F6 = "fp6wide256x256_w2x2_k128_s3_sk"  # INT4 on the FP6 cores, converted operands
SK_W8, SK_W8K64 = "spread128x128_w2x4_k128_s4_sk", "spread128x128_w2x4_k64_s4_sk"  # eight waves of 64 x 32
# tile counts just past one or two rounds of 256 workgroups (one per CU),
# K deep enough for the schedule to split the remaining tiles
SK_CASES = [
    ("f16", SK_WIDE, 4352, 4096, 4096),    # 272 tiles: 256 whole, 16 in 4 parts
    ("s8", SK_WIDE, 6144, 6400, 8192),     # 600 = 2 x 256 + 88 tiles, 2 parts
    ("f16", SK_WIDE, 2048, 2048, 8192),    # 64 tiles, all split
    ("s8", SK_WIDE, 4352, 4096, 6400),     # 50 slices in 3 parts of 16 or 17
    ("f16", SK_PIPE, 4000, 4400, 3200),    # ragged edges, 288 tiles
    ("s8", SK_PIPE, 4000, 4400, 6400),
    ("s4", SK_PIPE, 4000, 4400, 12800),
    ("f16", SK_SPREAD, 2100, 2000, 3200),  # 272 tiles of 128 x 128
    ("s8", SK_SPREAD, 128 * 16 + 5, 128 * 16, 8192),
    ("s4", SK_SPREAD, 2100, 2000, 12800),
    ("s4", SK_SPREAD, 128 * 23 + 5, 128 * 12, 16384),
    ("s4", SK_F6, 4352, 4096, 16384),      # 272 tiles: 16 in 4 parts of 32 slices
    ("s4", SK_F6, 6144, 6400, 32768),      # 600 tiles: 88 in 2 parts
    ("s4", SK_F6, 4000, 4400, 32768),      # ragged edges (shared epilogue), 288 tiles
    ("s4", SK_F6, 1000, 700, 30000),       # 12 tiles, all split; K padded to 30208
    ("f16", SK_WIDE, 4300, 4100, 4096),    # ragged edges: 289 tiles, 33 in 4 parts
    ("s8", SK_WIDE, 4300, 4100, 8192),
    ("f16", SK_W8, 2100, 2000, 3200),      # 272 tiles of 128 x 128, 3 parts
    ("s8", SK_W8, 2100, 2000, 8192),
    ("s4", SK_W8K64, 2100, 2000, 12800),   # 64-byte slices
    ("s4", SK_W8K64, 128 * 23 + 5, 128 * 12, 16384),
]


@pytest.mark.parametrize("dtype,name,M,N,K", SK_CASES, ids=[f"{c[0]}-{c[1][:-3]}-{c[2]}x{c[3]}x{c[4]}" for c in SK_CASES])
def test_stream_k_parity(dtype, name, M, N, K):
    """Stream-K variants where their schedule splits tiles into K-parts:
    every 13th row (and the last) against the oracle (bit-exact integers,
    FP16 within the bound), four launches on one workspace bit-identical
    (the sum does not depend on which part finishes last), the counter block
    left zero, and the same variant without a workspace (every tile whole):
    integers bit-identical over the whole output, FP16 on the sampled rows."""
    v = _named(dtype, name)
    dp, parts, grid = mp.sk_schedule(dtype, v, M, N, K)
    _log(f"stream-K {dtype} {name} {M}x{N}x{K}: {dp} whole tiles, then {parts} parts per tile, grid {grid}")
    assert parts > 1
    A, B = si.gen_operands(dtype, M, N, K, seed=M + N + K)
    Ad, Bd = dev(A), dev(B)
    ws = mp.new_workspace(mp.workspace_size(dtype, M, N, K, variant=v, splits=1), "cuda")
    C = mp.GEMM[dtype](Ad, Bd, variant=v, workspace=ws)
    for _ in range(3):
        assert torch.equal(C, mp.GEMM[dtype](Ad, Bd, variant=v, workspace=ws))
    # whole tiles: no room for partial tiles (the FP6 kernel still needs its
    # converted operands: a workspace of the whole-tile kernel's size)
    whole_ws = None
    if name == SK_F6:
        base = _named(dtype, name[:-3])
        whole_ws = mp.new_workspace(mp.workspace_size(dtype, M, N, K, variant=base, splits=1), "cuda")
    whole = mp.GEMM[dtype](Ad, Bd, variant=v, workspace=whole_ws)
    torch.cuda.synchronize()
    assert int(ws[:65536].count_nonzero()) == 0, "counters left non-zero"
    rows = np.array(sorted(set(range(0, M, 13)) | {M - 1}))
    ref = oracle_gemm(dtype, A, B, rows=rows)
    assert_parity(dtype, C.cpu().numpy()[rows], *ref, f"stream-K {dtype} {name} {M}x{N}x{K}")
    if dtype == "f16":
        assert_parity(dtype, whole.cpu().numpy()[rows], *ref, f"whole tiles {dtype} {name} {M}x{N}x{K}")
    else:
        assert torch.equal(C, whole)


@pytest.mark.parametrize("dtype", DTYPES)
def test_stream_k_scaled(dtype):
    """The scaled epilogue (and zero points for integers) through stream-K
    on the one-wave-per-SIMD kernels (FP16, INT8; INT4 on the FP6 cores) and
    the 128 x 128 one."""
    cases = [(SK_SPREAD, 2100, 2000, {"f16": 3200, "s8": 6400, "s4": 12800}[dtype]),
             (SK_W8K64 if dtype == "s4" else SK_W8, 2100, 2000, {"f16": 3200, "s8": 6400, "s4": 12800}[dtype])]
    if dtype != "s4":
        cases.append((SK_WIDE, 2048, 2048, {"f16": 4096, "s8": 8192}[dtype]))
    else:
        cases.append((SK_F6, 500, 700, 30000))  # 6 tiles in 5 parts, ragged
    for i, (name, M, N, K) in enumerate(cases):
        v = _named(dtype, name)
        assert mp.sk_schedule(dtype, v, M, N, K)[1] > 1
        out = OUTS[i % 3]
        zp = dtype != "f16"
        A, B = si.gen_operands(dtype, M, N, K, seed=2100 + i)
        sa, sb, za, zb = _scales(dtype, M, N, 2200 + i, zp)
        _log(f"stream-K scaled {dtype} {name} {M}x{N}x{K} {out}")
        C = _run_scaled(dtype, A, B, out, sa, sb, za, zb, variant=v)
        _, exact, D = oracle.gemm_scaled(dtype, A, B, out, sa, sb, za, zb)
        assert_scaled(C, exact, D, out, f"stream-K {dtype} {name} {M}x{N}x{K} {out} zp={zp}")


@pytest.mark.parametrize("dtype,K", [("f16", 8192), ("s8", 16384), ("s4", 16384)])
def test_stream_k_through_the_entry_point(dtype, K):
    """272 tiles of 256 x 256 with a workspace sized by the library for its
    own choice: the entry point takes the stream-K twin of its whole-tile
    kernel (INT4: the FP6 pre-pass one) and matches the oracle on sampled
    rows."""
    M, N = 4352, 4096
    v = mp.select_variant(dtype, M, N, K, with_ws=True)
    assert mp.variant_name(dtype, v).endswith("_sk") and mp.sk_schedule(dtype, v, M, N, K)[1] > 1
    _log(f"stream-K entry point {dtype} {M}x{N}x{K}: {mp.variant_name(dtype, v)}")
    A, B = si.gen_operands(dtype, M, N, K, seed=K + 7)
    C = mp.GEMM[dtype](dev(A), dev(B), workspace="auto")
    rows = np.array([0, 1, 255, 256, 2047, 4095, 4096, 4351])
    assert_parity(dtype, C.cpu().numpy()[rows], *oracle_gemm(dtype, A, B, rows=rows),
                  f"stream-K entry point {dtype} {M}x{N}x{K}")


def test_stream_k_wide_below_a_round_fp16():
    """FP16 with a workspace, 96 tiles of 256 x 256 and 128 K-slices: the
    entry point takes the one-wave-per-SIMD kernel's stream-K schedule over
    the 128 x 128 kernel, and matches the oracle on sampled rows."""
    M, N, K = 768, 8192, 8192
    v = mp.select_variant("f16", M, N, K, with_ws=True)
    assert mp.variant_name("f16", v) == "wide256x256_w2x2_k128_m16_sk"
    A, B = si.gen_operands("f16", M, N, K, seed=77)
    C = mp.GEMM["f16"](dev(A), dev(B), workspace="auto")
    rows = np.array([0, 1, 255, 256, 511, 767])
    assert_parity("f16", C.cpu().numpy()[rows], *oracle_gemm("f16", A, B, rows=rows), "stream-K wide f16 768")
    _log(f"stream-K wide below a round: {mp.sk_schedule('f16', v, M, N, K)}")


# ---------------------------------------------------------------- scaled outputs (fused epilogue)

from tests.gpu_util import TORCH_OUT, assert_scaled  # noqa: E402

OUTS = ("f32", "f16", "bf16")


def _scales(dtype, M, N, seed, zero_points):
    """Seeded scales that keep outputs inside FP16's range, optional zero points."""
    rng = np.random.default_rng(seed)
    lo, hi = {"f16": (0.5, 2.0), "s8": (2.0 ** -14, 2.0 ** -10), "s4": (2.0 ** -8, 2.0 ** -4)}[dtype]
    sa = rng.uniform(lo, hi, M).astype(np.float32)
    sb = rng.uniform(0.5, 2.0, N).astype(np.float32)
    za = zb = None
    if zero_points:
        r = 8 if dtype == "s8" else 3
        za = rng.integers(-r, r + 1, M).astype(np.int32)
        zb = rng.integers(-r, r + 1, N).astype(np.int32)
    return sa, sb, za, zb


def _run_scaled(dtype, A, B, out, sa, sb, za, zb, variant=None, splits=None):
    t = lambda x: None if x is None else dev(x)
    ws = "auto" if (variant is not None or za is not None or zb is not None) else None
    C = mp.gemm_scaled(dtype, dev(A), dev(B), t(sa), t(sb), t(za), t(zb), out_dtype=TORCH_OUT[out],
                       variant=variant, splits=splits, workspace=ws)
    torch.cuda.synchronize()
    return C


@pytest.mark.parametrize("dtype", DTYPES)
def test_scaled_epilogue_every_kernel(dtype):
    """Every kernel variant's epilogue with scales (and, for integers, zero
    points on every other variant), output types in rotation, on a ragged
    shape spanning several tiles."""
    for v in range(mp.num_variants(dtype)):
        shapes = _variant_shapes(dtype, v)
        if not shapes:  # a variant without a kernel for this dtype
            assert not mp.variant_supports(dtype, v, 256, 256, 1024)
            continue
        # the first shape with an odd side (a ragged edge tile), both sides above one
        M, N, K = next(s for s in shapes if (s[0] % 2 or s[1] % 2) and min(s[0], s[1]) > 1)
        out = OUTS[v % 3]
        zp = dtype != "f16" and v % 2 == 1
        A, B = si.gen_operands(dtype, M, N, K, seed=1500 + v)
        sa, sb, za, zb = _scales(dtype, M, N, 1600 + v, zp)
        C = _run_scaled(dtype, A, B, out, sa, sb, za, zb, variant=v)
        _, exact, D = oracle.gemm_scaled(dtype, A, B, out, sa, sb, za, zb)
        assert_scaled(C, exact, D, out, f"{dtype} {mp.variant_name(dtype, v)} {M}x{N}x{K} {out} zp={zp}")
    _log(f"{dtype} scaled epilogue, every variant: ok")


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("out", OUTS)
def test_scaled_entry_point(dtype, out):
    """Through gemm_scaled with the library's own kernel choice: a square tiled
    problem, a skinny split-K one, one-sided scales and zero points."""
    for i, (M, N, K, zp, one_sided) in enumerate([(512, 640, 1024, False, False), (16, 2048, 4096, True, False),
                                                   (300, 257, 512, True, True), (64, 64, 0, True, False)]):
        zp = zp and dtype != "f16"
        A, B = si.gen_operands(dtype, M, N, K, seed=1700 + i)
        sa, sb, za, zb = _scales(dtype, M, N, 1800 + i, zp)
        if one_sided:
            sb, za = None, None
        C = _run_scaled(dtype, A, B, out, sa, sb, za, zb)
        _, exact, D = oracle.gemm_scaled(dtype, A, B, out, sa, sb, za, zb)
        assert_scaled(C, exact, D, out, f"{dtype} {M}x{N}x{K} {out}")


def test_scaled_argument_errors():
    L = mp.lib()
    t = torch.zeros((64, 64), dtype=torch.int8, device="cuda")
    h = torch.zeros((64, 64), dtype=torch.float16, device="cuda")
    c = torch.zeros((64, 64), dtype=torch.float16, device="cuda")
    s = torch.ones(64, dtype=torch.float32, device="cuda")
    z = torch.zeros(64, dtype=torch.int32, device="cuda")
    E = mp.gemm.Epilogue
    call = lambda dt, A, epi, cptr=c.data_ptr(): L.gemm_scaled(dt, 64, 64, 64, A.data_ptr(), A.data_ptr(), cptr,
                                                               None if epi is None else ctypes.addressof(epi), 0)
    assert call(1, t, None) == INVALID
    assert call(1, t, E(s.data_ptr(), None, None, None, 0)) == INVALID      # no output type
    assert call(1, t, E(s.data_ptr(), None, None, None, 4)) == INVALID      # unknown output type
    assert call(0, h, E(None, None, z.data_ptr(), None, 2)) == INVALID      # zero points with FP16
    assert call(1, t, E(s.data_ptr() + 2, None, None, None, 2)) == INVALID  # misaligned scales
    assert call(1, t, E(None, None, None, None, 1), c.data_ptr() + 2) == INVALID  # FP32 output: 4-byte C
    assert call(1, t, E(None, None, None, None, 2), c.data_ptr() + 1) == INVALID  # FP16 output: 2-byte C
    assert call(1, t, E(None, None, z.data_ptr(), None, 2)) == INVALID      # zero points need a workspace
    assert call(1, t, E(s.data_ptr(), s.data_ptr(), None, None, 3)) == 0
    ws = mp.new_workspace(1 << 17, "cuda")
    epi = E(s.data_ptr(), s.data_ptr(), z.data_ptr(), z.data_ptr(), 3)
    assert L.mpgemm_gemm_ws(1, 64, 64, 64, t.data_ptr(), t.data_ptr(), c.data_ptr(), ctypes.addressof(epi),
                            ws.data_ptr(), ws.numel(), 0) == 0
    torch.cuda.synchronize()


# ------------------------------------------------- B stored K x N row-major


def _gpu_gemm_bt(dtype, A, B_kn):
    C = mp.gemm_bt(dtype, dev(A), dev(B_kn))
    torch.cuda.synchronize()
    return C.cpu().numpy()


def _to_kn(dtype, B):
    """The oracle's B (N rows of K, INT4 packed along K) as the transposed-B
    entry point takes it: K x N row-major (INT4 packed along N)."""
    if dtype == "s4":
        return si.pack_s4(np.ascontiguousarray(oracle.s4_unpack(B).T))
    return np.ascontiguousarray(B.T)


KSLICE = {"f16": 64, "s8": 128, "s4": 256}


@pytest.mark.parametrize("dtype", ["f16", "s8", "s4"])
def test_transposed_b_parity(dtype):
    """mpgemm_gemm_bt (B(k, j) at k * N + j; INT4 packed along N) against the
    oracle on the same B transposed on the host to the oracle's N rows of K:
    several tiles and K-slices, the 2-slice ring's steady state and tail,
    ragged M."""
    kslice = KSLICE[dtype]
    for (M, N, K) in [(256, 256, kslice), (512, 768, 5 * kslice), (300, 256, 3 * kslice),
                      (1, 512, 2 * kslice), (777, 1024, 7 * kslice)]:
        A, B = si.gen_operands(dtype, M, N, K, seed=900 + M + N + K)  # B: N rows of K
        C = _gpu_gemm_bt(dtype, A, _to_kn(dtype, B))
        assert_parity(dtype, C, *oracle_gemm(dtype, A, B), f"{dtype} transposed B {M}x{N}x{K}")
    _log(f"{dtype} transposed B: ok")


@pytest.mark.parametrize("dtype", ["f16", "s8", "s4"])
def test_transposed_b_full_size_sampled_rows(dtype):
    """N = 8192 (the measured size): 40 sampled rows against the oracle."""
    n = 8192
    A, B = si.gen_operands(dtype, n, n, n, seed=31)
    C = _gpu_gemm_bt(dtype, A, _to_kn(dtype, B))
    rows = np.random.default_rng(31).choice(n, size=38, replace=False).tolist() + [0, n - 1]
    C_ref, D = oracle_gemm(dtype, A, B, rows=rows)
    assert_parity(dtype, C[rows], C_ref, D, f"{dtype} transposed B {n}^3 sampled rows")


def test_transposed_b_closed_forms():
    """Identity as B: C = A exactly (integer-valued FP16, INT8, INT4); all-ones:
    C = K; INT4: every nibble value in every position of B's packed rows."""
    for dtype, K in (("f16", 256), ("s8", 256), ("s4", 512)):
        M = N = 256
        vals = np.random.default_rng(5).integers(-8, 8, size=(M, K))
        if dtype == "s4":
            A = si.pack_s4(vals.astype(np.int8))
            eye = si.pack_s4(np.eye(K, N, dtype=np.int8))
            ones_a = np.full((M, K // 2), 0x11, np.uint8)
            ones_b = np.full((K, N // 2), 0x11, np.uint8)
        else:
            A = vals.astype(np.float16) if dtype == "f16" else vals.astype(np.int8)
            eye = np.eye(K, N, dtype=A.dtype)
            ones_a, ones_b = np.ones((M, K), dtype=A.dtype), np.ones((K, N), dtype=A.dtype)
        C = _gpu_gemm_bt(dtype, A, eye)
        want = vals[:, :N].astype(np.float32 if dtype == "f16" else np.int32)
        assert np.array_equal(C, want), dtype
        assert np.all(_gpu_gemm_bt(dtype, ones_a, ones_b) == K), dtype
    # INT4: A = I (K = 512) and B cycling through all 256 byte values along N:
    # C = B logically, so every nibble of both halves of a byte is decoded
    K, N = 512, 512
    Bkn = (np.arange(K * (N // 2)) % 256).astype(np.uint8).reshape(K, N // 2)
    lo, hi = (Bkn & 0xF).astype(np.int64), (Bkn >> 4).astype(np.int64)
    want = np.empty((K, N), np.int64)
    want[:, 0::2] = np.where(lo >= 8, lo - 16, lo)
    want[:, 1::2] = np.where(hi >= 8, hi - 16, hi)
    C = _gpu_gemm_bt("s4", si.pack_s4(np.eye(K, dtype=np.int8)), Bkn)
    assert np.array_equal(C.astype(np.int64), want)


def test_transposed_b_argument_errors():
    A, B = si.gen_operands("f16", 256, 256, 64, seed=1)
    Ad, Bd = dev(A), dev(np.ascontiguousarray(B.T))
    for bad in [lambda: mp.gemm_bt("f16", Ad[:, :32].contiguous(), Bd[:32].contiguous()),  # K off the slice
                lambda: mp.gemm_bt("f16", Ad, Bd[:, :200].contiguous())]:                    # N off the tile
        with pytest.raises(mp.HipError):
            bad()
    with pytest.raises(ValueError):
        mp.gemm_bt("bf16", Ad, Bd)
    a4 = torch.zeros((256, 64), dtype=torch.uint8, device="cuda")    # INT4 K = 128: off the 256-k slice
    b4 = torch.zeros((128, 128), dtype=torch.uint8, device="cuda")
    with pytest.raises(mp.HipError):
        mp.gemm_bt("s4", a4, b4)
    L = mp.lib()
    assert L.mpgemm_gemm_bt(3, 256, 256, 64, Ad.data_ptr(), Bd.data_ptr(), Ad.data_ptr(), None) != 0
    assert L.mpgemm_gemm_bt(2, 256, 256, 256, Ad.data_ptr(), Bd.data_ptr(), Ad.data_ptr(), None) != 0  # C on A
    assert L.mpgemm_gemm_bt(0, 256, 256, 64, Ad.data_ptr() + 2, Bd.data_ptr(), None, None) != 0
    # K = 0: zero fill
    C = torch.full((4, 256), 7.0, dtype=torch.float32, device="cuda")
    assert L.mpgemm_gemm_bt(0, 4, 256, 0, Ad.data_ptr(), Bd.data_ptr(), C.data_ptr(), None) == 0
    torch.cuda.synchronize()
    assert torch.count_nonzero(C).item() == 0
