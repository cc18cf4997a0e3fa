"""Pins for the CPU oracle, independent of the oracle itself.

Each check rests on something other than the oracle's own code: the binary16
and two's-complement definitions, closed forms (all-ones, extremes, identity,
permutation, zeros), exact brute force in Python integers / fractions on tiny
shapes, and numpy's matmul on medium shapes. ``test_pins_catch_mutants`` builds
deliberately broken copies of oracle.c (a dropped term, a wrong sign, a
transposed operand, a swapped nibble order, an off-by-one exponent bias, a
wrong row index) and requires every one of them to fail at least one pin.
"""
import subprocess
from fractions import Fraction

import numpy as np
import pytest

import oracle
import seeded_inputs as si
from oracle.build import CFLAGS, SRC

# ---------------------------------------------------------------- definitions


def nibble_value(n):
    """Two's-complement meaning of a 4-bit pattern n in [0, 16)."""
    return n - 16 if n >= 8 else n


def ones(dtype, M, N, K):
    if dtype == "f16":
        return np.ones((M, K), np.float16), np.ones((N, K), np.float16)
    if dtype == "s8":
        return np.ones((M, K), np.int8), np.ones((N, K), np.int8)
    return np.full((M, K // 2), 0x11, np.uint8), np.full((N, K // 2), 0x11, np.uint8)


def run(orc, dtype, A, B, rows=None, threads=None):
    if dtype == "f16":
        return orc.gemm_f16(A, B, rows=rows, threads=threads)[0]
    if dtype == "s8":
        return orc.gemm_s8(A, B, rows=rows, threads=threads)
    return orc.gemm_s4(A, B, rows=rows, threads=threads)


def to_storage(dtype, logical):
    """Logical integer-valued matrix (rows, K) -> the dtype's storage array."""
    logical = np.asarray(logical)
    if dtype == "f16":
        return logical.astype(np.float16)
    if dtype == "s8":
        return logical.astype(np.int8)
    return si.pack_s4(logical.astype(np.int8))


def random_logical(dtype, rows, K, seed):
    w = si.splitmix64(seed, 0, rows * K)
    v = si.words_to_int4(w) if dtype == "s4" else si.words_to_int8(w)
    if dtype == "f16":
        v = si.words_to_int8(w) // 16  # small integers, exact in binary16
    return v.reshape(rows, K).astype(np.int64)


# ----------------------------------------------------------------- the pins
# Each pin takes an Oracle so the mutation test can run it on broken builds.


def pin_s4_decode(orc):
    dec = orc.s4_decode_bytes(np.arange(256))
    for b in range(256):
        assert tuple(dec[b]) == (nibble_value(b & 0xF), nibble_value(b >> 4)), hex(b)
    assert tuple(dec[0x08]) == (-8, 0)
    assert tuple(dec[0xF7]) == (7, -1)
    assert tuple(dec[0x80]) == (0, -8)


def pin_half_decode(orc):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = orc.half_to_double(bits)
    want = bits.view(np.float16).astype(np.float64)  # numpy's binary16 conversion
    finite = np.isfinite(want)
    assert np.array_equal(got[finite], want[finite])
    assert np.all(np.isnan(got[np.isnan(want)]))
    inf = np.isinf(want)
    assert np.array_equal(got[inf], want[inf])
    # a few values from the binary16 definition itself
    assert orc.half_to_double([0x3C00])[0] == 1.0
    assert orc.half_to_double([0x0001])[0] == 2.0 ** -24
    assert orc.half_to_double([0x7BFF])[0] == 65504.0
    assert orc.half_to_double([0xC000])[0] == -2.0


def pin_all_ones(orc):
    for dtype in ("f16", "s8", "s4"):
        for (M, N, K) in [(5, 7, 8), (3, 2, 30)]:
            A, B = ones(dtype, M, N, K)
            C = run(orc, dtype, A, B)
            assert C.shape == (M, N) and np.all(C == K), dtype


def pin_extremes(orc):
    K = 64
    A = np.full((3, K), -128, np.int8)
    assert np.all(orc.gemm_s8(A, np.full((2, K), -128, np.int8)) == 16384 * K)
    assert np.all(orc.gemm_s8(A, np.full((2, K), 127, np.int8)) == -16256 * K)
    A4 = np.full((3, K // 2), 0x88, np.uint8)  # every value -8
    assert np.all(orc.gemm_s4(A4, np.full((2, K // 2), 0x88, np.uint8)) == 64 * K)
    B4 = np.full((2, K // 2), 0x77, np.uint8)  # every value 7
    assert np.all(orc.gemm_s4(A4, B4) == -56 * K)
    # mixed signs inside a byte: (-8, 7) . (7, -8) = -112 per byte
    assert np.all(orc.gemm_s4(np.full((1, K // 2), 0x78, np.uint8),
                              np.full((1, K // 2), 0x87, np.uint8)) == -112 * (K // 2))
    Ah = np.full((2, K), -65504.0, np.float16)
    C, D = orc.gemm_f16(Ah, np.full((2, K), 2.0 ** -24, np.float16))
    assert np.all(C == -65504.0 * 2.0 ** -24 * K) and np.all(D == -C)


def pin_zeros(orc):
    for dtype in ("f16", "s8", "s4"):
        K = 16
        kw = K // 2 if dtype == "s4" else K
        z = np.zeros((4, kw), np.uint8 if dtype == "s4" else (np.float16 if dtype == "f16" else np.int8))
        A, _ = si.gen_operands(dtype, 4, 4, K, seed=1)
        assert np.all(run(orc, dtype, A, z) == 0)
        assert np.all(run(orc, dtype, z, A) == 0)


def pin_identity(orc):
    for dtype in ("f16", "s8", "s4"):
        K, N, M = 32, 12, 10
        I = np.eye(K, dtype=np.int64)
        Bl = random_logical(dtype, N, K, seed=11)  # B stored (N, K): B(k, j) = Bl[j, k]
        C = run(orc, dtype, to_storage(dtype, I), to_storage(dtype, Bl))
        assert np.array_equal(C, Bl.T), dtype  # I_K * B = B as a K x N matrix
        Al = random_logical(dtype, M, K, seed=12)
        C = run(orc, dtype, to_storage(dtype, Al), to_storage(dtype, I))
        assert np.array_equal(C, Al), dtype  # A * I_K = A


def pin_permutation(orc):
    rng = np.random.default_rng(5)
    for dtype in ("f16", "s8", "s4"):
        K, N = 24, 9
        perm = rng.permutation(K)
        P = np.zeros((K, K), np.int64)
        P[np.arange(K), perm] = 1  # row i of P selects k = perm[i]
        Bl = random_logical(dtype, N, K, seed=13)
        C = run(orc, dtype, to_storage(dtype, P), to_storage(dtype, Bl))
        assert np.array_equal(C, Bl.T[perm]), dtype


def brute(dtype, A, B):
    """Exact C from the definition in Python integers / fractions."""
    if dtype == "f16":
        Af = [[Fraction(float(x)) for x in row] for row in A]
        Bf = [[Fraction(float(x)) for x in row] for row in B]
    elif dtype == "s8":
        Af = [[int(x) for x in row] for row in A]
        Bf = [[int(x) for x in row] for row in B]
    else:
        def dec(row):
            out = []
            for byte in row:
                out += [nibble_value(int(byte) & 0xF), nibble_value(int(byte) >> 4)]
            return out
        Af = [dec(row) for row in A]
        Bf = [dec(row) for row in B]
    return [[sum(a * b for a, b in zip(ar, bc)) for bc in Bf] for ar in Af]


BRUTE_SHAPES = [(4, 4, 8), (1, 1, 2), (3, 5, 8), (7, 3, 6), (16, 16, 32)]


def pin_brute_force(orc):
    for dtype in ("f16", "s8", "s4"):
        for i, (M, N, K) in enumerate(BRUTE_SHAPES):
            A, B = si.gen_operands(dtype, M, N, K, seed=100 + i)
            want = brute(dtype, A, B)
            if dtype == "f16":
                C, D = orc.gemm_f16(A, B)
                for r in range(M):
                    for c in range(N):
                        err = abs(Fraction(C[r, c]) - want[r][c])
                        assert err <= Fraction(1, 10**15) * Fraction(D[r, c]) + Fraction(1, 10**300)
            else:
                C = run(orc, dtype, A, B)
                assert C.tolist() == want, (dtype, M, N, K)


def pin_numpy(orc):
    shapes = [(96, 80, 200), (64, 48, 130)]
    for (M, N, K) in shapes:
        A, B = si.gen_operands("s8", M, N, K, seed=21)
        assert np.array_equal(orc.gemm_s8(A, B), A.astype(np.int64) @ B.astype(np.int64).T)
        A, B = si.gen_operands("s4", M, N, K, seed=22)
        Au = np.array(brute_unpack(A)), np.array(brute_unpack(B))
        assert np.array_equal(orc.gemm_s4(A, B), Au[0] @ Au[1].T)
        A, B = si.gen_operands("f16", M, N, K, seed=23)
        C, D = orc.gemm_f16(A, B)
        ref = A.astype(np.float64) @ B.astype(np.float64).T
        Dref = np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64)).T
        assert np.max(np.abs(C - ref) / Dref) <= 1e-12
        assert np.max(np.abs(D - Dref) / Dref) <= 1e-12


def brute_unpack(P):
    out = np.empty((P.shape[0], 2 * P.shape[1]), np.int64)
    lo = (P & 0xF).astype(np.int64)
    hi = (P >> 4).astype(np.int64)
    out[:, 0::2] = np.where(lo >= 8, lo - 16, lo)
    out[:, 1::2] = np.where(hi >= 8, hi - 16, hi)
    return out


def pin_rows_and_threads(orc):
    for dtype in ("f16", "s8", "s4"):
        A, B = si.gen_operands(dtype, 37, 19, 40, seed=31)
        full = run(orc, dtype, A, B, threads=1)
        assert np.array_equal(full, run(orc, dtype, A, B, threads=7))
        rows = [36, 0, 5, 5, 17]
        assert np.array_equal(run(orc, dtype, A, B, rows=rows, threads=3), full[rows])


PINS = [pin_s4_decode, pin_half_decode, pin_all_ones, pin_extremes, pin_zeros,
        pin_identity, pin_permutation, pin_brute_force, pin_numpy, pin_rows_and_threads]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(oracle.get())


# ------------------------------------------------------------ error handling


def test_rejects_nonfinite_fp16():
    A = np.ones((2, 4), np.float16)
    A[1, 2] = np.inf
    with pytest.raises(ValueError):
        oracle.gemm_f16(A, np.ones((3, 4), np.float16))


def test_rejects_bad_rows_and_shapes():
    A, B = si.gen_operands("s8", 4, 4, 8, seed=1)
    with pytest.raises(ValueError):
        oracle.gemm_s8(A, B, rows=[4])
    with pytest.raises(ValueError):
        oracle.gemm_s8(A, B[:, :6])


def test_empty_shapes():
    C = oracle.gemm_s8(np.zeros((0, 8), np.int8), np.zeros((3, 8), np.int8))
    assert C.shape == (0, 3)
    C = oracle.gemm_s8(np.zeros((2, 0), np.int8), np.zeros((3, 0), np.int8))
    assert C.shape == (2, 3) and np.all(C == 0)  # K = 0: empty sums


# ---------------------------------------------------------------- mutants

MUTANTS = {
    # dropped term: the loop skips the last k
    "dropped_term": ("for (long k = 0; k < K; ++k)\n                    acc += (int64_t)arow[k]",
                     "for (long k = 0; k < K - 1; ++k)\n                    acc += (int64_t)arow[k]"),
    # wrong sign in the FP16 accumulation
    "wrong_sign": ("acc += ad[k] * bcol[k];", "acc -= ad[k] * bcol[k];"),
    # transposed B: reads B(j,k) as if B were row-major
    "transposed_b": ("acc += (int64_t)arow[k] * (int64_t)bcol[k];",
                     "acc += (int64_t)arow[k] * (int64_t)((const int8_t *)jb->B)[k * N + j];"),
    # nibble order swapped (high nibble for even k)
    "nibble_order": ("(k % 2 == 0) ? (byte & 0x0Fu) : (byte >> 4)",
                     "(k % 2 == 1) ? (byte & 0x0Fu) : (byte >> 4)"),
    # unsigned nibbles
    "unsigned_nibble": ("return nib >= 8 ? (int)nib - 16 : (int)nib;", "return (int)nib;"),
    # exponent bias off by one
    "bias": ("ldexp((double)(1024 + f), e - 25)", "ldexp((double)(1024 + f), e - 24)"),
    # subnormal scale wrong
    "subnormal": ("ldexp((double)f, -24)", "ldexp((double)f, -25)"),
    # row subset ignored (computes row r instead of rows[r])
    "row_index": ("long i = jb->rows ? (long)jb->rows[r] : r;", "long i = r;"),
    # B column index off by one for the nibble decode of B
    "s4_b_offset": ("d->src4 + j * (d->K / 2), k)", "d->src4 + j * (d->K / 2), k + (k < d->K - 1))"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutants(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutant {name} no longer applies to oracle.c"
    mutated = src.replace(old, new)
    path = tmp_path / "mut.c"
    path.write_text(mutated)
    lib = tmp_path / "libmut.so"
    flags = [f for f in CFLAGS if not f.startswith("-W")]
    subprocess.run(["gcc", *flags, str(path), "-o", str(lib), "-lm"], check=True)
    orc = oracle.Oracle(str(lib))
    failed = []
    for pin in PINS:
        try:
            pin(orc)
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"


# ---------------------------------------------------------------- scaled outputs


def _rne_exact(x, frac_bits, emin):
    """x rounded to frac_bits stored fraction bits (ties to even), exponent
    floor emin (fixed spacing below the smallest normal), in exact rationals."""
    from fractions import Fraction
    if x == 0:
        return 0.0
    f = abs(Fraction(x))
    e = 0
    while f >= 2:
        f /= 2
        e += 1
    while f < 1:
        f *= 2
        e -= 1
    scale = Fraction(2) ** (max(e, emin) - frac_bits)
    q = Fraction(x) / scale
    n = q.numerator // q.denominator
    r = q - n
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return float(n * scale)


def test_round_bf16_matches_exact_rounding():
    rng = np.random.default_rng(21)
    xs = rng.standard_normal(3000) * 10.0 ** rng.integers(-42, 38, 3000)
    ties = [1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 5 * 2 ** -8), 2 ** -130 * 1.5, 2 ** -134, 2 ** -133 * 3]
    xs = np.concatenate([xs, ties])
    want = np.array([_rne_exact(float(x), 7, -126) for x in xs])
    assert np.array_equal(oracle.round_bf16(xs), want)
    assert oracle.round_bf16(np.array([3.5e38]))[0] == np.inf
    assert oracle.round_out(np.array([1 + 2 ** -11, 1 + 3 * 2 ** -11]), "f16").tolist() == [1.0, 1 + 2 ** -9]


def test_scaled_oracle_pins():
    """Unit scales and no zero points: the plain exact sum, rounded once. Zero
    points: brute force over Python integers. Power-of-two scales: exact."""
    for dt in ("s8", "s4"):
        M, N, K = 3, 5, 8
        A, B = si.gen_operands(dt, M, N, K, seed=17)
        C = (oracle.gemm_s8(A, B) if dt == "s8" else oracle.gemm_s4(A, B)).astype(np.float64)
        got, exact, D = oracle.gemm_scaled(dt, A, B, "f32")
        assert D is None and np.array_equal(exact, C) and np.array_equal(got, C.astype(np.float32))
        za = np.array([3, -2, 0], np.int32)
        zb = np.array([1, 0, -4, 7, -1], np.int32)
        a = oracle.s4_unpack(A) if dt == "s4" else A.astype(np.int64)
        b = oracle.s4_unpack(B) if dt == "s4" else B.astype(np.int64)
        brute = np.array([[sum((int(a[i, k]) - int(za[i])) * (int(b[j, k]) - int(zb[j])) for k in range(K))
                           for j in range(N)] for i in range(M)], dtype=np.float64)
        sa = np.array([0.5, 2.0, 0.25], np.float32)
        sb = np.array([1.0, 4.0, 0.125, 2.0, 8.0], np.float32)
        got, exact, _ = oracle.gemm_scaled(dt, A, B, "f32", sa, sb, za, zb)
        assert np.array_equal(exact, brute * sa[:, None] * sb[None, :])
    A, B = si.gen_operands("f16", 4, 3, 16, seed=3)
    C, D = oracle.gemm_f16(A, B)
    sa = np.array([2.0, 0.5, 1.0, 4.0], np.float32)
    got, exact, Ds = oracle.gemm_scaled("f16", A, B, "bf16", sa, None)
    assert np.array_equal(exact, C * sa[:, None]) and np.array_equal(Ds, D * sa[:, None])
    assert np.array_equal(got, oracle.round_bf16(C * sa[:, None]))
