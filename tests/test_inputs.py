"""Seeded input generators: the random stream, the value maps and INT4 packing."""
import numpy as np
import pytest

import seeded_inputs as si


def test_splitmix64_published_vector():
    # Vigna's reference splitmix64.c started from state 0 yields these words.
    want = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    assert [si.splitmix64_scalar(0, c) for c in range(3)] == want
    assert [int(x) for x in si.splitmix64(0, 0, 3)] == want


@pytest.mark.parametrize("seed", [0, 1, 3, 12345, 2**64 - 1])
def test_vectorised_stream_matches_scalar(seed):
    starts = [0, 7, 1000, (1 << 22) - 3]  # last one straddles a chunk boundary
    for st in starts:
        v = si.splitmix64(seed, st, 8)
        assert [int(x) for x in v] == [si.splitmix64_scalar(seed, st + c) for c in range(8)]


def test_stream_slices_are_consistent():
    whole = si.splitmix64(5, 0, 5000)
    assert np.array_equal(whole[1234:2345], si.splitmix64(5, 1234, 1111))


def test_int8_and_int4_maps_use_top_bits():
    w = np.array([0, 1 << 63, (1 << 64) - 1, 0x7F << 56, 0x80 << 56, 0x8 << 60, 0x7 << 60],
                 dtype=np.uint64)
    assert list(si.words_to_int8(w)) == [0, -128, -1, 127, -128, -128, 112]
    assert list(si.words_to_int4(w)) == [0, -8, -1, 7, -8, -8, 7]


def test_distributions_cover_their_ranges():
    w = si.splitmix64(1, 0, 1 << 16)
    i8 = si.words_to_int8(w)
    assert i8.min() == -128 and i8.max() == 127
    counts = np.bincount(i8.astype(np.int64) + 128, minlength=256)
    assert counts.min() > 150  # 256 expected per value
    i4 = si.words_to_int4(w)
    assert set(np.unique(i4)) == set(range(-8, 8))
    u = si.words_to_uniform_pm1_f16(w).astype(np.float64)
    assert u.min() >= -1.0 and u.max() <= 1.0 and abs(u.mean()) < 0.02
    n = si.normal_f16(3, 0, 1 << 16).astype(np.float64)
    assert abs(n.mean()) < 0.02 and abs(n.std() - 1.0) < 0.02


def test_pack_layout_low_nibble_is_even_k():
    v = np.array([[1, -2, -8, 7]], dtype=np.int8)
    p = si.pack_s4(v)
    assert p.dtype == np.uint8 and p.shape == (1, 2)
    assert int(p[0, 0]) == (1 | (0xE << 4)) and int(p[0, 1]) == (0x8 | (0x7 << 4))


def test_pack_rejects_bad_input():
    with pytest.raises(ValueError):
        si.pack_s4(np.zeros((2, 3), np.int8))
    with pytest.raises(ValueError):
        si.pack_s4(np.array([[8, 0]], np.int8))


@pytest.mark.parametrize("dtype", ["f16", "s8", "s4"])
def test_gen_operands_shapes_and_determinism(dtype):
    M, N, K = 24, 40, 64
    A, B = si.gen_operands(dtype, M, N, K, seed=7)
    A2, B2 = si.gen_operands(dtype, M, N, K, seed=7)
    assert np.array_equal(A, A2) and np.array_equal(B, B2)
    kw = K // 2 if dtype == "s4" else K
    assert A.shape == (M, kw) and B.shape == (N, kw)
    A3, _ = si.gen_operands(dtype, M, N, K, seed=8)
    assert not np.array_equal(A, A3)


def test_b_continues_the_stream_after_a():
    M, N, K = 3, 5, 8
    A, B = si.gen_operands("s8", M, N, K, seed=9)
    w = si.splitmix64(9, 0, M * K + N * K)
    assert np.array_equal(A.ravel(), si.words_to_int8(w[:M * K]))
    assert np.array_equal(B.ravel(), si.words_to_int8(w[M * K:]))


def test_normal_f16_operands():
    A, B = si.gen_operands("f16", 16, 8, 33, seed=3, dist="normal")
    assert A.dtype == np.float16 and np.all(np.isfinite(A)) and np.all(np.isfinite(B))


def test_sample_rows():
    r = si.sample_rows(1003, 8192, 256, force=(0, 8191))
    assert r.dtype == np.int32
    assert 256 <= r.size <= 258 and r[0] == 0 and r[-1] == 8191
    assert len(set(r.tolist())) == r.size and np.all(np.diff(r) > 0)
    assert np.array_equal(r, si.sample_rows(1003, 8192, 256, force=(0, 8191)))


def test_sweep_seeds():
    pts = si.sweep_points()
    assert len(pts) == 15
    assert pts[0] == ("f16", 512, 10) and pts[4] == ("f16", 8192, 14)
    assert pts[5] == ("s8", 512, 15) and pts[14] == ("s4", 8192, 24)
