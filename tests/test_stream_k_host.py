"""Host-side checks of the stream-K schedule (no GPU): the plan the library
reports (mpgemm_sk_schedule) computes every (tile, K-slice) iteration
exactly once: whole tiles first, then the remaining tiles cut into K-parts
as the kernels cut them (sk_work), one workgroup and one partial slot each.
Without a visible device the library plans for 256 resident workgroups (one
per MI355X CU)."""
import ctypes
import math
import re

import pytest

import paper_2608_10103_amd as mp

G = 256
SK_NAMES = ("wide256x256_w2x2_k128_m16_sk", "pipe256x256_w2x4_k128_s2_sk", "spread128x128_w2x2_k128_s4_sk",
            "fp6wide256x256_w2x2_k128_s3_sk", "spread128x128_w2x4_k128_s4_sk", "spread128x128_w2x4_k64_s4_sk")
BYTES_PER_ELEM = {"f16": 2.0, "s8": 1.0, "s4": 0.5}


def _variant(dtype, name):
    return [v for v in range(mp.num_variants(dtype)) if mp.variant_name(dtype, v) == name][0]


def _tile(name):
    return tuple(int(x) for x in re.search(r"(\d+)x(\d+)_w", name).groups())


def _slices(dtype, name, K):
    """K-slices per tile: 128-byte slices of a row; the FP6 kernel's 128-k
    slices of K padded to 256 (its converted operands' padding)."""
    if name.startswith("fp6"):
        return -(-K // 256) * 2
    return int(K * BYTES_PER_ELEM[dtype]) // (64 if "_k64_" in name else 128)


def _f6_bytes(M, N, K):
    """The FP6 operand copies the INT4 pre-pass writes (24 bytes per row and
    run of 32 k, rows padded to 256, K to 256), 256-byte aligned."""
    runs = -(-K // 256) * 8
    b = (-(-M // 256) * 256 + -(-N // 256) * 256) * runs * 24
    return -(-b // 256) * 256


def _work(b, dp, parts, KT):
    """(tile, first slice, slices, slot) of workgroup b; the whole-tile
    workgroups' tiles are a permutation of 0 .. dp - 1 (XCD-contiguous), so
    only their count matters here."""
    if b < dp:
        return None
    u = b - dp
    j = u % parts
    k0, k1 = j * KT // parts, (j + 1) * KT // parts
    return dp + u // parts, k0, k1 - k0, u


CASES = [  # dtype, name, M, N, K
    ("f16", SK_NAMES[0], 4352, 4096, 4096),      # 272 tiles: 256 whole, 16 split, 64 slices: 4 parts
    ("f16", SK_NAMES[0], 4352, 4096, 8192),      # 128 slices: 5 parts
    ("s8", SK_NAMES[0], 4352, 4096, 8192),       # 64 slices
    ("s8", SK_NAMES[0], 4352, 4096, 4096),       # 32 slices: no gain expected, off
    ("s8", SK_NAMES[0], 6144, 6400, 16384),      # 600 = 2 x 256 + 88: at most 2 parts
    ("s8", SK_NAMES[0], 256 * 3, 256 * 86, 65536),  # 258 tiles, 512 slices: capped at 8
    ("f16", SK_NAMES[0], 2048, 2048, 8192),      # 64 tiles, fewer than the CUs
    ("f16", SK_NAMES[1], 4000, 4400, 6400),      # ragged, 288 tiles, 100 slices
    ("s4", SK_NAMES[1], 4000, 4400, 25600),
    ("s8", SK_NAMES[2], 2100, 2000, 8192),       # 272 tiles of 128 x 128
    ("s4", SK_NAMES[2], 128 * 23 + 5, 128 * 12, 32768),
    ("f16", SK_NAMES[2], 128 * 16 + 1, 128 * 16, 128 * 3),  # 3 slices: off
    ("s4", SK_NAMES[3], 4352, 4096, 16384),      # INT4 on the FP6 cores: 128 slices of 128 k
    ("s4", SK_NAMES[3], 4000, 4400, 12800),      # ragged: 288 tiles, 100 slices: off
    ("s4", SK_NAMES[3], 4000, 4400, 32768),      # 256 slices: on
    ("s4", SK_NAMES[3], 4352, 4096, 30000),      # K padded to 30208: 236 slices
    ("s4", SK_NAMES[3], 4352, 4096, 8192),       # 64 slices: off
    ("s4", SK_NAMES[3], 256 * 3, 256 * 86, 81920),  # 258 tiles, 640 slices: 8 parts
    ("s4", SK_NAMES[3], 33, 65, 1 << 18),        # one tile
    ("s8", SK_NAMES[4], 2100, 2000, 8192),       # eight-wave 128 x 128 kernel
    ("f16", SK_NAMES[4], 2100, 2000, 3200),
    ("s4", SK_NAMES[5], 2100, 2000, 12800),      # 64-byte slices: 100 slices of half the time
    ("s4", SK_NAMES[5], 128 * 23 + 5, 128 * 12, 32768),
]


@pytest.mark.parametrize("dtype,name,M,N,K", CASES)
def test_sk_schedule_covers_every_iteration_once(dtype, name, M, N, K):
    v = _variant(dtype, name)
    bm, bn = _tile(name)
    tiles = -(-M // bm) * -(-N // bn)
    KT = _slices(dtype, name, K)
    dp, parts, grid = mp.sk_schedule(dtype, v, M, N, K)
    q, r = divmod(tiles, G)
    # the library's cost model (slice time t, margin m: 1 and 0.1, 0.5 for
    # 64-byte slices, for the FP6 kernel 0.5 and 0.25): s = round(sqrt(KT t
    # / 5)) capped at G / r, 8 and KT / 2, taken when KT t (1 - 1/s) -
    # 5 (s - 1) - 13 exceeds m KT t
    t, m = (0.5, 0.25) if name.startswith("fp6") else ((0.5 if "_k64_" in name else 1.0), 0.1)
    small_tile_first_round = tiles < G and bm * bn < 256 * 256  # 128 x 128 tiles need a whole round first
    want_parts = (min(int(math.sqrt(KT * t / 5) + 0.5), G // r, 8, KT // 2)
                  if r and 2 * r <= G and not small_tile_first_round else 1)
    gain = KT * t * (1 - 1 / want_parts) - 5 * (want_parts - 1) - 13 if want_parts >= 2 else 0
    if want_parts < 2 or gain <= m * KT * t:
        assert (dp, parts, grid) == (tiles, 1, tiles)
        return
    assert (dp, parts, grid) == (q * G, want_parts, q * G + r * want_parts)
    assert grid - dp <= G, "the split remainder fits one round"
    covered = {t: [] for t in range(dp, tiles)}
    slots = set()
    for b in range(grid):
        w = _work(b, dp, parts, KT)
        if w is None:
            continue
        t, k0, n, u = w
        assert n >= KT // parts and u not in slots
        slots.add(u)
        covered[t].append((k0, n))
    for t, ps in covered.items():
        assert len(ps) == parts
        assert sorted(ps)[0][0] == 0
        assert all(a[0] + a[1] == b[0] for a, b in zip(sorted(ps), sorted(ps)[1:])), f"tile {t} parts not contiguous"
        assert sum(n for _, n in ps) == KT
    assert slots == set(range(grid - dp))
    # counters, then (FP6 kernel) the converted operands, then one partial slot per remainder part
    f6 = _f6_bytes(M, N, K) if name.startswith("fp6") else 0
    assert mp.workspace_size(dtype, M, N, K, variant=v, splits=1) == 65536 + f6 + (grid - dp) * bm * bn * 4


@pytest.mark.parametrize("dtype,name,M,N,K", [
    ("f16", SK_NAMES[0], 4096, 4096, 512),        # 256 tiles: one full round
    ("s8", SK_NAMES[0], 8192, 8192, 1024),        # 1024 tiles: whole rounds
    ("f16", SK_NAMES[1], 4000, 8000, 512),        # 16 x 32 = 512 tiles
    ("s8", SK_NAMES[0], 256 * 20, 256 * 20, 1024),  # 400 = 256 + 144: last round over half full
    ("s4", SK_NAMES[2], 2048, 2048, 512),         # 256 tiles
    ("s8", "pipe256x256_w2x4_k128_s2", 4352, 4096, 1024),  # not a stream-K variant
    ("s4", SK_NAMES[3], 8192, 8192, 8192),        # 1024 tiles: whole rounds
])
def test_sk_schedule_off(dtype, name, M, N, K):
    """Whole rounds, a last round over half full, or a variant without the
    schedule: every tile whole, one workgroup each, and no workspace."""
    v = _variant(dtype, name)
    bm, bn = _tile(name)
    tiles = -(-M // bm) * -(-N // bn)
    assert mp.sk_schedule(dtype, v, M, N, K) == (tiles, 1, tiles)
    # no scratch but the FP6 kernel's converted operands
    f6 = 65536 + _f6_bytes(M, N, K) if name.startswith("fp6") else 0
    assert mp.workspace_size(dtype, M, N, K, variant=v, splits=1) == f6


def test_sk_schedule_errors():
    L = mp.lib()
    x = ctypes.c_int()
    p = ctypes.byref(x)
    v = _variant("f16", SK_NAMES[0])
    assert L.mpgemm_sk_schedule(0, v, 4352, 4096, 512, None, p, p) == 1
    assert L.mpgemm_sk_schedule(0, -1, 4352, 4096, 512, p, p, p) == 1
    assert L.mpgemm_sk_schedule(7, v, 4352, 4096, 512, p, p, p) == 1
    # the one-wave-per-SIMD kernel needs 128-byte K-slices; it has no INT4 kernel
    assert L.mpgemm_sk_schedule(0, v, 4353, 4096, 520, p, p, p) == 1
    assert L.mpgemm_sk_schedule(0, v, 4353, 4096, 512, p, p, p) == 0
    assert L.mpgemm_sk_schedule(2, _variant("s4", SK_NAMES[0]), 4352, 4096, 512, p, p, p) == 1
    # the FP6 kernel: INT4 only, even K
    f6 = _variant("s4", SK_NAMES[3])
    assert L.mpgemm_sk_schedule(0, f6, 4352, 4096, 512, p, p, p) == 1
    assert L.mpgemm_sk_schedule(2, f6, 4352, 4096, 511, p, p, p) == 1
    assert L.mpgemm_sk_schedule(2, f6, 4352, 4096, 512, p, p, p) == 0


def test_sk_selection_with_a_workspace():
    """With a workspace the automatic choice takes the stream-K twin of the
    kernel it would pick where that twin's schedule is on; without one, or
    where the schedule is off, the whole-tile kernel."""
    name = lambda d, M, N, K, ws: mp.variant_name(d, mp.select_variant(d, M, N, K, with_ws=ws))
    for d, M, N, K, plain, twin in [
        ("f16", 4352, 4096, 8192, "wide256x256_w2x2_k128_m16", "wide256x256_w2x2_k128_m16_sk"),
        ("s8", 4352, 4096, 16384, "wide256x256_w2x2_k128_m16", "wide256x256_w2x2_k128_m16_sk"),
        # ragged, 288 tiles (rounds 56% filled): without a workspace the
        # 128 x 128 kernel, with one the stream-K schedule of the 256 x 256 one
        ("f16", 4000, 4400, 6400, "spread128x128_w2x4_k128_s4", "wide256x256_w2x2_k128_m16_sk"),
        ("s8", 2100, 2000, 6400, "spread128x128_w2x4_k128_s4", "spread128x128_w2x4_k128_s4_sk"),
        ("s4", 2100, 2000, 12800, "spread128x128_w2x4_k64_s4", "spread128x128_w2x4_k64_s4_sk"),
        ("f16", 2100, 2000, 6400, "spread128x128_w2x4_k128_s4", "spread128x128_w2x4_k128_s4_sk"),
    ]:
        assert name(d, M, N, K, False) == plain, (d, M, N, K)
        assert name(d, M, N, K, True) == twin, (d, M, N, K)
    # schedule off: too few slices, whole rounds, last round over half full
    for d, M, N, K in [("s8", 4352, 4096, 4096), ("f16", 8192, 8192, 8192), ("f16", 5120, 5120, 8192)]:
        assert not name(d, M, N, K, True).endswith("_sk"), (d, M, N, K)
    # FP16, 96..143 tiles of 256 x 256 and at least 128 K-slices: the
    # one-wave-per-SIMD kernel's stream-K schedule in place of 128 x 128
    for M, N, K in [(768, 8192, 8192), (1024, 8192, 8192), (2560, 2560, 8192)]:
        assert name("f16", M, N, K, False) == "spread128x128_w2x4_k128_s4"
        assert name("f16", M, N, K, True) == "wide256x256_w2x2_k128_m16_sk", (M, N, K)
    for d, M, N, K in [("f16", 1024, 4096, 8192), ("f16", 1024, 8192, 4096), ("s8", 768, 8192, 8192)]:
        assert not name(d, M, N, K, True).startswith("wide"), (d, M, N, K)  # 64 tiles, 64 slices, INT8
    # INT4 with a workspace: the FP6 pre-pass kernel, stream-K where its plan is on
    assert name("s4", 4352, 4096, 16384, True) == "fp6wide256x256_w2x2_k128_s3_sk"
    assert name("s4", 8192, 8192, 8192, True) == "fp6wide256x256_w2x2_k128_s3"
    # without one, 272 tiles (a partial second round): the 128 x 128 kernel
    # (4352 x 4096 x 8192: 170.8 against 214.4 us for the in-GEMM E2M3 one)
    assert name("s4", 4352, 4096, 16384, False) == "spread128x128_w2x4_k64_s4"
