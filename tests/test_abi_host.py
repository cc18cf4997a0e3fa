"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/mpgemm.h declares, and its argument checks and kernel
choice behave as documented (these entry points never touch the device)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2608_10103_amd as mp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mpgemm.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert {"gemm_f16_f32", "gemm_s8_s32", "gemm_s4_s32"} <= set(names)
    lib = ctypes.CDLL(mp.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in mpgemm.h but not exported"
    assert set(names) == set(mp.EXPORTED_SYMBOLS)


def test_variant_table():
    for dt in ("f16", "s8", "s4"):
        n = mp.num_variants(dt)
        assert n >= 2
        assert mp.variant_name(dt, 0).startswith("generic")
        prefixes = ("tile", "pipe", "spread", "staged", "pingpong", "deep", "skinny", "wide") + \
            (("fp6pipe", "fp6wide", "e2m3wide") if dt == "s4" else ())
        assert all(mp.variant_name(dt, v).startswith(prefixes) for v in range(1, n))
        assert mp.variant_name(dt, n) == ""
    assert mp.lib().mpgemm_num_variants(7) == -1


@pytest.mark.parametrize("dt", ["f16", "s8", "s4"])
@pytest.mark.parametrize("n", [512, 1024, 2048, 4096, 8192])
def test_sweep_sizes_take_tiled_kernels(dt, n):
    v = mp.select_variant(dt, n, n, n)
    assert v > 0, f"{dt} {n} falls back to the bounds-checked kernel"


def test_selection_falls_back_when_needed():
    assert mp.select_variant("s8", 1000, 1024, 1024) > 0   # ragged M: predicated edge tiles
    assert mp.select_variant("s8", 1024, 777, 1024) > 0    # ragged N
    assert mp.select_variant("s8", 1024, 1024, 1000) == 0  # K off the K-slice
    assert mp.select_variant("s8", 1024, 1024, 1024, a_ptr=(1 << 20) + 4) == 0  # unaligned A
    assert mp.select_variant("s4", 256, 256, 262144) == 0  # scaled INT4 range exceeded
    assert mp.select_variant("s4", 256, 256, 0) == 0       # K = 0: zero fill


def test_invalid_arguments_rejected_on_host():
    L = mp.lib()
    sel = lambda dt, M, N, K, a=1 << 20, b=1 << 40, c=1 << 44: L.mpgemm_select_variant(dt, M, N, K, a, b, c)
    assert sel(1, -1, 8, 8) == -1
    assert sel(2, 8, 8, 7) == -1                 # odd K for INT4
    assert sel(1, 8, 8, 8, a=0) == -1            # NULL A
    assert sel(1, 8, 8, 8, c=0) == -1            # NULL C
    assert sel(1, 8, 8, 8, c=(1 << 44) + 2) == -1  # C not 4-byte aligned
    assert sel(0, 8, 8, 8, a=(1 << 20) + 1) == -1  # FP16 A not 2-byte aligned
    assert sel(1, 8, 8, 8, c=(1 << 20) + 16) == -1  # C overlaps A
    assert sel(5, 8, 8, 8) == -1                 # unknown dtype
    assert sel(1, 0, 8, 8, a=0, b=0, c=0) == 0   # empty: valid no-op
    assert L.mpgemm_variant_supports(9, 0, 8, 8, 8, 1 << 20, 1 << 40, 1 << 44) == -1
    assert L.mpgemm_run_variant(1, -1, 8, 8, 8, 1 << 20, 1 << 40, 1 << 44, None) != 0


def _swz(ch, q):
    # the LDS chunk swizzle of device_common.hpp (swz<CH>)
    if ch == 8:
        return (q ^ (q >> 3)) & 7
    return ((q >> 3) ^ (q >> 4)) & 3


# Swizzles of 64-byte rows, ((q >> a) ^ (q >> b)) & 3, that read at the rate
# of the conflict-free 128-byte layout (within 3%) under the MFMA operand-read
# pattern, measured on MI355X with an LDS micro-benchmark (eight 1 KiB
# ds_read_b128 per wave and iteration, 8 waves per CU). A 16-lane bank model does not predict them: it
# calls ((q >> 1) ^ (q >> 3)) & 3 conflict-free, which measured 1.75x slower.
MEASURED_FAST_64B = {(3, 7), (3, 4), (2, 5), (2, None), (3, 6), (3, 5), (2, 7), (2, 3), (2, 6),
                     (3, None), (1, 4), (0, 2), (1, 2), (0, 3)}


def test_lds_swizzle_128_byte_rows_is_conflict_free():
    """An MFMA operand fetch reads chunk c of 32 consecutive 128-byte LDS rows
    (16 bytes per lane): in 8-lane groups (128 bytes per cycle) and in 16-lane
    groups (256 bytes per cycle) every lane hits a different 16-byte bank
    group (SQ_LDS_BANK_CONFLICT reads 0 on the kernels that use it)."""
    ch = 8
    row_bytes = 16 * ch
    for base in range(0, 512, 32):
        for c in range(ch):
            addrs = [(base + r) * row_bytes + 16 * (c ^ _swz(ch, base + r)) for r in range(32)]
            for group, width in ((8, 128), (16, 256)):
                for g0 in range(0, 32, group):
                    slots = {(a % width) // 16 for a in addrs[g0:g0 + group]}
                    assert len(slots) == group, (ch, base, c, group)


def test_lds_swizzle_64_byte_rows_is_a_measured_fast_one():
    for q in range(512):
        assert _swz(4, q) == ((q >> 3) ^ (q >> 4)) & 3
    assert (3, 4) in MEASURED_FAST_64B


@pytest.mark.parametrize("ch", [8, 4])
def test_lds_swizzle_is_a_permutation(ch):
    # every row stores each of its chunks exactly once
    for q in range(512):
        assert sorted(c ^ _swz(ch, q) for c in range(ch)) == list(range(ch))


def test_selection_large_tile_threshold():
    """Whole 256 x 256 tiles from 144 tiles (56% of the 256 CUs) up for FP16,
    INT8 and INT4 with a workspace; INT4's in-GEMM conversion from 192; the
    eight-wave 128 x 128 kernels below (measured crossovers on MI355X)."""
    name = lambda d, M, N, K, ws=False: mp.variant_name(d, mp.select_variant(d, M, N, K, with_ws=ws))
    for n, tiles in [(2816, 121), (3072, 144), (3328, 169), (3584, 196), (3840, 225)]:
        big = tiles >= 144
        for d in ("f16", "s8"):
            assert name(d, n, n, n) == ("wide256x256_w2x2_k128_m16" if big else "spread128x128_w2x4_k128_s4"), (d, n)
        assert name("s4", n, n, n, True) == ("fp6wide256x256_w2x2_k128_s3" if big else "spread128x128_w2x4_k64_s4"), n
        assert name("s4", n, n, n) == ("e2m3wide256x256_w2x2_k256" if tiles >= 192 else "spread128x128_w2x4_k64_s4"), n
    # 128 tiles of 256 x 256: the 128 x 128 kernels
    assert name("f16", 4096, 2048, 4096) == "spread128x128_w2x4_k128_s4"


def test_selection_at_sweep_sizes():
    """The kernels the sweep runs (chosen from interleaved MI355X timings)."""
    want = {
        8192: ("wide256x256_w2x2_k128_m16",) * 2 + ("e2m3wide256x256_w2x2_k256",),
        4096: ("wide256x256_w2x2_k128_m16",) * 2 + ("e2m3wide256x256_w2x2_k256",),
        2048: ("spread128x128_w2x4_k128_s4",) * 2 + ("spread128x128_w2x4_k64_s4",),
        # 64 tiles of 128 x 128 would fill a quarter of the CUs: the narrow
        # tiles (FP16 64 x 128 8.0 against 10.3 us, INT8 64 x 64 7.1 against
        # 7.6, INT4 7.1 against 7.9)
        1024: ("spread64x128_w2x4_k128_s4",) + ("spread64x64_w2x2_k128_s4_m16",) * 2,
        512: ("spread64x128_w2x4_k128_s4",) + ("spread64x64_w2x2_k128_s4_m16",) * 2,  # launch bound, ~7 us
    }
    for n, names in want.items():
        got = tuple(mp.variant_name(d, mp.select_variant(d, n, n, n)) for d in ("f16", "s8", "s4"))
        assert got == names, (n, got)
    # with a workspace INT4 takes the FP6 kernel fed by the conversion pre-pass
    for n in (4096, 8192):
        assert mp.variant_name("s4", mp.select_variant("s4", n, n, n, with_ws=True)) == "fp6wide256x256_w2x2_k128_s3"
        for d in ("f16", "s8"):
            assert mp.select_variant(d, n, n, n, with_ws=True) == mp.select_variant(d, n, n, n)
    for n in (512, 1024, 2048):
        assert mp.select_variant("s4", n, n, n, with_ws=True) == mp.select_variant("s4", n, n, n)
    # ragged edges: the one-wave-per-SIMD kernel (its panels bounded by the
    # rows inside the matrix) where the rounds of 256 x 256 tiles are at least
    # 60% filled and K >= 4096, the 8-wave one for shorter K, the 128 x 128
    # kernel below 60%; K off its 128-byte slices: the 64-byte kernels
    assert mp.variant_name("f16", mp.select_variant("f16", 7000, 7000, 7168)) == "wide256x256_w2x2_k128_m16"
    assert mp.variant_name("f16", mp.select_variant("f16", 1800, 7000, 2048)) == "pipe256x256_w2x4_k128_s2"
    assert mp.variant_name("s8", mp.select_variant("s8", 7040, 7168, 2048)) == "pipe256x256_w2x4_k128_s2"
    assert mp.variant_name("f16", mp.select_variant("f16", 4096 + 64, 4096, 4096)) == "spread128x128_w2x4_k128_s4"
    assert mp.variant_name("s8", mp.select_variant("s8", 6784, 2432, 4096)) == "spread128x128_w2x4_k128_s4"
    assert mp.variant_name("s8", mp.select_variant("s8", 4000, 4400, 6400)) == "spread128x128_w2x4_k128_s4"
    # with a workspace the stream-K schedule splits the partial last round
    assert mp.variant_name("s8", mp.select_variant("s8", 4000, 4400, 6400, with_ws=True)).startswith("wide256x256")
    assert mp.variant_name("s8", mp.select_variant("s8", 8000, 8000, 8000)) == "spread128x128_w2x4_k64_s4"


def _e3m2_value(c):
    """Value of a 6-bit FP6 E3M2 code from the format's definition: sign bit 5,
    exponent bits 4..2 with bias 3, mantissa bits 1..0, subnormals at
    exponent 0 (OCP Microscaling Formats v1.0)."""
    sign = -1.0 if c & 0x20 else 1.0
    e, m = (c >> 2) & 7, c & 3
    mag = (m / 4.0) * 2.0 ** (1 - 3) if e == 0 else (1 + m / 4.0) * 2.0 ** (e - 3)
    return sign * mag


def test_s4_to_fp6_encoding_is_exact():
    """Every nibble's FP6 code decodes to the nibble's two's-complement value,
    each nibble lands in exactly one of the 32 six-bit fields, at field
    8d + 4h + i for byte i, half h of word d (k offset 8d + 2i + h)."""
    rng = np.random.default_rng(5)
    runs = [bytes((2 * i) | ((2 * i + 1) << 4) for i in range(8)) * 2]  # nibbles 0..15, twice
    runs += [rng.integers(0, 256, 16, dtype=np.uint8).tobytes() for _ in range(200)]
    runs += [b"\x88" * 16, b"\x77" * 16, b"\x00" * 16, b"\xff" * 16]
    for run in runs:
        words = mp.s4_run_to_fp6(run)
        assert len(words) == 6
        bits = sum(int(w) << (32 * i) for i, w in enumerate(words))
        assert bits >> 192 == 0
        fields = set()
        for e in range(32):
            d, i, h = e // 8, (e % 8) // 2, e % 2
            f = 8 * d + 4 * h + i
            fields.add(f)
            nib = (run[e // 2] >> (4 * (e % 2))) & 0xF
            want = nib - 16 if nib >= 8 else nib
            assert _e3m2_value((bits >> (6 * f)) & 0x3F) == want, (run.hex(), e)
        assert fields == set(range(32))


def test_fp6_variants_bound_k():
    """The FP6 path accumulates in FP32: exact only while K (padded to 256)
    is at most 2^18, and every such K must be accepted."""
    fp6 = [v for v in range(mp.num_variants("s4")) if mp.variant_name("s4", v).startswith("fp6")]
    assert fp6
    for v in fp6:
        assert mp.variant_supports("s4", v, 64, 64, 1 << 18)
        assert mp.variant_supports("s4", v, 65, 3, 2)
        assert not mp.variant_supports("s4", v, 64, 64, (1 << 18) + 2)
        assert not mp.variant_supports("s4", v, 64, 64, 3)  # odd K is not INT4
    for dt in ("f16", "s8"):
        assert not any(mp.variant_name(dt, v).startswith("fp6") for v in range(mp.num_variants(dt)))


def test_fp6_wide_workspace_offset_bound():
    """The one-wave-per-SIMD FP6 kernel addresses each workspace part with
    32-bit byte offsets: 16 bytes per padded row and 32-k run of the larger
    operand must stay within 2^31 - 1; beyond that the 8-wave FP6 kernel
    takes the problem."""
    names = [mp.variant_name("s4", v) for v in range(mp.num_variants("s4"))]
    wide, pipe = names.index("fp6wide256x256_w2x2_k128_s3"), names.index("fp6pipe256x256_w2x4_k128_s2")
    # 65536 rows x 4096 runs x 16 bytes = 2^32: too far; 2^30 fits
    assert not mp.variant_supports("s4", wide, 65536, 256, 1 << 17)
    assert not mp.variant_supports("s4", wide, 256, 65536, 1 << 17)
    assert mp.variant_supports("s4", pipe, 65536, 256, 1 << 17)
    assert mp.variant_supports("s4", wide, 16384, 256, 1 << 17)
    # kernels fed by the pre-pass need a workspace: never the automatic choice
    for shape in [(65536, 4096, 1 << 17), (16384, 4096, 1 << 17), (8192, 8192, 8192), (4096, 4096, 70000)]:
        assert not mp.variant_name("s4", mp.select_variant("s4", *shape)).startswith("fp6")


def test_skinny_selection():
    """The streaming kernel while its workgroups stay few and long: up to 7
    rows (FP16, INT8) on the small side with 1024..8192 on the large one, 16
    rows with at most 4096, 32 rows for INT4; with a larger large side
    only for a large operand of at most 32 MiB or at least 32 K-steps per wave.
    16 large-side rows per workgroup with more than 8 K-steps of 64 bytes per
    wave, 32 with fewer, one 8-step prefetch group with exactly 8; never
    split."""
    name = lambda dt, M, N, K, **kw: mp.variant_name(dt, mp.select_variant(dt, M, N, K, **kw))
    for dt in ("f16", "s8", "s4"):
        for M in (1, 7) if dt != "s4" else (1, 7, 8):
            assert name(dt, M, 8192, 8192).startswith("skinny16x"), (dt, M)
            assert name(dt, 8192, M, 8192).startswith("skinny16x"), (dt, M)  # small N: operands swapped
            v = mp.select_variant(dt, M, 8192, 8192)
            assert mp.select_splits(dt, v, M, 8192, 8192) == 1
        assert name(dt, 16, 4096, 4096).startswith("skinny16x")
        assert not name(dt, 16, 1000, 8192).startswith("skinny")  # large side too small
        assert not name(dt, 8, 8192, 8192, a_ptr=(1 << 20) + 4).startswith("skinny")  # unaligned A
    assert name("f16", 7, 8192, 8192) == "skinny16x16_k64"       # 32 K-steps per wave
    assert name("f16", 7, 8192, 2048) == "skinny16x32_k64_d8"    # 8 K-steps per wave
    assert name("s8", 7, 8192, 8192) == "skinny16x16_k64"        # 16 K-steps per wave
    for dt in ("f16", "s8"):  # from 8 rows the narrow tile with the eight-slice ring
        assert name(dt, 8, 8192, 8192) == "spread32x64_w1x2_k128_s8_m16"
        assert name(dt, 8192, 12, 8192) == "spread64x32_w2x1_k128_s8_m16"
    assert name("s8", 16, 4096, 4096) == "skinny16x32_k64_d8"    # 8 K-steps per wave
    assert name("s8", 16, 4096, 2048) == "skinny16x32_k64"       # 4 K-steps per wave
    assert name("s4", 16, 8192, 8192) == "skinny16x32_k64_d8"    # 8 K-steps per wave
    assert name("s4", 16, 4096, 14336) == "skinny16x16_k64"      # 14 K-steps per wave
    assert name("s4", 16, 14336, 4096) == "skinny16x32_k64"      # 4 K-steps; 28 MiB large operand
    assert name("s4", 24, 8192, 8192) == "skinny32x32_k64"
    assert name("s4", 8192, 32, 8192) == "skinny32x32_k64"
    # a large side beyond 8192: only a small large operand or long waves
    assert not name("f16", 1, 14336, 4096).startswith("skinny")  # 112 MiB, 16 K-steps per wave
    assert not name("s8", 1, 14336, 4096).startswith("skinny")   # 56 MiB, 8 K-steps per wave
    assert not name("s4", 1, 28672, 8192).startswith("skinny")   # 112 MiB, 8 K-steps per wave
    assert name("f16", 4, 28672, 8192) == "skinny16x16_k64"      # 32 K-steps per wave
    assert not name("s8", 16, 8192, 8160).startswith("skinny")  # K off the 64-byte step


def test_int4_large_tile_conditions():
    """INT4 on the 256 x 256 kernels: the one-wave-per-SIMD FP6 kernel only
    for M and N multiples of 256 (else, with a workspace, the 8-wave FP6 one),
    each only where its partial last round costs less than the FP6 rate gains
    at that K; without a workspace the in-GEMM E2M3 kernel only for whole
    tiles in one round or in whole rounds (K >= 4096), else the 128 x 128
    INT8-MFMA kernel (the 256 x 256 INT8-MFMA one for whole rounds E2M3
    cannot run)."""
    name = lambda M, N, K, ws: mp.variant_name("s4", mp.select_variant("s4", M, N, K, with_ws=ws))
    assert name(2944, 4608, 3328, True) == "fp6pipe256x256_w2x4_k128_s2"      # ragged, 84% filled
    assert name(7040, 7168, 2048, True) == "fp6pipe256x256_w2x4_k128_s2"      # ragged, 784 tiles
    assert name(3200, 6528, 8192, True) == "fp6pipe256x256_w2x4_k128_s2"      # ragged, 66%, long K
    assert name(3200, 6528, 4096, True) == "spread128x128_w2x4_k64_s4"        # ragged, 66%
    assert name(6784, 2432, 4096, True) == "spread128x128_w2x4_k64_s4"        # ragged, 53%
    assert name(6272, 3968, 2048, True) == "spread128x128_w2x4_k64_s4"        # ragged, short K
    assert name(4096, 6144, 4096, True).startswith("fp6wide256x256_w2x2_k128_s3")
    assert name(4608, 4608, 2048, True).startswith("fp6wide256x256_w2x2_k128_s3")  # 63%
    assert name(4352, 4096, 2048, True).startswith("spread128x128_w2x4_k64_s4")    # 53%, short K
    assert name(6784, 2432, 4096, False) == "spread128x128_w2x4_k64_s4"       # ragged
    assert name(4096, 6144, 4096, False) == "spread128x128_w2x4_k64_s4"       # 1.5 rounds
    assert name(3584, 3584, 3584, False) == "e2m3wide256x256_w2x2_k256"       # one round (196 tiles)
    assert name(8192, 4096, 4096, False) == "e2m3wide256x256_w2x2_k256"       # two whole rounds
    assert name(8192, 4096, 2048, False) == "staged256x256_w2x4_k128_n1"      # whole rounds, K < 4096


def test_narrow_selection():
    """8..512 rows on one side (past the streaming kernel) and at least 1024
    on the other: the narrow tiles, small side first; mirrored when N is the
    small side; from 65 rows also the eight-wave 128 x 128 kernel (for INT4
    its 64-byte-slice form). The picks below were each within 16% of the
    fastest candidate measured on MI355X (every narrow tile at 1, 2 and 4
    K-ranges)."""
    name = lambda dt, M, N, K, **kw: mp.variant_name(dt, mp.select_variant(dt, M, N, K, **kw))
    # the tile that copies the fewest bytes per CU (32 x 64: 224 tiles;
    # 64 x 128: 32 tiles, 4 K-ranges)
    assert name("f16", 1, 14336, 4096) == "spread32x64_w1x2_k128_s4_m16"   # 224 tiles
    assert name("s8", 32, 14336, 4096) == "spread32x64_w1x2_k128_s4_m16"
    assert name("s4", 64, 8192, 8192) == "spread32x64_w1x2_k128_s4_m16"    # 256 tiles
    assert name("f16", 64, 4096, 14336) == "spread64x128_w2x4_k128_s4"     # 32 tiles, 4 K-ranges
    # the eight-slice ring, unsplit, where K is long (at least 64 slices) and
    # 128..256 tiles fill one round: 32 x 64 with 128 or 256 tiles (FP16
    # 16 x 8192 x 8192: 24.9 against 27.1 us for 32 x 128 in 2 K-ranges)
    for M in (16, 32, 64):
        assert name("f16", M, 8192, 8192) == "spread32x64_w1x2_k128_s8_m16", M
    assert name("s8", 16, 8192, 8192) == "spread32x64_w1x2_k128_s8_m16"
    assert name("s8", 64, 8192, 8192) == "spread64x64_w2x2_k128_s8_m16"   # 256 tiles of 32 x 64: 64 slices too few
    assert name("f16", 16, 8192, 16384) == "spread32x64_w1x2_k128_s8_m16"
    assert name("f16", 16, 14336, 4096) == "spread32x64_w1x2_k128_s4_m16"  # 224 tiles of 64 slices
    assert name("f16", 32, 28672, 8192) == "spread32x128_w1x4_k128_s8_m16"  # 224 tiles of 128 slices
    want = {  # (M, N, K): f16, s8, s4 (INT4 never takes the eight-slice ring)
        (128, 8192, 8192): ("spread64x64_w2x2_k128_s8_m16", "spread64x64_w2x2_k128_s4_m16", "spread64x64_w2x2_k128_s4_m16"),
        (8192, 128, 8192): ("spread64x64_w2x2_k128_s8_m16", "spread64x64_w2x2_k128_s4_m16", "spread64x64_w2x2_k128_s4_m16"),
        (8192, 32, 8192): ("spread64x32_w2x1_k128_s8_m16", "spread64x32_w2x1_k128_s8_m16", "skinny32x32_k64"),
        (256, 8192, 8192): ("spread64x128_w2x4_k128_s4",) * 3,
        (8192, 256, 8192): ("spread128x64_w4x2_k128_s4",) * 3,
        (64, 14336, 4096): ("spread64x64_w2x2_k128_s4_m16",) * 3,
        # 224 tiles beat 448; INT4 takes the 64-byte-slice 128 x 128 kernel
        (128, 28672, 8192): ("spread128x128_w2x4_k128_s4",) * 2 + ("spread128x128_w2x4_k64_s4",),
        (256, 14336, 4096): ("spread128x128_w2x4_k128_s4",) * 2 + ("spread128x128_w2x4_k64_s4",),
        # 257 .. 512 rows (measured at 320, 384, 512 x 2048 .. 14336 x 2048 ..
        # 8192: 1.12x / 1.15x / 1.21x faster on average than the 128 x 128
        # kernel taken before, FP16 / INT8 / INT4)
        (512, 4096, 4096): ("spread64x128_w2x4_k128_s4",) * 3,
        (4096, 512, 4096): ("spread128x64_w4x2_k128_s4",) * 3,
        # above 256 rows, 64 x 64 tiles in one round (at most 256) and at
        # least 32 slices: the eight-slice ring (FP16 and INT8; 1.03-1.34x
        # the four-slice candidates at 30 of 50 measured shapes)
        (384, 2048, 4096): ("spread64x64_w2x2_k128_s8_m16",) * 2 + ("spread64x64_w2x2_k128_s4_m16",),
        (512, 2048, 8192): ("spread64x64_w2x2_k128_s8_m16",) * 2 + ("spread64x64_w2x2_k128_s4_m16",),  # unsplit
        (384, 2048, 2048): ("spread64x64_w2x2_k128_s8_m16",) + ("spread64x64_w2x2_k128_s4_m16",) * 2,  # INT8: 16 slices
        # from 257 rows, wherever 128 x 128 tiles would fill under half the CUs
        # (FP16 above 256 rows: the eight-wave 64 x 128 rather than 64 x 64)
        (1024, 1024, 4096): ("spread64x64_w2x2_k128_s8_m16",) * 2 + ("spread64x64_w2x2_k128_s4_m16",),
        (768, 768, 8192): ("spread64x64_w2x2_k128_s8_m16",) * 2 + ("spread64x64_w2x2_k128_s4_m16",),
        (1100, 1300, 4096): ("spread64x128_w2x4_k128_s4",) * 3,          # 378 tiles of 64 x 64
        (1280, 1280, 4096): ("spread64x128_w2x4_k128_s4",) * 3,          # 100 tiles of 128 x 128
        (1408, 1408, 2048): ("spread64x128_w2x4_k128_s4",) * 3,          # 121
        (384, 14336, 4096): ("spread128x128_w2x4_k128_s4",) * 2 + ("spread128x128_w2x4_k64_s4",),
        # 129 .. 256 rows, 64 x 64 tiles in one round: the eight-slice ring
        # (FP16 256 x 4096 x 4096: 18.6 against 22.7 us)
        (256, 4096, 14336): ("spread64x64_w2x2_k128_s8_m16",) * 2 + ("spread64x64_w2x2_k128_s4_m16",),
        (192, 2048, 4096): ("spread32x64_w1x2_k128_s8_m16",) * 2 + ("spread128x128_w2x4_k64_s4",),
    }
    for (M, N, K), names in want.items():
        assert tuple(name(dt, M, N, K) for dt in ("f16", "s8", "s4")) == names, (M, N, K)
    for dt in ("f16", "s8", "s4"):
        assert not name(dt, 1025, 4096, 4096).startswith(("spread32", "spread64"))  # past the narrow tiles
        assert not name(dt, 1536, 1536, 1536).startswith(("spread32", "spread64"))  # square: 144 tiles of 128
        assert mp.select_splits(dt, mp.select_variant(dt, 384, 2048, 8192), 384, 2048, 8192) == 1
        assert name(dt, 64, 1000, 8192).startswith("spread128")  # large side too small
        assert name(dt, 64, 8192, 8192 - 8).startswith("generic") or \
            name(dt, 64, 8192, 8192 - 8).startswith("spread128")  # K off the 128-byte slice
    assert name("s8", 8192, 64, 8192) == "spread64x64_w2x2_k128_s8_m16"
    for dt in ("f16", "s8"):  # the eight-slice ring is never split
        for v in range(mp.num_variants(dt)):
            if "_s8_m16" in mp.variant_name(dt, v):
                assert mp.select_splits(dt, v, 16, 8192, 8192) == 1


def test_split_k_selection():
    """Only problems with M or N <= 128 that neither the streaming kernel nor
    the narrow tiles take, and the narrow tiles themselves, are split: the
    128x128 tiles up to 256 workgroups (FP16 up to 4 K-ranges, integers up to
    2), the narrow tiles up to 128 workgroups and 4 K-ranges; square sweep
    sizes never."""
    for dt, most in (("f16", 4), ("s8", 2), ("s4", 2)):
        for n in (512, 1024, 2048, 4096, 8192):
            v = mp.select_variant(dt, n, n, n)
            assert mp.select_splits(dt, v, n, n, n) == 1
        for M in (64, 128):
            v = mp.select_variant(dt, M, 1000, 8192)  # large side too small for the narrow tiles
            assert mp.variant_name(dt, v).startswith("spread128")
            assert mp.select_splits(dt, v, M, 1000, 8192) == most
        v = mp.select_variant(dt, 64, 8192, 1024)
        assert mp.select_splits(dt, v, 64, 8192, 1024) <= most  # every range keeps >= 8 slices
    sel = lambda dt, M, N, K: mp.select_splits(dt, mp.select_variant(dt, M, N, K), M, N, K)
    split = lambda dt, name, M, N, K: mp.select_splits(
        dt, [v for v in range(mp.num_variants(dt)) if mp.variant_name(dt, v) == name][0], M, N, K)
    assert split("f16", "spread32x128_w1x4_k128_s4_m16", 32, 8192, 8192) == 2  # 64 tiles
    assert split("f16", "spread128x32_w4x1_k128_s4_m16", 8192, 32, 8192) == 2
    assert split("f16", "spread64x128_w2x4_k128_s4", 64, 8192, 8192) == 2      # 64 tiles
    assert split("f16", "spread128x128_w2x4_k128_s4", 128, 8192, 8192) == 2   # the narrow tiles' rule
    assert split("s8", "spread32x128_w1x4_k128_s4_m16", 32, 8192, 8192) == 2
    assert sel("f16", 32, 8192, 8192) == 1     # the eight-slice ring instead
    assert split("f16", "spread128x128_w2x4_k128_s4", 256, 4096, 14336) == 2
    assert sel("f16", 256, 4096, 14336) == 1   # the eight-slice 64 x 64 tiles instead
    assert sel("f16", 64, 4096, 8192) == 4     # 32 tiles
    assert sel("s8", 32, 14336, 4096) == 1     # 224 tiles of 32 x 64
    assert sel("s8", 128, 8192, 8192) == 1
    assert sel("f16", 256, 8192, 8192) == 1
    assert mp.select_splits("s8", 0, 16, 8192, 8192) == 1  # the bounds-checked kernel never splits
    L = mp.lib()
    assert L.mpgemm_select_splits(7, 1, 16, 16, 16) == -1
    assert L.mpgemm_select_splits(1, 999, 16, 16, 16) == -1
    assert L.mpgemm_select_splits(1, 1, -1, 16, 16) == -1
    assert L.mpgemm_select_splits(2, 1, 16, 16, 15) == -1  # odd K is not INT4


def test_every_variant_has_a_kernel_source_family():
    # stored counters are matched to a kernel through the hash of its sources
    import bench
    for dt in ("f16", "s8", "s4"):
        for v in range(mp.num_variants(dt)):
            assert len(bench.kernel_source_hash(mp.variant_name(dt, v))) == 16


def test_wide_variant_support():
    """The one-wave-per-SIMD kernel takes 128-byte K-slices of 16-byte
    aligned FP16 or INT8 operands, any M and N, nothing else."""
    for dt, e in (("f16", 64), ("s8", 128), ("s4", 256)):
        v = [i for i in range(mp.num_variants(dt)) if mp.variant_name(dt, i) == "wide256x256_w2x2_k128_m16"]
        assert len(v) == 1
        v = v[0]
        ok = dt != "s4"
        assert mp.variant_supports(dt, v, 256, 256, e) == ok
        assert mp.variant_supports(dt, v, 8192, 4096, 64 * e) == ok
        assert mp.variant_supports(dt, v, 257, 256, e) == ok      # ragged M
        assert mp.variant_supports(dt, v, 1, 200, e) == ok        # ragged N, one row
        assert not mp.variant_supports(dt, v, 256, 256, e + 2)   # K off the slice
        assert not mp.variant_supports(dt, v, 256, 256, e, a_ptr=(1 << 20) + 4)  # unaligned A


def _e2m3_value(c):
    """Value of a 6-bit FP6 E2M3 code from the format's definition: sign bit 5,
    exponent bits 4..3 with bias 1, mantissa bits 2..0, subnormals at
    exponent 0 (OCP Microscaling Formats v1.0)."""
    sign = -1.0 if c & 0x20 else 1.0
    e, m = (c >> 3) & 3, c & 7
    mag = (m / 8.0) * 2.0 ** (1 - 1) if e == 0 else (1 + m / 8.0) * 2.0 ** (e - 1)
    return sign * mag


# field order of each 16 codes from a word pair (x, y): x0 y1 x3 y4 x6 y7 x1 y2
# x4 y5 x7 y0 x2 y3 x5 y6 (nibble n of a word at bits 4n..4n+3)
E2M3_FIELDS = [(0, 0), (1, 1), (0, 3), (1, 4), (0, 6), (1, 7), (0, 1), (1, 2),
               (0, 4), (1, 5), (0, 7), (1, 0), (0, 2), (1, 3), (0, 5), (1, 6)]


def test_s4_to_e2m3_encoding_is_exact():
    """The in-GEMM INT4 conversion: every nibble v lands in exactly one of the
    32 fields, in the documented order, as an E2M3 code whose value is
    exactly (v + 8) / 8 (non-negative, below 2): the kernel's biased sums then
    differ from the integer sums by 8 Sa + 8 Sb + 64 K."""
    rng = np.random.default_rng(6)
    runs = [bytes((2 * i) | ((2 * i + 1) << 4) for i in range(8)) * 2]  # nibbles 0..15, twice
    runs += [rng.integers(0, 256, 16, dtype=np.uint8).tobytes() for _ in range(300)]
    runs += [b"\x88" * 16, b"\x77" * 16, b"\x00" * 16, b"\xff" * 16]
    for run in runs:
        words = mp.s4_run_to_e2m3(run)
        assert len(words) == 6
        bits = sum(int(w) << (32 * i) for i, w in enumerate(words))
        assert bits >> 192 == 0
        nib = [(run[e // 2] >> (4 * (e % 2))) & 0xF for e in range(32)]  # nibble e = k offset e
        for f in range(32):
            p, g = divmod(f, 16)
            which, n = E2M3_FIELDS[g]
            k = 8 * (2 * p + which) + n  # word 2p + which, nibble n
            v = nib[k] - 16 if nib[k] >= 8 else nib[k]
            code = (bits >> (6 * f)) & 0x3F
            assert _e2m3_value(code) == (v + 8) / 8.0, (run.hex(), f)
        used = sorted(8 * (2 * (f // 16) + E2M3_FIELDS[f % 16][0]) + E2M3_FIELDS[f % 16][1] for f in range(32))
        assert used == list(range(32))


def test_e2m3_bias_identity_is_exact():
    """The bias removal the kernel applies, checked on integers: with
    u = v + 8, sum u_a u_b - 8 Sa - 8 Sb - 64 K = sum a b, and the largest
    biased sum 225 K stays below 2^24 for every K the kernel takes."""
    rng = np.random.default_rng(7)
    for K in (256, 4096, 65536):
        a = rng.integers(-8, 8, K)
        b = rng.integers(-8, 8, K)
        ua, ub = a + 8, b + 8
        assert int(ua @ ub) - 8 * int(a.sum()) - 8 * int(b.sum()) - 64 * K == int(a @ b)
        assert 225 * K < 2 ** 24


def test_e2m3_wide_support():
    """The INT4 kernel with the conversion inside the GEMM: K a multiple of
    256 up to 65536 (225 K < 2^24), 16-byte aligned rows, any M and N."""
    v = [i for i in range(mp.num_variants("s4")) if mp.variant_name("s4", i) == "e2m3wide256x256_w2x2_k256"]
    assert len(v) == 1
    v = v[0]
    assert mp.variant_supports("s4", v, 256, 256, 256)
    assert mp.variant_supports("s4", v, 300, 77, 65536)            # ragged M and N
    assert not mp.variant_supports("s4", v, 256, 256, 65536 + 256)  # beyond the exact range
    assert not mp.variant_supports("s4", v, 256, 256, 384)          # K off the 256 grid
    assert not mp.variant_supports("s4", v, 256, 256, 512, a_ptr=(1 << 20) + 8)
    for dt in ("f16", "s8"):
        assert not any(mp.variant_name(dt, i).startswith("e2m3") for i in range(mp.num_variants(dt)))
    # beyond its K range INT4 runs on the INT8 MFMA (K < 131072), then the bounds-checked kernel
    assert mp.variant_name("s4", mp.select_variant("s4", 4096, 4096, 65536 + 256)).startswith("staged")
    assert mp.select_variant("s4", 256, 256, 131072) == 0


def test_workspace_sizes():
    """The plain entry points' kernels need no workspace; split K needs the
    counter block plus its partial tiles, zero points their row sums, the FP6
    pre-pass variants their converted operands."""
    counters = 64 * 1024
    for dt in ("f16", "s8", "s4"):
        for n in (512, 1024, 2048, 4096, 8192):
            want = counters + 2 * n * n * 3 // 4 if (dt == "s4" and n >= 4096) else 0  # FP6 pre-pass operands
            assert mp.workspace_size(dt, n, n, n) == want, (dt, n)
            if dt == "s4" and n >= 4096:  # the workspace-free choice of the plain entry point needs none
                assert mp.workspace_size(dt, n, n, n, variant=mp.select_variant(dt, n, n, n)) == 0
        assert mp.workspace_size(dt, 0, 5, 8) == 0
    # 128 rows on the small side: 128x128 tiles split 4 ways (FP16)
    v = mp.select_variant("f16", 64, 1000, 8192)
    sp = mp.select_splits("f16", v, 64, 1000, 8192)
    assert sp == 4
    assert mp.workspace_size("f16", 64, 1000, 8192) == counters + 8 * sp * 128 * 128 * 4
    assert mp.workspace_size("f16", 64, 1000, 8192, variant=v, splits=1) == 0
    # zero points: 4 (M + N) bytes rounded to 256, after the counter block
    E = mp.gemm.Epilogue
    zp = E(None, None, 1 << 20, None, 2)
    assert mp.workspace_size("s8", 512, 512, 512, epi=zp) == counters + 4096
    assert mp.workspace_size("s8", 100, 3, 512, epi=zp) == counters + 512
    assert mp.workspace_size("s8", 512, 512, 512, epi=E(1 << 20, None, None, None, 2)) == 0
    # an FP6 pre-pass variant: 0.75 byte per padded element of A and B
    names = [mp.variant_name("s4", i) for i in range(mp.num_variants("s4"))]
    f6 = names.index("fp6wide256x256_w2x2_k128_s3")
    assert mp.workspace_size("s4", 1000, 300, 1000, variant=f6) == counters + (1024 + 512) * 1024 * 3 // 4
    with pytest.raises(mp.HipError):
        mp.workspace_size("s8", -1, 8, 8)
    with pytest.raises(mp.HipError):
        mp.workspace_size("f16", 256, 256, 256, epi=zp)  # zero points with FP16 inputs
    with pytest.raises(mp.HipError):
        mp.workspace_size("s8", 256, 256, 256, variant=0, splits=2)  # the bounds-checked kernel does not split


def test_workspace_arguments_rejected_on_host():
    """A misaligned workspace, one overlapping an operand, or none where the
    call cannot do without: refused before anything is enqueued."""
    L = mp.lib()
    A, B, C = 1 << 20, 1 << 40, 1 << 44
    W = 1 << 46
    gw = lambda ws, n, M=64, N=64, K=64, epi=None: L.mpgemm_gemm_ws(1, M, N, K, A, B, C, epi, ws, n, None)
    assert gw(W + 16, 1 << 20) == 1               # not 256-byte aligned
    assert gw(C, 1 << 20) == 1                    # overlaps C
    assert gw(A - 256, 1 << 20) == 1              # overlaps A
    E = mp.gemm.Epilogue
    zp = E(None, None, 1 << 30, None, 2)
    import ctypes as ct
    assert L.gemm_scaled(1, 64, 64, 64, A, B, C, ct.addressof(zp), None) == 1   # zero points need a workspace
    assert L.mpgemm_gemm_ws(1, 64, 64, 64, A, B, C, ct.addressof(zp), W, 256, None) == 1  # too small
    names = [mp.variant_name("s4", i) for i in range(mp.num_variants("s4"))]
    f6 = names.index("fp6wide256x256_w2x2_k128_s3")
    assert L.mpgemm_run_variant_ws(2, f6, 0, 256, 256, 256, A, B, C, None, None, 0, None) == 1
    v = mp.select_variant("s8", 64, 1000, 8192)
    assert L.mpgemm_run_variant_ws(1, v, 2, 64, 1000, 8192, A, B, C, None, None, 0, None) == 1
    assert L.mpgemm_run_variant_ws(1, v, -1, 64, 1000, 8192, A, B, C, None, None, 0, None) == 1


def test_int8_short_k_takes_64_byte_slices_past_one_round():
    """INT8 with K <= 2048 and more than 256 tiles of 128 x 128: the
    64-byte-slice kernel (measured 1.02-1.22x faster there on MI355X); one
    round or longer K: the 128-byte one."""
    name = lambda M, N, K: mp.variant_name("s8", mp.select_variant("s8", M, N, K))
    assert name(2048, 4096, 2048) == "spread128x128_w2x4_k64_s4"
    assert name(2304, 3456, 2048) == "spread128x128_w2x4_k64_s4"
    assert name(2048, 2048, 2048) == "spread128x128_w2x4_k128_s4"   # 256 tiles
    assert name(2560, 2560, 4096) == "spread128x128_w2x4_k128_s4"   # 32 slices
    assert mp.variant_name("f16", mp.select_variant("f16", 2048, 4096, 2048)) == "spread128x128_w2x4_k128_s4"
