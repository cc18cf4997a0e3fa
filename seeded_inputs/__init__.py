"""Seeded synthetic inputs for the dense GEMM workloads.

Both the CPU oracle tests and the GPU path draw their operands from here. The
module holds no GEMM arithmetic: it only produces random words, maps them to the
workload value distributions, and lays the values out in the storage formats the
library takes.

Random stream: counter-based SplitMix64 (Steele, Lea and Flood, "Fast
splittable pseudorandom number generators", OOPSLA 2014, with the constants of
Vigna's public-domain reference). Word ``c`` of the stream with seed ``s`` is
``mix(s + (c + 1) * GAMMA)`` modulo 2**64, so any slice of the stream can be
generated independently, which keeps large matrices vectorised and chunked.

Storage formats (the paper's operand layouts: A row-major, B column-major, in
its description of the ``.row.col`` MMA shapes):
  * A is M x K row-major: element (i, k) at offset i*K + k.
  * B is K x N column-major: element (k, j) at offset j*K + k. In numpy this is
    an (N, K) C-contiguous array, called ``B`` throughout.
  * INT4 values are packed two per byte along K: the low nibble holds the even
    k, the high nibble the odd k, both two's complement.

Counter assignment for one (A, B) pair: A takes words 0 .. M*K-1 in its storage
order, B takes the next K*N words in its storage order. INT4 draws one word per
logical element (not per byte).
"""
from __future__ import annotations

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
_MIX1 = 0xBF58476D1CE4E5B9
_MIX2 = 0x94D049BB133111EB
_MASK64 = (1 << 64) - 1
_CHUNK = 1 << 22

# Sweep order for the precision x size points: precision-major (FP16, INT8,
# INT4), N ascending; point i uses seed SWEEP_SEED0 + i.
SWEEP_DTYPES = ("f16", "s8", "s4")
SWEEP_SIZES = (512, 1024, 2048, 4096, 8192)
SWEEP_SEED0 = 10


def splitmix64_scalar(seed: int, counter: int) -> int:
    """Word ``counter`` of the stream, in plain Python integers (the reference
    form; the vectorised generator is tested against it)."""
    z = (seed + (counter + 1) * GAMMA) & _MASK64
    z = ((z ^ (z >> 30)) * _MIX1) & _MASK64
    z = ((z ^ (z >> 27)) * _MIX2) & _MASK64
    return z ^ (z >> 31)


def splitmix64(seed: int, start: int, count: int) -> np.ndarray:
    """Words ``start .. start+count-1`` of the stream as a uint64 array."""
    out = np.empty(count, dtype=np.uint64)
    g = np.uint64(GAMMA)
    s = np.uint64(seed & _MASK64)
    m1 = np.uint64(_MIX1)
    m2 = np.uint64(_MIX2)
    with np.errstate(over="ignore"):
        for lo in range(0, count, _CHUNK):
            n = min(_CHUNK, count - lo)
            z = np.arange(start + lo + 1, start + lo + 1 + n, dtype=np.uint64)
            z *= g
            z += s
            z ^= z >> np.uint64(30)
            z *= m1
            z ^= z >> np.uint64(27)
            z *= m2
            z ^= z >> np.uint64(31)
            out[lo:lo + n] = z
    return out


# --- word -> value maps --------------------------------------------------------

def words_to_int8(w: np.ndarray) -> np.ndarray:
    """Top 8 bits as a signed byte: uniform over [-128, 127]."""
    return (w >> np.uint64(56)).astype(np.uint8).view(np.int8)


def words_to_int4(w: np.ndarray) -> np.ndarray:
    """Top 4 bits as a two's-complement nibble: uniform over [-8, 7] (int8)."""
    nib = (w >> np.uint64(60)).astype(np.int8)
    return np.where(nib >= 8, nib - 16, nib).astype(np.int8)


def words_to_unit(w: np.ndarray) -> np.ndarray:
    """Top 53 bits scaled to [0, 1) in float64."""
    return (w >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def words_to_uniform_pm1_f16(w: np.ndarray) -> np.ndarray:
    """U[-1, 1) in float64, rounded to binary16 (round to nearest even)."""
    return (2.0 * words_to_unit(w) - 1.0).astype(np.float16)


def normal_f16(seed: int, start: int, count: int) -> np.ndarray:
    """N(0, 1) by Box-Muller on consecutive word pairs, rounded to binary16.

    Element e uses words (start + 2*(e//2), +1) when start is even: u1 in
    (0, 1], u2 in [0, 1); even e takes r*cos(2*pi*u2), odd e r*sin(2*pi*u2).
    """
    if start % 2:
        raise ValueError("normal_f16 needs an even start counter")
    npairs = (count + 1) // 2
    w = splitmix64(seed, start, 2 * npairs)
    u1 = 1.0 - words_to_unit(w[0::2])
    u2 = words_to_unit(w[1::2])
    r = np.sqrt(-2.0 * np.log(u1))
    out = np.empty(2 * npairs, dtype=np.float64)
    out[0::2] = r * np.cos(2.0 * np.pi * u2)
    out[1::2] = r * np.sin(2.0 * np.pi * u2)
    return out[:count].astype(np.float16)


# --- INT4 storage --------------------------------------------------------------

def pack_s4(v: np.ndarray) -> np.ndarray:
    """Pack signed 4-bit values (int8 in [-8, 7], last axis even) two per byte:
    low nibble = even index, high nibble = odd index."""
    v = np.asarray(v)
    if v.shape[-1] % 2:
        raise ValueError("INT4 packing needs an even length along K")
    if v.size and (v.min() < -8 or v.max() > 7):
        raise ValueError("INT4 values must lie in [-8, 7]")
    u = v.astype(np.int16) & 0xF
    return (u[..., 0::2] | (u[..., 1::2] << 4)).astype(np.uint8)


# --- matrices -----------------------------------------------------------------

def gen_operands(dtype: str, M: int, N: int, K: int, seed: int,
                 dist: str = "default"):
    """Seeded A (M x K row-major) and B (K x N column-major, as an (N, K) array).

    dtype "f16": dist "uniform" (U[-1,1], the default) or "normal" (N(0,1)),
                 returned as float16 arrays.
    dtype "s8":  uniform over [-128, 127], int8 arrays.
    dtype "s4":  uniform over [-8, 7], packed uint8 arrays of shape (M, K/2)
                 and (N, K/2).
    """
    na, nb = M * K, N * K
    if dtype == "f16":
        if dist in ("default", "uniform"):
            a = words_to_uniform_pm1_f16(splitmix64(seed, 0, na))
            b = words_to_uniform_pm1_f16(splitmix64(seed, na, nb))
        elif dist == "normal":
            # pairs must not straddle A and B: B starts at the next even word
            a = normal_f16(seed, 0, na)
            b = normal_f16(seed, na + (na % 2), nb)
        else:
            raise ValueError(f"unknown f16 distribution {dist!r}")
        return a.reshape(M, K), b.reshape(N, K)
    if dtype == "s8":
        a = words_to_int8(splitmix64(seed, 0, na))
        b = words_to_int8(splitmix64(seed, na, nb))
        return a.reshape(M, K), b.reshape(N, K)
    if dtype == "s4":
        if K % 2:
            raise ValueError("INT4 needs even K")
        a = words_to_int4(splitmix64(seed, 0, na)).reshape(M, K)
        b = words_to_int4(splitmix64(seed, na, nb)).reshape(N, K)
        return pack_s4(a), pack_s4(b)
    raise ValueError(f"unknown dtype {dtype!r}")


def sample_rows(seed: int, n: int, count: int, force=(0,)) -> np.ndarray:
    """``count`` distinct rows of [0, n) by a partial Fisher-Yates shuffle driven
    by the stream ``seed``, plus the rows in ``force``; sorted, as int32."""
    perm = np.arange(n, dtype=np.int64)
    w = splitmix64(seed, 0, count)
    for t in range(min(count, n)):
        j = t + int(w[t] % np.uint64(n - t))
        perm[t], perm[j] = perm[j], perm[t]
    rows = set(int(r) for r in perm[:count]) | {int(r) % n for r in force}
    return np.array(sorted(rows), dtype=np.int32)


def sweep_points():
    """The precision x size sweep: list of (dtype, N, seed)."""
    pts = []
    i = 0
    for dt in SWEEP_DTYPES:
        for n in SWEEP_SIZES:
            pts.append((dt, n, SWEEP_SEED0 + i))
            i += 1
    return pts


# Named workloads with their seeds and distributions.
WORKLOADS = {
    "f16_512": dict(dtype="f16", n=512, seed=0, dist="uniform"),
    "s8_2048": dict(dtype="s8", n=2048, seed=1, dist="default"),
    "s4_4096": dict(dtype="s4", n=4096, seed=2, dist="default"),
    "f16_8192": dict(dtype="f16", n=8192, seed=3, dist="normal"),
}
# rows of the 8192 FP16 output checked in full: 256 drawn, plus the first and last
F16_8192_ROW_SEED = 3 + 1000
F16_8192_ROW_COUNT = 256
