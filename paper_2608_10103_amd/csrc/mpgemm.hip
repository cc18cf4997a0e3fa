// mpgemm.hip - the C-ABI entry points: argument checks, kernel choice, launch.
//
// Every entry point validates its arguments on the host, picks a kernel
// variant (a tiled kernel when the problem fits its constraints, the
// bounds-checked kernel otherwise) and launches it on the caller's stream with
// hipLaunchKernel, returning the launch status. Nothing here allocates,
// frees, copies or synchronises, and no state is kept between calls: the
// kernels that need scratch memory (split K, the FP6 pre-pass variants, the
// zero-point row sums) take it from a workspace the caller passes in.
#include <hip/hip_runtime.h>
#include <limits.h>
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "mpgemm.h"
#include "variants.hpp"

using namespace mpg;

namespace {

const Variant *table(int dtype) {
    switch (dtype) {
        case F16: return kF16;
        case S8: return kS8;
        case S4: return kS4;
        default: return nullptr;
    }
}

int num_variants(int dtype) {
    switch (dtype) {
        case F16: return kNumF16;
        case S8: return kNumS8;
        case S4: return kNumS4;
        default: return -1;
    }
}

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// Byte ranges [p, p + n) and [q, q + m) intersect (empty ranges never do).
bool overlap(const void *p, uint64_t n, const void *q, uint64_t m) {
    if (n == 0 || m == 0) return false;
    const uintptr_t a = reinterpret_cast<uintptr_t>(p), b = reinterpret_cast<uintptr_t>(q);
    return a < b + m && b < a + n;
}

// Argument checks shared by every entry point (see the header's Errors);
// c_elem = bytes per element of C (4, or 2 for FP16/BF16 scaled outputs).
bool valid_args(int dtype, int M, int N, int K, const void *A, const void *B, const void *C,
                int c_elem = 4) {
    if (dtype < F16 || dtype > S4) return false;
    if (M < 0 || N < 0 || K < 0) return false;
    if (K > INT_MAX - 64) return false;
    if (dtype == S4 && (K & 1)) return false;
    if (M == 0 || N == 0) return true;
    if (!C || !aligned(C, (uintptr_t)c_elem)) return false;
    if (K > 0) {
        if (!A || !B) return false;
        if (dtype == F16 && (!aligned(A, 2) || !aligned(B, 2))) return false;
    }
    const uint64_t rb = (uint64_t)row_bytes(dtype, K);
    const uint64_t a_bytes = (uint64_t)M * rb, b_bytes = (uint64_t)N * rb;
    const uint64_t c_bytes = (uint64_t)M * (uint64_t)N * (uint64_t)c_elem;
    if (c_bytes / (uint64_t)c_elem / (uint64_t)N != (uint64_t)M) return false;
    if (uintptr_t(-1) - reinterpret_cast<uintptr_t>(C) < c_bytes) return false;
    if (K > 0 && (overlap(C, c_bytes, A, a_bytes) || overlap(C, c_bytes, B, b_bytes))) return false;
    // the bounds-checked kernel indexes tiles with a 32-bit grid
    const uint64_t tiles = ((uint64_t)M + 31) / 32 * (((uint64_t)N + 31) / 32);
    if (tiles > (uint64_t)INT_MAX) return false;
    return true;
}

// FP6 path limits: partial sums stay exact in FP32 while K <= 2^18 (after
// padding); the conversion grid indexes rows in 32-row blocks (grid.y).
constexpr long kF6MaxK = 1L << 18;
constexpr long kF6MaxRows = 65535L * 32;

// Split-K buffer: kSplitCounters tile counters, then the partial tiles.
constexpr int kSplitCounters = 16384;
constexpr size_t kSplitCounterBytes = (size_t)kSplitCounters * 4;

constexpr int kMaxDevices = 64;

bool supports(int dtype, const Variant &v, int M, int N, int K, const void *A, const void *B,
              const void *C) {
    if (v.kind == GENERIC) return true;
    if (M == 0 || N == 0 || K == 0) return false;
    if (v.kind == SKINNY) {
        // the small operand (A if M is small, else B) has at most bm rows;
        // whole 64-byte K-steps; 16-byte aligned rows
        if (M > v.bm && N > v.bm) return false;
        const long kb = row_bytes(dtype, K);
        if (kb % v.bkb || kb > INT_MAX) return false;
        if (!aligned(A, 16) || !aligned(B, 16)) return false;
        if (dtype == S4 && K >= 131072) return false;  // INT4 sums carried times 256
        return true;
    }
    if (v.kind == WIDE || v.kind == WIDE_SK) {
        // 128-byte K-slices, 16-byte aligned rows (M and N any); the copy
        // buffers span 128 rows of K bytes (32-bit range)
        if (!v.fn) return false;
        const long kb = row_bytes(dtype, K);
        if (kb % v.bkb || 128 * kb > INT_MAX) return false;
        return aligned(A, 16) && aligned(B, 16);
    }
    if (v.kind == FP6 || v.kind == FP6WIDE || v.kind == FP6WIDE_SK) {
        if (dtype != S4 || !v.fn) return false;
        if (F6Geom::runs_pad(K) * 32 > kF6MaxK) return false;
        if (F6Geom::rows_pad(M) > kF6MaxRows || F6Geom::rows_pad(N) > kF6MaxRows) return false;
        // the one-wave-per-SIMD kernel addresses each workspace part (P: 16
        // bytes per row and run) with 32-bit byte offsets
        if (v.kind == FP6WIDE || v.kind == FP6WIDE_SK)
            return F6Geom::runs_pad(K) * 16 * (F6Geom::rows_pad(M) > F6Geom::rows_pad(N) ? F6Geom::rows_pad(M)
                                                                                          : F6Geom::rows_pad(N)) <= INT_MAX;
        return true;
    }
    if (v.kind == I4WIDE) {
        // whole 256-k slice pairs, K within the exact range of the biased
        // E2M3 sums, 16-byte aligned rows; M and N may be ragged
        if (dtype != S4 || K % v.bkb || K > WideI4Cfg::MAX_K) return false;
        return aligned(A, 16) && aligned(B, 16);
    }
    const long kb = row_bytes(dtype, K);
    // edge tiles are predicated in M and N; K must fill whole slices
    if (kb % v.bkb) return false;
    if (!aligned(A, 16) || !aligned(B, 16)) return false;
    // INT4 partial sums are carried scaled by 256 (see s4_lo_x16)
    if (dtype == S4 && K >= 131072) return false;
    if (kb > INT_MAX) return false;
    return true;
}

// Split-K (pipelined variants only): `splits` K-ranges of whole slices per
// tile, at most kMaxSplits, the tile count within the counter block.
constexpr int kMaxSplits = 16;

long tile_count(const Variant &v, int M, int N) {
    return (long)((M + v.bm - 1) / v.bm) * ((N + v.bn - 1) / v.bn);
}

bool splits_ok(int dtype, const Variant &v, int M, int N, int K, int splits) {
    if (splits == 1) return true;
    if (!v.splitk || splits < 1 || splits > kMaxSplits) return false;
    if (tile_count(v, M, N) > kSplitCounters) return false;
    return row_bytes(dtype, K) % ((long)v.bkb * splits) == 0;
}

// Workgroups of the stream-K kernels resident at once on the current device:
// one per CU (their LDS use allows no second). 256, MI355X's count, when no
// device is visible (size queries on a host without one).
int resident_groups() {
    static std::atomic<int> cus[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
    int n = cus[dev].load(std::memory_order_relaxed);
    if (n > 0) return n;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev].store(n, std::memory_order_relaxed);
    return n;
}

// Stream-K schedule of a call (stream_k.hpp): with T tiles, G resident
// workgroups and T = q G + r, 0 < r <= G / 2, the first q G tiles whole,
// then the r remaining tiles in `parts` K-parts each. Off (every tile whole,
// one workgroup each) for other variants, when the tiles fill whole rounds
// or the last round more than half, beyond the counter block, or where the
// cost model below expects no gain.
//
// Cost model, in microseconds (timelines of the kernels at 4352 x 4096 x
// {4096, 8192} on MI355X): a remainder tile's time without stream-K is
// KT t (KT K-slices of t each: t about 1 us for a 128-byte slice of a
// 256 x 256 tile, FP16 and INT8 alike, proportionally less for 128 x 128
// tiles, whose partials are proportionally smaller, so t = 1 for them too;
// half for 64-byte slices; about 0.5 us for the FP6 kernel's 128-k slices);
// with s parts it is KT t / s, plus about 5 per partial tile the finishing
// part loads (s - 1; one workgroup reads them at about 50 GB/s) and about
// 13 for publishing, fencing and counting. Gain(s) = KT t (1 - 1/s) -
// 5 (s - 1) - 13 peaks near s = sqrt(KT t / 5); stream-K is taken when that
// gain exceeds a tenth of KT t (K-ranges of about 48 slices and more: FP16
// K >= 3072, INT8 K >= 6144 with 256 x 256 tiles), a quarter for the FP6
// kernel (interleaved timings of both schedules at 6 INT4 shapes: gains
// of 9% at 4352 x 4096 x 16384 and 6% at 2048 x 2048 x 16384, losses of up
// to 4% where a tenth was cleared and a quarter is not).
struct SkPlan {
    bool on;
    int dp_tiles, parts, grid;
};

constexpr int kSkMaxParts = 8;

bool is_sk(const Variant &v) { return v.kind == TILED_SK || v.kind == WIDE_SK || v.kind == FP6WIDE_SK; }

SkPlan sk_off(long tiles) { return SkPlan{false, (int)tiles, 1, (int)tiles}; }

SkPlan sk_plan(int dtype, const Variant &v, int M, int N, int K) {
    const long tiles = tile_count(v, M, N);
    if (!is_sk(v) || tiles > kSplitCounters) return sk_off(tiles);
    const long G = resident_groups(), r = tiles % G;
    if (r == 0 || 2 * r > G) return sk_off(tiles);
    // 128 x 128 tiles with no whole round before the remainder: splitting the
    // few tiles measured slower (FP16 1200 x 1100 x 4096, 90 tiles in 2 parts:
    // 31.3 against 28.8 us)
    if (tiles < G && (long)v.bm * v.bn < 256 * 256) return sk_off(tiles);
    // slices per tile (the FP6 kernel: 128-k slices of the padded K), the
    // time of a lone remainder tile's slice in microseconds, and the margin
    // the modelled gain must clear (a fraction of the remainder round)
    const bool f6 = v.kind == FP6WIDE_SK;
    const long KT = f6 ? F6Geom::runs_pad(K) / v.bkb : row_bytes(dtype, K) / v.bkb;
    const double t = f6 ? 0.5 : v.bkb / 128.0, margin = f6 ? 0.25 : 0.1;
    long parts = (long)(sqrt(KT * t / 5.0) + 0.5);
    if (parts > G / r) parts = G / r;
    if (parts > kSkMaxParts) parts = kSkMaxParts;
    if (parts > KT / 2) parts = KT / 2;  // at least two slices per part
    if (parts < 2) return sk_off(tiles);
    const double gain = KT * t * (1.0 - 1.0 / parts) - 5.0 * (parts - 1) - 13.0;
    if (gain <= margin * KT * t) return sk_off(tiles);
    const long dp = tiles - r;
    return SkPlan{true, (int)dp, (int)parts, (int)(dp + r * parts)};
}

// Variant indices in the tables above that the selection uses.
enum : int {
    V_PIPE256_W2X4 = 9,      // pipe256x256_w2x4_k128_s2
    V_WIDE = 50,             // wide256x256_w2x2_k128_m16
    V_SPREAD128W8 = 54,      // spread128x128_w2x4_k128_s4
    V_SPREAD128W8_K64 = 55,  // spread128x128_w2x4_k64_s4
    V_SPREAD128_K128 = 20,   // spread128x128_w2x2_k128_s4
    V_SPREAD128_K64 = 21,    // spread128x128_w2x2_k64_s4
    V_STAGED256_W2X4 = 25,   // staged256x256_w2x4_k128_n1
    V_PIPE64 = 13,           // pipe64x64_w1x1_k128_s4
    V_SKINNY = 38,           // skinny16x16_k64; then 16x32, 32x16, 32x32
    V_SKINNY16_D8 = 42,      // skinny16x32_k64_d8
};
// The stream-K schedules of five of them, the last entries of the common
// list.
constexpr int V_WIDE_SK = kNumCommon - 5, V_PIPE256_SK = kNumCommon - 4, V_SPREAD128_SK = kNumCommon - 3,
              V_SPREAD128W8_SK = kNumCommon - 2, V_SPREAD128W8_K64_SK = kNumCommon - 1;

// INT4-only variants follow the common list in kS4.
constexpr int V_FP6_256_S2 = kNumCommon + 1;  // fp6pipe256x256_w2x4_k128_s2
constexpr int V_FP6_WIDE = kNumCommon + 8;    // fp6wide256x256_w2x2_k128_s3
constexpr int V_I4WIDE = kNumCommon + 9;      // e2m3wide256x256_w2x2_k256
constexpr int V_FP6_WIDE_SK = kNumCommon + 16;  // fp6wide256x256_w2x2_k128_s3_sk

// The stream-K twin of a variant (the same kernel with the stream-K
// schedule), or -1. The FP6 indices exist only in the INT4 table, where the
// INT4 preferences are the only callers that name them.
int sk_twin(int variant) {
    switch (variant) {
        case V_WIDE: return V_WIDE_SK;
        case V_PIPE256_W2X4: return V_PIPE256_SK;
        case V_SPREAD128_K128: return V_SPREAD128_SK;
        case V_SPREAD128W8: return V_SPREAD128W8_SK;
        case V_SPREAD128W8_K64: return V_SPREAD128W8_K64_SK;
        case V_FP6_WIDE: return V_FP6_WIDE_SK;
        default: return -1;
    }
}

// The variant a stream-K twin schedules differently, or -1.
int sk_base(int variant) {
    switch (variant) {
        case V_WIDE_SK: return V_WIDE;
        case V_PIPE256_SK: return V_PIPE256_W2X4;
        case V_SPREAD128_SK: return V_SPREAD128_K128;
        case V_SPREAD128W8_SK: return V_SPREAD128W8;
        case V_SPREAD128W8_K64_SK: return V_SPREAD128W8_K64;
        case V_FP6_WIDE_SK: return V_FP6_WIDE;
        default: return -1;
    }
}

// Narrow-tile variants (select_narrow): three tiles with the small side on
// A's rows, then the same three mirrored; and three with more waves (64 x 64,
// 64 x 128 and its mirror).
constexpr int V_NARROW = 44;  // spread32x64_w1x2_k128_s4_m16, 32x128, 64x128; 64x32, 128x32, 128x64
constexpr int kNumNarrow = 6;
constexpr int V_NARROW64 = 56;      // spread64x64_w2x2_k128_s4_m16
constexpr int V_NARROW64W8 = 57;    // spread64x128_w2x4_k128_s4; then its mirror 128 x 64
constexpr int kNumNarrowW = 3;
// The same narrow tiles with an eight-slice ring, never split: 32 x 64,
// 32 x 128, their mirrors 64 x 32 and 128 x 32, then 64 x 64.
constexpr int V_DEEP = 59;          // spread32x64_w1x2_k128_s8_m16
constexpr int kNumDeep = 5;

// Problems the narrow tiles serve: at most 1024 rows on the small side and
// at least 1024 on the large one, with the small side at most 512 rows or
// the large one at least twice as long; or, from 257 rows on, any problem
// whose 128 x 128 tiles would fill fewer than half the CUs (128 tiles).
// There the 128 x 128 kernel leaves CUs idle: 1280^2 x 4096 FP16 29.8 against
// 23.7 us with 64 x 128 tiles, 1024^2 x 4096 INT8 16.3 against 11.6 with
// 64 x 64, 512^2 x 8192 FP16 47.4 against 19.7; from 144 tiles on (1536^2
// and up) it is 1.2-1.4x faster than any narrow tile.
bool narrow_shape(int M, int N) {
    const int small = M < N ? M : N, large = M < N ? N : M;
    const long tiles128 = (long)((small + 127) / 128) * ((large + 127) / 128);
    return (small <= 1024 && large >= 1024 && (small <= 512 || large >= 2 * small)) ||
           (small > 256 && tiles128 < 128);
}

// The eight-wave 128 x 128 kernel that competes with the narrow tiles: the
// 64-byte-slice form for INT4 (as for square INT4 problems: 1.02-1.13x
// faster than the 128-byte one at 320 .. 512 x 8192 .. 14336), else the
// 128-byte one.
int spread128w8(int dtype) { return dtype == S4 ? V_SPREAD128W8_K64 : V_SPREAD128W8; }

// Variants split by the narrow tiles' rule (choose_splits): the narrow tiles,
// and on narrow shapes the eight-wave 128 x 128 kernel they compete with.
bool is_narrow(int dtype, const Variant &v, int M, int N) {
    const Variant *t = table(dtype);
    if ((&v >= t + V_NARROW && &v < t + V_NARROW + kNumNarrow) ||
        (&v >= t + V_NARROW64 && &v < t + V_NARROW64 + kNumNarrowW))
        return true;
    return &v == t + spread128w8(dtype) && narrow_shape(M, N);
}

bool is_deep(int dtype, const Variant &v) {
    const Variant *t = table(dtype);
    return &v >= t + V_DEEP && &v < t + V_DEEP + kNumDeep;
}

// Splits the entry points use. Only skinny problems (M or N at most 128, the
// LLM-inference shapes) are split: they stream one large operand from HBM,
// and splitting K lets more CUs stream it. Measured on MI355X at M = 16,
// N = K = 8192: FP16 51 -> 38 us with 4 ranges, INT8 28 -> 26 us with 2; for
// square problems with too few tiles the fixup (partials written back to L2
// with a device-scope release) costs more than the extra parallelism gains
// (N = 1024: 11 -> 15 us with 2 ranges), so they are not split. Each range
// keeps at least 8 slices. The narrow tiles split only while the grid stays
// within 128 workgroups (at 32 x 8192 x 8192 FP16 with 32 x 128 tiles:
// 27.4 us with 2 ranges, 30.5 us with 4; INT8 with 32 x 64 tiles: 17.6 us
// unsplit, 22.1 us with 2). The narrow tiles with the eight-slice ring are
// never split: their deeper ring is what the split bought.
int choose_splits(int dtype, const Variant &v, int M, int N, int K) {
    if (!v.splitk || v.kind != TILED || is_deep(dtype, v)) return 1;
    if (M > 128 && N > 128 && !is_narrow(dtype, v, M, N)) return 1;
    const bool narrow = is_narrow(dtype, v, M, N);
    // Above 256 rows on the small side the narrow choice runs unsplit: its
    // best unsplit tile is within 1% of the best split one on average
    // (320 .. 1024 rows), while the split 128 x 128 kernel the cost model
    // would take is up to 1.4x slower (FP16 768 x 768 x 8192).
    if (narrow && (M < N ? M : N) > 256) return 1;
    const int most = narrow ? 4 : (dtype == F16 ? 4 : 2);
    const long tiles = tile_count(v, M, N);
    const long slices = row_bytes(dtype, K) / v.bkb;
    int s = 1;
    while ((narrow ? tiles * 2 * s <= 128 : tiles * s < 256) && 2 * s <= most && slices % (2 * s) == 0 &&
           slices / (2 * s) >= 8 && splits_ok(dtype, v, M, N, K, 2 * s))
        s *= 2;
    return s;
}

// Preferred tiled variants per dtype, largest tile first; a candidate is
// taken when it supports the problem and yields at least `min_tiles`
// workgroups (256 = one per CU). Chosen from interleaved timings of every
// variant at N = 512 ... 8192 on MI355X.
struct Pref { int variant; long min_tiles; };
// INT4 without a workspace: the FP6 kernel with the conversion inside the
// GEMM (no pre-pass, no workspace) once 256 x 256 tiles fill the CUs (at
// 8192^3 415-455 us against 478 us for the INT8-MFMA kernels; at 2048^3 with
// 64 tiles it takes 36 us against 21 us for the 128 x 128 INT8-MFMA kernel);
// below that, or for K beyond its exact range or off its 256-k grid, the
// INT8-MFMA kernels.
// INT4 with a workspace large enough for the converted operands: the
// one-wave-per-SIMD FP6 kernel fed by the conversion pre-pass first (at
// 8192^3: 483k + 100k cycles per XCD for kernel and pre-pass, against 911k
// for the in-GEMM conversion, whose 16-half-line register loads and
// conversion do not overlap the MFMAs), then the 8-wave one where the first's
// 32-bit workspace offsets do not reach.
// FP16, INT8: below 256 tiles of 256 x 256 the 128 x 128 kernel with eight
// waves of 64 x 32 and 128-byte slices, the 64-byte one when K does not fill
// 128-byte slices. Against the four-wave 128 x 128 kernel (64 x 64 waves)
// chosen before, interleaved on MI355X at 512^3 ... 2560^3, 1024 x 8192 x
// 2048, 2048 x 4096 x 1024, 2000 x 1900 x 2048, 1000 x 3000 x 4096,
// 3968^2 x 4096 and 2100 x 2000 x 6400: FP16 1.06-1.32x, INT8 1.10-1.43x
// faster (more waves keep more copies and MFMAs in flight per CU).
// INT4 (no FP6 kernel): the eight-wave kernel with 64-byte slices (128 k),
// 1.11-1.37x faster than the four-wave 128-byte-slice kernel at the same
// shapes.
// FP16, INT8: the one-wave-per-SIMD kernel first where whole 256 x 256 tiles
// fill the CUs (1.09-1.21x the 8-wave kernel for FP16, 1.12-1.23x for INT8,
// at 2048..16384 x 4096..16384 x 2048..16384). Where M or N is not a
// multiple of 256 (checked by ragged_pref_ok) both 256 x 256 kernels need the
// rounds of tiles at least 65% filled, and the one-wave-per-SIMD one also
// K >= 4096; the 8-wave one is then taken from 144 tiles. Interleaved on
// MI355X at 38 ragged shapes (1800 .. 12000 x 2432 .. 7168 x 2048 .. 8192):
// at fill 0.53-0.63 the 128 x 128 kernel was fastest (FP16 6784 x 2432 x
// 4096: 161.9 against 226.4 us one-wave-per-SIMD, 216.3 8-wave; 4700 x 4300
// x 6144: 307.7 against 388.4 and 380.2), from 0.66 on the 256 x 256 ones
// (3700 x 5900 x 4096: 277.0 and 270.1 against 290.0); with
// K < 4096 the 8-wave kernel beat the one-wave-per-SIMD one at every shape
// (FP16 7040 x 7168 x 2048: 264.4 against 311.1; 1800 x 7000 x 2048: 69.6
// against 76.4; INT8 12000 x 3000 x 2048: 122.6 against 136.0); from K =
// 4096 they were within 7% of each other either way. The whole-tile
// kernels (this one, and for INT4 the FP6 pre-pass one) are taken from 144
// tiles (56% of the CUs) up, the INT4 in-GEMM-conversion one from 192: at
// 2304^3 .. 3840^3 and {4096 x 2048, 2048 x 4096, 4096 x 2560} on MI355X
// the 128 x 128 eight-wave kernels win up to 128 tiles (FP16 2816^3: 59.7
// against 69.7 us) and lose from 144 on (3072^3: 84.6 against 74.1 us;
// 3840^3: 155.8 against 112.2 us); INT4 in-GEMM conversion against the
// 64-byte eight-wave kernel: 53.0 against 58.9 us at 169 tiles, 61.9
// against 68.9 at 196.
const Pref kPrefF16[] = {{V_WIDE, 144}, {V_PIPE256_W2X4, 144}, {V_SPREAD128W8, 1}, {V_SPREAD128W8_K64, 1},
                         {V_PIPE64, 1}};
const Pref kPrefS8[] = {{V_WIDE, 144}, {V_PIPE256_W2X4, 144}, {V_SPREAD128W8, 1}, {V_SPREAD128W8_K64, 1},
                        {V_PIPE64, 1}};
// INT4 on the 256 x 256 kernels (checked by int4_pref_ok): M and N must be
// multiples of 256 for the one-wave-per-SIMD FP6 kernel and for the in-GEMM
// E2M3 one (their edge tiles take the general epilogue), which the latter
// also needs at most one round of tiles or whole rounds (with K >= 4096) and
// K >= 2048; otherwise, with a workspace, the 8-wave FP6 kernel, and without
// one the 128 x 128 INT8-MFMA kernel (the 256 x 256 INT8-MFMA one only for
// whole tiles in whole rounds, where E2M3 cannot run: at 8192^3 415 against
// 543 us, on ragged shapes mostly slower than 128 x 128). Interleaved on MI355X at 2688 ..
// 8192 x 2432 .. 8192 x 2048 .. 8192 (44 shapes): with a workspace, on ragged
// shapes the 8-wave FP6 kernel beat the one-wave-per-SIMD one at all 11
// (1.02-1.17x); without, the E2M3 kernel was the slowest candidate at every
// ragged shape and at partial second rounds (4096 x 6144 x 4096: 142.1
// against 127.4 us for 128 x 128), ahead only in one round (4096^3: 71.9
// against 79.2 us) or whole rounds (8192 x 4096 x 4096: 151.1 against 173.3).
// The FP6 kernels' gain over 128 x 128 grows with K (whole tiles in one round:
// 1.12x at K = 2048, 1.37x at 4096, 1.58x at 8192), so the partial last round
// they can afford does too: the one-wave-per-SIMD kernel needs K >= 3072 or
// 60% of the CU slots filled (4352 x 4096 x 2048, 272 tiles: 55.8 against
// 50.7 us), the 8-wave one on ragged shapes 75% from K = 3072, 60% from
// K = 8192 or three rounds (6784 x 2432 x 4096, 270 tiles: 94.3 against
// 77.2; 4300 x 4100 x 4096: 100.7 against 92.9; 7040 x 7168 x 2048, 784
// tiles: 124.5 against 132.6).
const Pref kPrefS4[] = {{V_I4WIDE, 192}, {V_STAGED256_W2X4, 256}, {V_SPREAD128W8_K64, 1}, {V_PIPE64, 1}};
const Pref kPrefS4Ws[] = {{V_FP6_WIDE, 144}, {V_FP6_256_S2, 144}, {V_I4WIDE, 192}, {V_STAGED256_W2X4, 256},
                          {V_SPREAD128W8_K64, 1}, {V_PIPE64, 1}};

// Streaming kernel for problems with a small side (LLM decoding), against the
// narrow tiles below (measured on MI355X at 1..32 x {4096, 8192, 14336,
// 28672} x {4096, 8192, 14336}). It is the faster one while its workgroups
// stay few and long: up to 7 rows (FP16, INT8) with a large side of at most
// 8192, 16 rows with at most 4096, 32 rows for INT4; with a larger large
// side only when the large operand is small (at most 32 MiB: INT4 at
// 14336 x 4096) or each wave has at least 32 K-steps (FP16 at K = 16384).
// Up to 3.7x faster than the 128x128 split-K kernel, 1.1-1.6x faster than
// the narrow tiles where taken, at most 1.13x slower elsewhere in its range.
// The large side is split into groups of 16 rows per workgroup, or 32 when a
// wave has at most 8 K-steps of 64 bytes or the small side needs two 16-row
// blocks; with exactly 8 K-steps per wave, one 8-step prefetch group
// (skinny16x32_k64_d8) is 1.3-1.4x faster than two 4-step ones. Negative:
// not taken. From 8 rows at 8192 x 8192 the narrow 32 x 64 tile with the
// eight-slice ring is faster (FP16 25.1 against 26.9 us, INT8 15.0 against
// 15.8; at 6 rows 25.2 against 25.0 and 15.0 against 14.8).
int select_skinny(int dtype, int M, int N, int K, const void *A, const void *B, const void *C) {
    const int small = M < N ? M : N, large = M < N ? N : M;
    const int most = dtype == S4 ? 32 : (large <= 4096 ? 16 : 7);
    if (small > most || large < 1024) return -1;
    const long steps_per_wave = row_bytes(dtype, K) / 64 / SKINNY_WAVES;
    if (large > 8192 && (long)large * row_bytes(dtype, K) > (32l << 20) && steps_per_wave < 32) return -1;
    int v;
    if (small > 16) v = V_SKINNY + 3;                               // 32x32
    else if (steps_per_wave == 8) v = V_SKINNY16_D8;
    else v = V_SKINNY + (steps_per_wave < 8 ? 1 : 0);               // 16x32 or 16x16
    return supports(dtype, table(dtype)[v], M, N, K, A, B, C) ? v : -1;
}

// Narrow tiles for the problems `narrow_shape` admits (LLM prefill, batched
// decoding, and problems whose 128 x 128 tiles would leave CUs idle) where
// the streaming kernel is not taken: 32 x 64, 32 x 128 (up to 256 rows on
// the small side), 64 x 64 (FP16 up to 256 rows) or 64 x 128 tiles (small
// side first; the last two with four and eight waves of 32 x 32), and above
// 64 rows also the eight-wave 128 x 128 kernel (split by the same rule, which
// splits nothing above 256 rows).
// These problems stream the operands through LDS at a per-CU rate that
// varies little between the tiles, so the choice minimises the bytes one CU
// copies: (tile rows of both operands) x (K range of a workgroup) x (rounds
// of 256 workgroups). Within 10% of the minimum, long rows (at least 12 KiB)
// take the largest tile (fewer, longer workgroups amortise the per-slice
// overhead) and short rows the most workgroups. Measured on MI355X at
// 1..256 x {4096, 8192, 11008, 14336, 28672} x {2048 .. 14336} against the
// 128x128 split-K kernel: FP16 1.1-1.7x, INT8 1.1-1.5x, INT4 1.1-1.5x faster.
// With the 64 x 64 and eight-wave tiles the pick is within 1.5% of the
// fastest kernel measured (every candidate at 1, 2 and 4 K-ranges) on
// average over 30 LLM shapes, at most 1.13x (INT8 256 x 4096 x 14336),
// against 10% on average for the three-tile set before (FP16 256 x 4096 x
// 14336: 72.4 -> 53.9 us; INT8 128 x 28672 x 8192: 58.2 -> 46.9 us).
// Where K is long and one round of workgroups holds the tiles, the same
// tiles with an eight-slice ring, unsplit, take over (below): FP16 16 x
// 8192 x 8192 27.1 -> 24.9 us, 128 x 8192 x 8192 36.7 -> 30.1 us; INT8
// 16 x 8192 x 8192 17.1 -> 15.2 us. From 257 to 512 rows (the eight-wave
// 128 x 128 kernel alone before) at 320, 384, 512 x 2048 .. 14336 x 2048 ..
// 8192 and two mirrored shapes: FP16 1.12x, INT8 1.15x, INT4 1.21x faster
// (geometric means; up to 1.32x, 1.49x, 1.78x; slower nowhere), the pick
// within 1.5% of the fastest kernel timed on average. Negative: not taken.
int select_narrow(int dtype, int M, int N, int K, const void *A, const void *B, const void *C) {
    const int small = M < N ? M : N;
    if (!narrow_shape(M, N)) return -1;
    const Variant *t = table(dtype);
    const long kb = row_bytes(dtype, K);
    int cands[5], nc = 0;
    const int mir = M <= N ? 0 : 3;
    if (small <= 256) {  // 32-row tiles: too little work per wave above that
        cands[nc++] = V_NARROW + mir;                   // 32 x 64 (64 x 32)
        cands[nc++] = V_NARROW + 1 + mir;               // 32 x 128 (128 x 32)
    }
    // 64 x 64 (four waves); FP16 above 256 rows does as well or better with
    // the eight-wave 64 x 128 (512 x 512 x 8192: 19.7 against 25.4 us)
    if (dtype != F16 || small <= 256) cands[nc++] = V_NARROW64;
    cands[nc++] = V_NARROW64W8 + (M <= N ? 0 : 1);      // 64 x 128 (128 x 64), eight waves
    if (small > 64) cands[nc++] = spread128w8(dtype);   // 128 x 128, eight waves
    int best = -1;
    double best_cost = 0, costs[5];
    long wgs[5];
    for (int i = 0; i < nc; ++i) {
        const Variant &v = t[cands[i]];
        costs[i] = -1;
        if (!supports(dtype, v, M, N, K, A, B, C)) continue;
        const int sp = choose_splits(dtype, v, M, N, K);
        wgs[i] = tile_count(v, M, N) * sp;
        costs[i] = (double)((wgs[i] + 255) / 256) * (v.bm + v.bn) * kb / sp;
        if (best < 0 || costs[i] < best_cost) best = i, best_cost = costs[i];
    }
    if (best < 0) return -1;
    for (int i = 0; i < nc; ++i) {
        if (costs[i] < 0 || costs[i] > 1.1 * best_cost || i == best) continue;
        const Variant &v = t[cands[i]], &b = t[cands[best]];
        const bool bigger = (long)v.bm * v.bn > (long)b.bm * b.bn;
        if (kb >= 12288 ? bigger : (wgs[i] > wgs[best] || (wgs[i] == wgs[best] && bigger))) best = i;
    }
    // The eight-slice ring, unsplit, one workgroup per CU (96 to 160 KiB of
    // LDS) in a single round: the same tile streams its rows 1.1-1.3x faster
    // than through the four-slice ring at 16 ... 128 x 8192 x 8192 (FP16,
    // INT8), so its cost is scaled by 0.7 against the four-slice candidates,
    // split or not. Measured on MI355X, up to 128 rows on the small side it
    // gains with at least 64 slices of K and 128 to 256 workgroups, and with
    // more than 192 only from 128 slices on (224 tiles at 14336 x 4096: 4-6%
    // slower); never where its tiles need more than one round (256 x 8192:
    // they copy twice the bytes of 128 x 128 ones); INT4, with its nibble
    // unpacking, gained at no measured shape.
    // Above 128 rows they gain wherever their tiles fit one round, from 32
    // slices: 64 x 64 at 900 x 900 x 8192 32.1 against 40.1 us for 64 x 128
    // (FP16), 18.6 against 20.3 for four-slice 64 x 64 (INT8); 1024 x 1024 x
    // 8192 32.9 against 41.0 (FP16); 32 x 64 at 700 x 700 x 8192 26.8
    // against 36.2; 160 x 4096 x 8192 29.5 against 38.5 for 128 x 128 split
    // in two (FP16); 192 x 2048 x 4096 INT8 9.9 against 13.9. With more
    // tiles (1100 x 1300, 384 .. 1200 x 1200 .. 4096) they lose.
    int deep = -1;
    double deep_cost = 0;
    const long slices = kb / 128;
    const bool wide_small = small > 128;
    if (dtype != S4 && ((small <= 128 && slices >= 64) || (wide_small && slices >= 32))) {
        const int dmir = M <= N ? 0 : 2;
        for (int cand : {V_DEEP + dmir, V_DEEP + 1 + dmir, V_DEEP + 4}) {
            const Variant &v = t[cand];
            const long tiles = tile_count(v, M, N);
            if (tiles < 128 || tiles > 256 || (!wide_small && tiles > 192 && slices < 128) ||
                !supports(dtype, v, M, N, K, A, B, C))
                continue;
            // above 128 rows the four-slice candidates' split-K costs its
            // fix-up too: scaled by 0.5 (192 x 2048 x 4096: 15.0 against
            // 19.2 us for 128 x 128 split in four, whose cost is lower at 0.7)
            const double c = (wide_small ? 0.5 : 0.7) * (v.bm + v.bn) * kb;
            if (deep < 0 || c < deep_cost) deep = cand, deep_cost = c;
        }
    }
    if (deep >= 0 && deep_cost < best_cost) return deep;
    return cands[best];
}

// The conditions of the INT4 256 x 256 preferences (see kPrefS4).
bool int4_pref_ok(int variant, int M, int N, int K) {
    const bool whole = M % 256 == 0 && N % 256 == 0;
    const long tiles = (long)((M + 255) / 256) * ((N + 255) / 256);
    // share of the CU slots the rounds of 256 x 256 tiles keep busy
    const double fill = (double)tiles / (double)(((tiles + 255) / 256) * 256);
    if (variant == V_FP6_WIDE) return whole && (K >= 3072 || fill >= 0.6);
    if (variant == V_FP6_256_S2) return tiles >= 768 || (K >= 3072 && fill >= 0.75) || (K >= 8192 && fill >= 0.6);
    if (variant == V_I4WIDE) return whole && K >= 2048 && (tiles <= 256 || (tiles % 256 == 0 && K >= 4096));
    if (variant == V_STAGED256_W2X4) return whole && tiles % 256 == 0;
    return true;
}

// The conditions of the FP16 and INT8 256 x 256 preferences where M or N is
// not a multiple of 256 (see kPrefF16).
bool ragged_pref_ok(int variant, int M, int N, int K) {
    if ((M % 256 == 0 && N % 256 == 0) || (variant != V_WIDE && variant != V_PIPE256_W2X4)) return true;
    const long tiles = (long)((M + 255) / 256) * ((N + 255) / 256);
    const double fill = (double)tiles / (double)(((tiles + 255) / 256) * 256);
    if (fill < 0.65) return false;
    return variant != V_WIDE || K >= 4096;
}

// with_ws: the choice for a call that has a workspace (INT4 may then take
// the FP6 kernels fed by the conversion pre-pass).
int select_variant(int dtype, int M, int N, int K, const void *A, const void *B, const void *C,
                   bool with_ws = false) {
    const Variant *t = table(dtype);
    const int sk = select_skinny(dtype, M, N, K, A, B, C);
    if (sk >= 0) return sk;
    // FP16 with a workspace, 96 to 143 tiles of 256 x 256 and at least 128
    // K-slices: the one-wave-per-SIMD kernel under its stream-K schedule
    // (each tile in parts, so every CU has work) beats the eight-wave
    // 128 x 128 kernel the preferences give below 144 tiles: 768 x 8192 x
    // 8192 126.2 against 142.1 us, 1024 x 8192 x 8192 150.5 against 155.6 (its
    // own stream-K twin), 2560 x 2560 x 8192 127.2 against 135.8; with 64
    // tiles, fewer slices or INT8 it does not. Checked before the narrow
    // tiles, which would take 128 x 128 at 768 and 1024 x 8192 x 8192.
    if (dtype == F16 && with_ws && (M < N ? M : N) > 512) {
        const Variant &w = t[V_WIDE_SK];
        const long wt = tile_count(w, M, N);
        if (wt >= 96 && wt < 144 && row_bytes(dtype, K) / w.bkb >= 128 && supports(dtype, w, M, N, K, A, B, C) &&
            sk_plan(dtype, w, M, N, K).on)
            return V_WIDE_SK;
    }
    const int nv = select_narrow(dtype, M, N, K, A, B, C);
    if (nv >= 0) return nv;
    // Skinny problems (M or N at most 128: LLM-inference shapes) are bound by
    // streaming the large operand from HBM; the 4-wave 128x128 pipelined
    // kernel with split-K keeps every CU streaming, and the padding rows it
    // computes cost MFMA time only.
    if (M <= 128 || N <= 128) {
        for (int cand : {V_SPREAD128_K128, V_SPREAD128_K64})
            if (supports(dtype, t[cand], M, N, K, A, B, C)) return cand;
    }
    const bool s4ws = dtype == S4 && with_ws;
    const Pref *prefs = dtype == F16 ? kPrefF16 : (dtype == S8 ? kPrefS8 : (s4ws ? kPrefS4Ws : kPrefS4));
    const int n = dtype == F16 ? (int)(sizeof(kPrefF16) / sizeof(Pref))
                               : (dtype == S8 ? (int)(sizeof(kPrefS8) / sizeof(Pref))
                                              : (s4ws ? (int)(sizeof(kPrefS4Ws) / sizeof(Pref))
                                                      : (int)(sizeof(kPrefS4) / sizeof(Pref))));
    for (int i = 0; i < n; ++i) {
        const Variant &v = t[prefs[i].variant];
        if (!supports(dtype, v, M, N, K, A, B, C)) continue;
        if (dtype == S4 && !int4_pref_ok(prefs[i].variant, M, N, K)) continue;
        // (with a workspace, where the stream-K schedule splits the partial
        // last round, the fill of the rounds does not apply)
        // INT8 with K <= 2048 (at most 16 slices of 128 bytes) past one round
        // of 128 x 128 tiles: the 64-byte-slice kernel (twice the slices to
        // pipeline). Interleaved on MI355X at 14 shapes: 1.02-1.22x faster
        // with 384 .. 512 tiles (2304 x 3456 x 2048: 29.3 against 35.7 us),
        // 0.965-0.996x with 144 .. 256 tiles or K = 3072, 4096.
        if (dtype == S8 && prefs[i].variant == V_SPREAD128W8 && K <= 2048 && tile_count(v, M, N) > 256) continue;
        if (dtype != S4 && !ragged_pref_ok(prefs[i].variant, M, N, K)) {
            const int tw = sk_twin(prefs[i].variant);
            if (!(with_ws && tw >= 0 && supports(dtype, t[tw], M, N, K, A, B, C) && sk_plan(dtype, t[tw], M, N, K).on &&
                  (prefs[i].variant != V_WIDE || K >= 4096)))
                continue;
        }
        const long tm = (M + v.bm - 1) / v.bm, tn = (N + v.bn - 1) / v.bn;
        // skip a tile that would mostly compute padding
        if (4 * (long)M * N < 3 * tm * v.bm * tn * v.bn && i + 1 < n) continue;
        if (tm * tn * choose_splits(dtype, v, M, N, K) >= prefs[i].min_tiles) {
            // with a workspace, the stream-K schedule of the same kernel where
            // its plan is on
            const int twin = sk_twin(prefs[i].variant);
            if (with_ws && twin >= 0 && supports(dtype, t[twin], M, N, K, A, B, C) &&
                sk_plan(dtype, t[twin], M, N, K).on)
                return twin;
            return prefs[i].variant;
        }
    }
    return 0;
}

// Caller workspace. Layout: [0, 64 KiB) the split-K and stream-K tile
// counters (zero before the first such call on a workspace; every call
// leaves the counters it used zero again), then the zero-point row sums
// (4 (M + N) bytes), then the split-K partial tiles, or the FP6 operand
// copies followed by the stream-K partial tiles (either may be absent);
// every part 256-byte aligned. A problem that needs no scratch needs no
// workspace.
constexpr size_t kWsAlign = 256;

size_t align_up(size_t x) { return (x + kWsAlign - 1) / kWsAlign * kWsAlign; }

struct WsPlan {
    size_t sums_off, data_off, total;  // total 0: no workspace needed
};

// Offset of the stream-K partial tiles in the data part: after the FP6
// operand copies for the FP6 kernels (which need those copies stream-K or
// not), at its start for the others.
size_t sk_partials_off(const Variant &v, int M, int N, int K) {
    if (v.kind != FP6 && v.kind != FP6WIDE && v.kind != FP6WIDE_SK) return 0;
    return align_up(F6Geom::bytes(M, K) + F6Geom::bytes(N, K));
}

WsPlan ws_plan(const Variant &v, int splits, int M, int N, int K, bool zero_points, const SkPlan &sk) {
    const size_t sums = zero_points ? align_up(((size_t)M + N) * 4) : 0;
    size_t data = 0;
    if (splits > 1) {
        data = (size_t)tile_count(v, M, N) * splits * v.bm * v.bn * 4;
    } else {
        data = sk_partials_off(v, M, N, K);
        if (sk.on) data += (size_t)(sk.grid - sk.dp_tiles) * v.bm * v.bn * 4;  // one slot per remainder part
    }
    if (!sums && !data) return WsPlan{0, 0, 0};
    return WsPlan{kSplitCounterBytes, kSplitCounterBytes + sums, kSplitCounterBytes + sums + data};
}

struct Ws {
    uint8_t *p;    // caller's device workspace, or null
    size_t bytes;  // its size (0 without one)
};

// INT4 on the FP6 matrix cores fed by the conversion pre-pass: convert both
// operands into the workspace's data part w, then run the FP6 tile kernel
// (the stream-K one with its counters and partial tiles: counters, and the
// data part past the operand copies).
hipError_t launch_fp6(const Variant &v, const SkPlan &sk, int M, int N, int K, const uint8_t *A,
                      const uint8_t *B, void *C, EpiParams epi, uint8_t *w, int *counters,
                      hipStream_t stream) {
    const long Ma = F6Geom::rows_pad(M), Nb = F6Geom::rows_pad(N), runs = F6Geom::runs_pad(K);
    const uint64_t a_bytes = F6Geom::bytes(M, K);
    F6Prep pa{A, w, w + (size_t)Ma * runs * 16, M, (int)Ma, K, (int)runs};
    F6Prep pb{B, w + a_bytes, w + a_bytes + (size_t)Nb * runs * 16, N, (int)Nb, K, (int)runs};
    hipError_t e;
    {
        void *args[] = {&pa, &pb};
        dim3 grid((unsigned)((runs + F6_PREP_RUNS - 1) / F6_PREP_RUNS),
                  (unsigned)((Ma > Nb ? Ma : Nb) / F6_PREP_ROWS), 2);
        e = hipLaunchKernel(reinterpret_cast<const void *>(&s4_to_e3m2), grid, dim3(256), args, 0, stream);
    }
    if (e == hipSuccess) {
        const uint8_t *ap = pa.p, *aq = pa.q, *bp = pb.p, *bq = pb.q;
        int32_t *c = static_cast<int32_t *>(C);
        int ma = (int)Ma, nb = (int)Nb, kt = (int)(runs / v.bkb);
        int tiles_m = (M + v.bm - 1) / v.bm, tiles_n = (N + v.bn - 1) / v.bn;
        // the one-wave-per-SIMD kernel's table entry stores raw sums of whole
        // tiles; ragged or scaled outputs take its shared-epilogue instantiation
        const void *fn = v.fn;
        if ((v.kind == FP6WIDE || v.kind == FP6WIDE_SK) && (epi.out != OUT_PLAIN || M % v.bm || N % v.bn))
            fn = v.fn_epi;
        if (v.kind == FP6WIDE_SK) {
            SkArgs sa{sk.dp_tiles, sk.parts, nullptr, nullptr};
            if (sk.on) {
                sa.counters = counters;
                sa.partials = reinterpret_cast<uint32_t *>(w + sk_partials_off(v, M, N, K));
            }
            void *args[] = {&ap, &aq, &bp, &bq, &c, &M, &N, &ma, &nb, &kt, &tiles_m, &tiles_n, &sa, &epi};
            e = hipLaunchKernel(fn, dim3(sk.grid), dim3(v.threads), args, 0, stream);
        } else {
            void *args[] = {&ap, &aq, &bp, &bq, &c, &M, &N, &ma, &nb, &kt, &tiles_m, &tiles_n, &epi};
            e = hipLaunchKernel(fn, dim3(tiles_m * tiles_n), dim3(v.threads), args, 0, stream);
        }
    }
    return e;
}

hipError_t launch(int dtype, const Variant &v, int splits, const SkPlan &sk, int M, int N, int K, const void *A,
                  const void *B, void *C, EpiParams epi, const WsPlan &plan, Ws ws, hipStream_t stream) {
    const uint8_t *a = static_cast<const uint8_t *>(A);
    const uint8_t *b = static_cast<const uint8_t *>(B);
    if (v.kind == FP6 || v.kind == FP6WIDE || v.kind == FP6WIDE_SK)
        return launch_fp6(v, sk, M, N, K, a, b, C, epi, ws.p + plan.data_off, reinterpret_cast<int *>(ws.p),
                          stream);
    if (v.kind == SKINNY) {
        // X = the operand with at most bm rows (A when M is small), W = the other
        int trans = M <= v.bm ? 0 : 1;
        const uint8_t *x = trans ? b : a, *w = trans ? a : b;
        int R = trans ? N : M, Q = trans ? M : N, kb = (int)row_bytes(dtype, K), ldc = N;
        void *args[] = {&x, &w, &C, &R, &Q, &kb, &ldc, &trans, &epi};
        return hipLaunchKernel(v.fn, dim3((Q + v.bn - 1) / v.bn), dim3(v.threads), args, 0, stream);
    }
    if (v.kind == GENERIC) {
        int tiles_n = (N + 31) / 32;
        int tiles = ((M + 31) / 32) * tiles_n;
        void *args[] = {&a, &b, &C, &M, &N, &K, &tiles_n, &epi};
        return hipLaunchKernel(v.fn, dim3(tiles), dim3(v.threads), args, 0, stream);
    }
    int kb = (int)row_bytes(dtype, K);
    int tiles_m = (M + v.bm - 1) / v.bm, tiles_n = (N + v.bn - 1) / v.bn;
    if (is_sk(v)) {
        SkArgs sa{sk.dp_tiles, sk.parts, nullptr, nullptr};
        if (sk.on) {
            sa.counters = reinterpret_cast<int *>(ws.p);
            sa.partials = reinterpret_cast<uint32_t *>(ws.p + plan.data_off);
        }
        // the one-wave-per-SIMD kernel's raw-sum instantiation stores whole
        // tiles; scaled outputs and ragged edges take its shared epilogue
        const void *fn =
            (v.kind == WIDE_SK && (epi.out != OUT_PLAIN || M % v.bm || N % v.bn)) ? v.fn_epi : v.fn;
        void *args[] = {&a, &b, &C, &M, &N, &kb, &tiles_m, &tiles_n, &sa, &epi};
        return hipLaunchKernel(fn, dim3(sk.grid), dim3(v.threads), args, 0, stream);
    }
    if (!v.splitk) {
        const void *fn = v.fn;
        // the one-wave-per-SIMD kernels' table entries store raw sums of whole
        // tiles; scaled outputs and ragged edges take their instantiation with
        // the shared epilogue
        if (v.kind == WIDE && (epi.out != OUT_PLAIN || M % v.bm || N % v.bn)) fn = v.fn_epi;
        if (v.kind == I4WIDE && (epi.out != OUT_PLAIN || M % v.bm || N % v.bn)) fn = v.fn_epi;
        void *args[] = {&a, &b, &C, &M, &N, &kb, &tiles_m, &tiles_n, &epi};
        return hipLaunchKernel(fn, dim3(tiles_m * tiles_n), dim3(v.threads), args, 0, stream);
    }
    int *counters = nullptr;
    uint32_t *partials = nullptr;
    if (splits > 1) {
        counters = reinterpret_cast<int *>(ws.p);
        partials = reinterpret_cast<uint32_t *>(ws.p + plan.data_off);
    }
    void *args[] = {&a, &b, &C, &M, &N, &kb, &tiles_m, &tiles_n, &splits, &counters, &partials, &epi};
    return hipLaunchKernel(v.fn, dim3(tiles_m * tiles_n * splits), dim3(v.threads), args, 0, stream);
}

// Row sums for the zero-point terms into the workspace's sums part.
hipError_t zero_point_sums(int dtype, int M, int N, int K, const void *A, const void *B,
                           EpiParams &epi, int *sums, hipStream_t stream) {
    if (!epi.zero_a && !epi.zero_b) return hipSuccess;
    const void *fn = dtype == S8 ? reinterpret_cast<const void *>(&row_sums<S8>)
                                 : reinterpret_cast<const void *>(&row_sums<S4>);
    if (epi.zero_b) {  // needs the row sums of A
        const uint8_t *x = static_cast<const uint8_t *>(A);
        int r = M, k = K;
        int *out = sums;
        void *args[] = {&x, &r, &k, &out};
        const hipError_t e = hipLaunchKernel(fn, dim3(M), dim3(256), args, 0, stream);
        if (e != hipSuccess) return e;
        epi.sum_a = out;
    }
    if (epi.zero_a) {  // needs the column sums of B (rows of its N x K storage)
        const uint8_t *x = static_cast<const uint8_t *>(B);
        int r = N, k = K;
        int *out = sums + M;
        void *args[] = {&x, &r, &k, &out};
        const hipError_t e = hipLaunchKernel(fn, dim3(N), dim3(256), args, 0, stream);
        if (e != hipSuccess) return e;
        epi.sum_b = out;
    }
    return hipSuccess;
}

EpiParams plain_epilogue(int K) { return EpiParams{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, K, OUT_PLAIN}; }

// Scaled-output arguments: a known output type; zero points only for integer
// inputs; scale and zero-point vectors 4-byte aligned.
bool valid_epilogue(int dtype, const mpgemm_epilogue *e) {
    if (!e) return false;
    if (e->out_type != MPGEMM_OUT_F32 && e->out_type != MPGEMM_OUT_F16 && e->out_type != MPGEMM_OUT_BF16)
        return false;
    if (dtype == F16 && (e->zero_a || e->zero_b)) return false;
    for (const void *p : {(const void *)e->scale_a, (const void *)e->scale_b, (const void *)e->zero_a,
                          (const void *)e->zero_b})
        if (p && !aligned(p, 4)) return false;
    return true;
}

// The kernel choice of a call: variant (< 0: the automatic selection) and
// splits (< 0: the automatic choice, which splits only when the workspace
// holds the split's scratch), validated; the workspace plan of that choice.
struct Choice {
    int variant, splits;
    SkPlan sk;
    WsPlan plan;
};

hipError_t choose(int dtype, int variant, int splits, int M, int N, int K, const void *A, const void *B,
                  const void *C, bool zero_points, size_t ws_bytes, Choice &out) {
    const Variant *t = table(dtype);
    if (variant < 0) {
        // the choice with a workspace where it holds that choice's scratch
        // (the FP6 pre-pass operands; split K is decided below), else the
        // choice without one
        variant = select_variant(dtype, M, N, K, A, B, C, ws_bytes > 0);
        const Variant &v = t[variant];
        if (ws_plan(v, 1, M, N, K, zero_points, sk_plan(dtype, v, M, N, K)).total > ws_bytes) {
            // a stream-K twin whose partial tiles do not fit: its own kernel
            // with whole tiles where that fits (the FP6 one still needs its
            // operand copies), else the choice without a workspace
            const int base = sk_base(variant);
            const Variant *b = base >= 0 ? &t[base] : nullptr;
            if (b && ws_plan(*b, 1, M, N, K, zero_points, sk_off(tile_count(*b, M, N))).total <= ws_bytes)
                variant = base;
            else
                variant = select_variant(dtype, M, N, K, A, B, C, false);
        }
    }
    if (variant >= num_variants(dtype)) return hipErrorInvalidValue;
    const Variant &v = t[variant];
    if (!supports(dtype, v, M, N, K, A, B, C)) return hipErrorInvalidValue;
    if (splits < 0) {
        splits = choose_splits(dtype, v, M, N, K);
        if (splits > 1 && ws_plan(v, splits, M, N, K, zero_points, SkPlan{}).total > ws_bytes) splits = 1;
    }
    if (!splits_ok(dtype, v, M, N, K, splits)) return hipErrorInvalidValue;
    // a stream-K variant without room for its partial tiles runs every tile whole
    SkPlan sk = sk_plan(dtype, v, M, N, K);
    if (sk.on && ws_plan(v, splits, M, N, K, zero_points, sk).total > ws_bytes) sk = sk_off(tile_count(v, M, N));
    out = Choice{variant, splits, sk, ws_plan(v, splits, M, N, K, zero_points, sk)};
    return hipSuccess;
}

// variant < 0: the selection; splits < 0: the automatic choice for the variant.
hipError_t run(int dtype, int variant, int splits, int M, int N, int K, const void *A, const void *B, void *C,
               hipStream_t stream, const mpgemm_epilogue *scaled, Ws ws) {
    int c_elem = 4;
    if (scaled) {
        if (dtype < F16 || dtype > S4 || !valid_epilogue(dtype, scaled)) return hipErrorInvalidValue;
        c_elem = scaled->out_type == MPGEMM_OUT_F32 ? 4 : 2;
    }
    if (!valid_args(dtype, M, N, K, A, B, C, c_elem)) return hipErrorInvalidValue;
    if (!ws.p) ws.bytes = 0;
    if (ws.bytes && !aligned(ws.p, kWsAlign)) return hipErrorInvalidValue;
    if (M == 0 || N == 0) return hipSuccess;
    if (ws.bytes) {
        // the workspace must not overlap the operands or the output
        const uint64_t rb = (uint64_t)row_bytes(dtype, K);
        if (uintptr_t(-1) - reinterpret_cast<uintptr_t>(ws.p) < ws.bytes) return hipErrorInvalidValue;
        if (overlap(ws.p, ws.bytes, C, (uint64_t)M * (uint64_t)N * (uint64_t)c_elem) ||
            (K > 0 && (overlap(ws.p, ws.bytes, A, (uint64_t)M * rb) || overlap(ws.p, ws.bytes, B, (uint64_t)N * rb))))
            return hipErrorInvalidValue;
    }
    const bool zp = scaled && (scaled->zero_a || scaled->zero_b);
    Choice ch;
    hipError_t e = choose(dtype, variant, splits, M, N, K, A, B, C, zp, ws.bytes, ch);
    if (e != hipSuccess) return e;
    if (ch.plan.total > ws.bytes) return hipErrorInvalidValue;  // scratch needed, no (large enough) workspace
    EpiParams epi = plain_epilogue(K);
    if (scaled) {
        epi.scale_a = scaled->scale_a;
        epi.scale_b = scaled->scale_b;
        epi.zero_a = scaled->zero_a;
        epi.zero_b = scaled->zero_b;
        epi.out = scaled->out_type;
        e = zero_point_sums(dtype, M, N, K, A, B, epi, reinterpret_cast<int *>(ws.p + ch.plan.sums_off), stream);
        if (e != hipSuccess) return e;
    }
    return launch(dtype, table(dtype)[ch.variant], ch.splits, ch.sk, M, N, K, A, B, C, epi, ch.plan, ws, stream);
}

// ---- scratch for callers that cannot allocate (mpgemm_gemm_noalloc) ----
// A file-scope device array: each GPU the library runs on holds its own copy
// until the process ends. Host code must not use the name as an address (it
// is a host-side stand-in): the device address comes from
// hipGetSymbolAddress, once per device, with that device current.
constexpr size_t kStaticScratchBytes = (size_t)32 << 20;
static_assert(kStaticScratchBytes % kWsAlign == 0, "whole workspace granules");
__device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

hipError_t static_scratch(uint8_t **out) {
    static std::mutex mu;
    static uint8_t *ptr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        ptr[dev] = static_cast<uint8_t *>(p);
    }
    *out = ptr[dev];
    return hipSuccess;
}

// Fill kernel for the counter block of a reused scratch (a kernel rather than
// hipMemsetAsync, so the call can also be recorded into a graph).
__global__ void zero_words(uint32_t *p, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

}  // namespace

extern "C" {

hipError_t mpgemm_gemm_bt(int dtype, int M, int N, int K, const void *A, const void *B, void *C,
                          hipStream_t stream) {
    if (dtype != F16 && dtype != S8 && dtype != S4) return hipErrorInvalidValue;
    // the size, pointer and overlap checks of the plain entry points (B
    // occupies K * N elements either way)
    if (!valid_args(dtype, M, N, K, A, B, C)) return hipErrorInvalidValue;
    if (M == 0 || N == 0) return hipSuccess;
    if (K == 0) return run(dtype, -1, -1, M, N, K, A, B, C, stream, nullptr, Ws{nullptr, 0});  // zero fill
    typedef TileCfg<256, 256, 2, 4, 128, 2, 4> T;
    const long kb = row_bytes(dtype, K);
    if (N % T::BN || kb % T::BKB || !aligned(A, 16) || !aligned(B, 16)) return hipErrorInvalidValue;
    if (kb > INT_MAX || (long)K * N > (long)INT_MAX * 16) return hipErrorInvalidValue;
    if (dtype == S4 && K >= 131072) return hipErrorInvalidValue;  // INT4 sums carried times 256
    const uint8_t *a = static_cast<const uint8_t *>(A), *b = static_cast<const uint8_t *>(B);
    int kbi = (int)kb, tiles_m = (M + T::BM - 1) / T::BM, tiles_n = N / T::BN;
    EpiParams epi = plain_epilogue(K);
    void *args[] = {&a, &b, &C, &M, &N, &kbi, &tiles_m, &tiles_n, &epi};
    return hipLaunchKernel(tposeb_kernel(dtype), dim3(tiles_m * tiles_n), dim3(T::NTHREADS), args, 0,
                           stream);
}

hipError_t gemm_f16_f32(int M, int N, int K, const void *A, const void *B, float *C,
                        hipStream_t stream) {
    return run(F16, -1, -1, M, N, K, A, B, C, stream, nullptr, Ws{nullptr, 0});
}

hipError_t gemm_s8_s32(int M, int N, int K, const int8_t *A, const int8_t *B, int32_t *C,
                       hipStream_t stream) {
    return run(S8, -1, -1, M, N, K, A, B, C, stream, nullptr, Ws{nullptr, 0});
}

hipError_t gemm_s4_s32(int M, int N, int K, const uint8_t *A, const uint8_t *B, int32_t *C,
                       hipStream_t stream) {
    return run(S4, -1, -1, M, N, K, A, B, C, stream, nullptr, Ws{nullptr, 0});
}

hipError_t gemm_scaled(int dtype, int M, int N, int K, const void *A, const void *B, void *C,
                       const mpgemm_epilogue *epi, hipStream_t stream) {
    if (!epi) return hipErrorInvalidValue;
    return run(dtype, -1, -1, M, N, K, A, B, C, stream, epi, Ws{nullptr, 0});
}

hipError_t mpgemm_gemm_ws(int dtype, int M, int N, int K, const void *A, const void *B, void *C,
                          const mpgemm_epilogue *epi, void *workspace, size_t workspace_bytes,
                          hipStream_t stream) {
    return run(dtype, -1, -1, M, N, K, A, B, C, stream, epi,
               Ws{static_cast<uint8_t *>(workspace), workspace_bytes});
}

hipError_t mpgemm_workspace_size(int dtype, int variant, int splits, int M, int N, int K,
                                 const mpgemm_epilogue *epi, size_t *bytes) {
    if (!bytes || splits < 0) return hipErrorInvalidValue;
    int c_elem = 4;
    if (epi) {
        if (dtype < F16 || dtype > S4 || !valid_epilogue(dtype, epi)) return hipErrorInvalidValue;
        c_elem = epi->out_type == MPGEMM_OUT_F32 ? 4 : 2;
    }
    // sizes only: stand-in pointers, 256-byte aligned and far apart
    const void *A = reinterpret_cast<const void *>(uintptr_t(1) << 20);
    const void *B = reinterpret_cast<const void *>(uintptr_t(1) << 44);
    const void *C = reinterpret_cast<const void *>(uintptr_t(1) << 46);
    if (!valid_args(dtype, M, N, K, A, B, C, c_elem)) return hipErrorInvalidValue;
    *bytes = 0;
    if (M == 0 || N == 0) return hipSuccess;
    Choice ch;
    const bool zp = epi && (epi->zero_a || epi->zero_b);
    const hipError_t e = choose(dtype, variant, splits == 0 ? -1 : splits, M, N, K, A, B, C, zp, SIZE_MAX, ch);
    if (e != hipSuccess) return e;
    *bytes = ch.plan.total;
    return hipSuccess;
}

hipError_t mpgemm_gemm_noalloc(int dtype, int M, int N, int K, const void *A, const void *B, void *C,
                               const mpgemm_epilogue *epi, hipStream_t stream) {
    // the checks of mpgemm_gemm_ws first: nothing is looked up or enqueued
    // for arguments it would refuse
    int c_elem = 4;
    if (epi) {
        if (dtype < F16 || dtype > S4 || !valid_epilogue(dtype, epi)) return hipErrorInvalidValue;
        c_elem = epi->out_type == MPGEMM_OUT_F32 ? 4 : 2;
    }
    if (!valid_args(dtype, M, N, K, A, B, C, c_elem)) return hipErrorInvalidValue;
    if (M == 0 || N == 0) return hipSuccess;
    // the choice with a workspace of the scratch's size: a split that does
    // not fit is not taken; scratch the call cannot do without (zero points
    // beyond it) is refused
    Choice ch;
    const bool zp = epi && (epi->zero_a || epi->zero_b);
    hipError_t e = choose(dtype, -1, -1, M, N, K, A, B, C, zp, kStaticScratchBytes, ch);
    if (e != hipSuccess) return e;
    if (ch.plan.total > kStaticScratchBytes) return hipErrorInvalidValue;
    uint8_t *ws = nullptr;
    if (ch.plan.total) {
        e = static_scratch(&ws);
        if (e != hipSuccess) return e;
    }
    if (ch.splits > 1 || ch.sk.on) {
        // the array keeps the last call's contents: clear the tile counters
        uint32_t *words = reinterpret_cast<uint32_t *>(ws);
        int n = (int)tile_count(table(dtype)[ch.variant], M, N);
        void *args[] = {&words, &n};
        e = hipLaunchKernel(reinterpret_cast<const void *>(&zero_words), dim3((n + 255) / 256), dim3(256), args,
                            0, stream);
        if (e != hipSuccess) return e;
    }
    return run(dtype, ch.variant, ch.splits, M, N, K, A, B, C, stream, epi, Ws{ws, ch.plan.total ? kStaticScratchBytes : 0});
}

int mpgemm_num_variants(int dtype) { return num_variants(dtype); }

const char *mpgemm_variant_name(int dtype, int variant) {
    const Variant *t = table(dtype);
    if (!t || variant < 0 || variant >= num_variants(dtype)) return "";
    return t[variant].name;
}

int mpgemm_select_variant(int dtype, int M, int N, int K, const void *A, const void *B,
                          const void *C) {
    if (!valid_args(dtype, M, N, K, A, B, C)) return -1;
    return select_variant(dtype, M, N, K, A, B, C);
}

int mpgemm_select_variant_ws(int dtype, int M, int N, int K, const void *A, const void *B,
                             const void *C) {
    if (!valid_args(dtype, M, N, K, A, B, C)) return -1;
    return select_variant(dtype, M, N, K, A, B, C, true);
}

int mpgemm_variant_supports(int dtype, int variant, int M, int N, int K, const void *A,
                            const void *B, const void *C) {
    const Variant *t = table(dtype);
    if (!t) return -1;
    if (variant < 0 || variant >= num_variants(dtype)) return 0;
    if (!valid_args(dtype, M, N, K, A, B, C)) return 0;
    return supports(dtype, t[variant], M, N, K, A, B, C) ? 1 : 0;
}

hipError_t mpgemm_run_variant(int dtype, int variant, int M, int N, int K, const void *A,
                              const void *B, void *C, hipStream_t stream) {
    if (variant < 0) return hipErrorInvalidValue;
    return run(dtype, variant, -1, M, N, K, A, B, C, stream, nullptr, Ws{nullptr, 0});
}

hipError_t mpgemm_run_variant_ws(int dtype, int variant, int splits, int M, int N, int K, const void *A,
                                 const void *B, void *C, const mpgemm_epilogue *epi, void *workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
    if (variant < 0 || splits < 0) return hipErrorInvalidValue;
    return run(dtype, variant, splits == 0 ? -1 : splits, M, N, K, A, B, C, stream, epi,
               Ws{static_cast<uint8_t *>(workspace), workspace_bytes});
}

hipError_t mpgemm_sk_schedule(int dtype, int variant, int M, int N, int K, int *dp_tiles, int *parts,
                              int *grid) {
    const Variant *t = table(dtype);
    if (!t || variant < 0 || variant >= num_variants(dtype) || !dp_tiles || !parts || !grid)
        return hipErrorInvalidValue;
    if (M <= 0 || N <= 0 || K <= 0 || (dtype == S4 && (K & 1)) ||
        !supports(dtype, t[variant], M, N, K, nullptr, nullptr, nullptr))
        return hipErrorInvalidValue;
    const SkPlan sk = sk_plan(dtype, t[variant], M, N, K);
    *dp_tiles = sk.dp_tiles;
    *parts = sk.parts;
    *grid = sk.grid;
    return hipSuccess;
}

int mpgemm_select_splits(int dtype, int variant, int M, int N, int K) {
    const Variant *t = table(dtype);
    if (!t || variant < 0 || variant >= num_variants(dtype) || M < 0 || N < 0 || K < 0) return -1;
    if (dtype == S4 && (K & 1)) return -1;
    if (M == 0 || N == 0 || !supports(dtype, t[variant], M, N, K, nullptr, nullptr, nullptr))
        return 1;
    return choose_splits(dtype, t[variant], M, N, K);
}

void mpgemm_s4_run_to_fp6(const uint8_t *in, uint32_t *out) {
    uint32_t w[4] = {0, 0, 0, 0}, o[6];
    for (int e = 0; e < 16; ++e) w[e >> 2] |= (uint32_t)in[e] << (8 * (e & 3));
    s4_run_to_e3m2(w, o);
    for (int i = 0; i < 6; ++i) out[i] = o[i];
}

void mpgemm_s4_run_to_e2m3(const uint8_t *in, uint32_t *out) {
    uint32_t w[4] = {0, 0, 0, 0}, o[6];
    for (int e = 0; e < 16; ++e) w[e >> 2] |= (uint32_t)in[e] << (8 * (e & 3));
    s4_run_to_e2m3(w, o);
    for (int i = 0; i < 6; ++i) out[i] = o[i];
}

}  // extern "C"
