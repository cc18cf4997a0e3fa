// mpgemm.hip - the C-ABI entry points: argument checks, kernel choice, launch.
//
// Every entry point validates its arguments on the host, picks a kernel
// variant (a tiled kernel when the problem is tile-aligned and 16-byte
// aligned, the bounds-checked kernel otherwise) and launches it on the
// caller's stream with hipLaunchKernel, returning the launch status. Nothing
// here allocates, copies or synchronises.
#include <hip/hip_runtime.h>
#include <limits.h>
#include <stdint.h>

#include "mpgemm.h"
#include "generic_gemm.hpp"
#include "tiled_gemm.hpp"

using namespace mpg;

// Tile configurations (kernel template arguments need external linkage).
namespace mpg {
//                BM   BN  WGM WGN BKB STG GROUP_M
typedef TileCfg<256, 256, 2, 2, 128, 2, 4> T256x256_w4_s2;
typedef TileCfg<256, 256, 2, 4, 128, 2, 4> T256x256_w8_s2;
typedef TileCfg<256, 256, 4, 2, 128, 2, 4> T256x256_w8t_s2;
typedef TileCfg<256, 256, 4, 4, 128, 2, 4> T256x256_w16_s2;
typedef TileCfg<256, 256, 4, 2, 64, 4, 4> T256x256_w8t_k64_s4;
typedef TileCfg<256, 256, 4, 4, 64, 4, 4> T256x256_w16_k64_s4;
typedef TileCfg<256, 256, 2, 2, 64, 4, 4> T256x256_w4_k64_s4b;
typedef TileCfg<128, 128, 2, 2, 64, 4, 4> T128x128_w4_k64_s4;
typedef TileCfg<256, 256, 2, 2, 64, 2, 4> T256x256_w4_k64_s2;
typedef TileCfg<256, 256, 4, 2, 64, 2, 4> T256x256_w8t_k64_s2;
typedef TileCfg<128, 128, 2, 2, 128, 2, 4> T128x128_w4_k128_s2;
typedef TileCfg<256, 256, 2, 4, 64, 2, 4> T256x256_w8_k64_s2;
typedef TileCfg<128, 128, 2, 2, 128, 4, 4, 16> T128x128_w4_s4_m16;
typedef TileCfg<256, 256, 2, 2, 64, 4, 4> T256x256_w4_k64_s4;
typedef TileCfg<256, 128, 2, 2, 128, 3, 4> T256x128_w4_s3;
typedef TileCfg<128, 128, 2, 2, 128, 2, 4> T128x128_w4_s2;
typedef TileCfg<128, 128, 2, 2, 128, 4, 4> T128x128_w4_s4;
typedef TileCfg<64, 64, 1, 1, 128, 4, 4> T64x64_w1_s4;

}  // namespace mpg

namespace {

enum Kind { GENERIC = 0, TILED = 1 };

struct Variant {
    const char *name;
    int kind;
    int bm, bn, bkb;  // tile (TILED only)
    int threads;
    const void *fn;
};

typedef void (*kernel_fn)(const uint8_t *, const uint8_t *, void *, int, int, int, int, int);
typedef void (*generic_fn)(const uint8_t *, const uint8_t *, void *, int, int, int, int);

template <int DT, class T>
Variant tiled(const char *name) {
    kernel_fn f = &tiled_gemm<DT, T>;
    return Variant{name, TILED, T::BM, T::BN, T::BKB, T::NTHREADS, reinterpret_cast<const void *>(f)};
}

template <int DT, class T, bool SPREAD = false>
Variant pipelined(const char *name) {
    kernel_fn f = &tiled_gemm_pf<DT, T, SPREAD>;
    return Variant{name, TILED, T::BM, T::BN, T::BKB, T::NTHREADS, reinterpret_cast<const void *>(f)};
}

template <int DT, class T, int NSETS>
Variant staged(const char *name) {
    kernel_fn f = &tiled_gemm_rs<DT, T, NSETS>;
    return Variant{name, TILED, T::BM, T::BN, T::BKB, T::NTHREADS, reinterpret_cast<const void *>(f)};
}

template <int DT, class T, int LEFT>
Variant pingpong(const char *name) {
    kernel_fn f = &tiled_gemm_pp<DT, T, LEFT>;
    return Variant{name, TILED, T::BM, T::BN, T::BKB, T::NTHREADS, reinterpret_cast<const void *>(f)};
}

template <int DT>
Variant generic(const char *name) {
    generic_fn f = &generic_gemm<DT>;
    return Variant{name, GENERIC, 32, 32, 0, 64, reinterpret_cast<const void *>(f)};
}

#define VARIANT_LIST(DT)                                                   \
    {generic<DT>("generic_32x32"),                                         \
     tiled<DT, T256x256_w4_s2>("tile256x256_w2x2_k128_s2"),                \
     tiled<DT, T256x256_w8_s2>("tile256x256_w2x4_k128_s2"),                \
     tiled<DT, T256x256_w4_k64_s4>("tile256x256_w2x2_k64_s4"),             \
     tiled<DT, T256x128_w4_s3>("tile256x128_w2x2_k128_s3"),                \
     tiled<DT, T128x128_w4_s2>("tile128x128_w2x2_k128_s2"),                \
     tiled<DT, T128x128_w4_s4>("tile128x128_w2x2_k128_s4"),                \
     tiled<DT, T64x64_w1_s4>("tile64x64_w1x1_k128_s4"),                    \
     pipelined<DT, T256x256_w4_s2>("pipe256x256_w2x2_k128_s2"),            \
     pipelined<DT, T256x256_w8_s2>("pipe256x256_w2x4_k128_s2"),            \
     pipelined<DT, T256x256_w4_k64_s4>("pipe256x256_w2x2_k64_s4"),         \
     pipelined<DT, T256x128_w4_s3>("pipe256x128_w2x2_k128_s3"),            \
     pipelined<DT, T128x128_w4_s4>("pipe128x128_w2x2_k128_s4"),            \
     pipelined<DT, T64x64_w1_s4>("pipe64x64_w1x1_k128_s4"),                \
     pipelined<DT, T256x256_w8t_s2>("pipe256x256_w4x2_k128_s2"),           \
     pipelined<DT, T256x256_w16_s2>("pipe256x256_w4x4_k128_s2"),           \
     pipelined<DT, T256x256_w8t_k64_s4, true>("spread256x256_w4x2_k64_s4"), \
     pipelined<DT, T256x256_w8t_s2, true>("spread256x256_w4x2_k128_s2"),   \
     pipelined<DT, T256x256_w16_k64_s4, true>("spread256x256_w4x4_k64_s4"), \
     pipelined<DT, T256x256_w4_k64_s4b, true>("spread256x256_w2x2_k64_s4"), \
     pipelined<DT, T128x128_w4_s4, true>("spread128x128_w2x2_k128_s4"),    \
     pipelined<DT, T128x128_w4_k64_s4, true>("spread128x128_w2x2_k64_s4"), \
     staged<DT, T256x256_w4_s2, 2>("staged256x256_w2x2_k128_n2"),          \
     staged<DT, T256x256_w4_s2, 1>("staged256x256_w2x2_k128_n1"),          \
     staged<DT, T256x256_w8t_s2, 1>("staged256x256_w4x2_k128_n1"),         \
     staged<DT, T256x256_w8_s2, 1>("staged256x256_w2x4_k128_n1"),          \
     staged<DT, T256x256_w4_k64_s2, 2>("staged256x256_w2x2_k64_n2"),       \
     staged<DT, T256x256_w8t_k64_s2, 2>("staged256x256_w4x2_k64_n2"),      \
     staged<DT, T128x128_w4_k128_s2, 2>("staged128x128_w2x2_k128_n2"),     \
     pingpong<DT, T256x256_w8_s2, 4>("pingpong256x256_k128_c4"),          \
     pingpong<DT, T256x256_w8_s2, 2>("pingpong256x256_k128_c2"),          \
     pingpong<DT, T256x256_w8_s2, 6>("pingpong256x256_k128_c6"),          \
     pingpong<DT, T256x256_w8_k64_s2, 4>("pingpong256x256_k64_c4"),       \
     pipelined<DT, T128x128_w4_s4_m16, true>("spread128x128_w2x2_k128_s4_m16")}

const Variant kF16[] = VARIANT_LIST(F16);
const Variant kS8[] = VARIANT_LIST(S8);
const Variant kS4[] = VARIANT_LIST(S4);
constexpr int kNumVariants = sizeof(kF16) / sizeof(kF16[0]);
static_assert(sizeof(kS8) / sizeof(kS8[0]) == kNumVariants, "");
static_assert(sizeof(kS4) / sizeof(kS4[0]) == kNumVariants, "");

const Variant *table(int dtype) {
    switch (dtype) {
        case F16: return kF16;
        case S8: return kS8;
        case S4: return kS4;
        default: return nullptr;
    }
}

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// Byte ranges [p, p + n) and [q, q + m) intersect (empty ranges never do).
bool overlap(const void *p, uint64_t n, const void *q, uint64_t m) {
    if (n == 0 || m == 0) return false;
    const uintptr_t a = reinterpret_cast<uintptr_t>(p), b = reinterpret_cast<uintptr_t>(q);
    return a < b + m && b < a + n;
}

// Argument checks shared by every entry point (see the header's Errors).
bool valid_args(int dtype, int M, int N, int K, const void *A, const void *B, const void *C) {
    if (dtype < F16 || dtype > S4) return false;
    if (M < 0 || N < 0 || K < 0) return false;
    if (K > INT_MAX - 64) return false;
    if (dtype == S4 && (K & 1)) return false;
    if (M == 0 || N == 0) return true;
    if (!C || !aligned(C, 4)) return false;
    if (K > 0) {
        if (!A || !B) return false;
        if (dtype == F16 && (!aligned(A, 2) || !aligned(B, 2))) return false;
    }
    const uint64_t rb = (uint64_t)row_bytes(dtype, K);
    const uint64_t a_bytes = (uint64_t)M * rb, b_bytes = (uint64_t)N * rb;
    const uint64_t c_bytes = (uint64_t)M * (uint64_t)N * 4u;
    if (c_bytes / 4u / (uint64_t)N != (uint64_t)M) return false;
    if (uintptr_t(-1) - reinterpret_cast<uintptr_t>(C) < c_bytes) return false;
    if (K > 0 && (overlap(C, c_bytes, A, a_bytes) || overlap(C, c_bytes, B, b_bytes))) return false;
    // the bounds-checked kernel indexes tiles with a 32-bit grid
    const uint64_t tiles = ((uint64_t)M + 31) / 32 * (((uint64_t)N + 31) / 32);
    if (tiles > (uint64_t)INT_MAX) return false;
    return true;
}

bool supports(int dtype, const Variant &v, int M, int N, int K, const void *A, const void *B,
              const void *C) {
    if (v.kind == GENERIC) return true;
    if (M == 0 || N == 0 || K == 0) return false;
    const long kb = row_bytes(dtype, K);
    // edge tiles are predicated in M and N; K must fill whole slices
    if (kb % v.bkb) return false;
    if (!aligned(A, 16) || !aligned(B, 16) || !aligned(C, 4)) return false;
    // INT4 partial sums are carried scaled by 256 (see s4_lo_x16)
    if (dtype == S4 && K >= 131072) return false;
    if (kb > INT_MAX) return false;
    return true;
}

// Variant indices in the tables above that the selection uses.
enum : int {
    V_PIPE256_W2X4 = 9,      // pipe256x256_w2x4_k128_s2
    V_SPREAD128_K128 = 20,   // spread128x128_w2x2_k128_s4
    V_SPREAD128_K64 = 21,    // spread128x128_w2x2_k64_s4
    V_STAGED256_W2X4 = 25,   // staged256x256_w2x4_k128_n1
    V_PIPE64 = 13,           // pipe64x64_w1x1_k128_s4
};

// Preferred tiled variants per dtype, largest tile first; a candidate is
// taken when it supports the problem and yields at least `min_tiles`
// workgroups (256 = one per CU). Chosen from interleaved timings of every
// variant at N = 512 ... 8192 on MI355X.
struct Pref { int variant; long min_tiles; };
const Pref kPrefF16[] = {{V_PIPE256_W2X4, 256}, {V_SPREAD128_K128, 256}, {V_SPREAD128_K64, 1}, {V_PIPE64, 1}};
const Pref kPrefS8[] = {{V_PIPE256_W2X4, 256}, {V_SPREAD128_K128, 256}, {V_SPREAD128_K64, 1}, {V_PIPE64, 1}};
const Pref kPrefS4[] = {{V_STAGED256_W2X4, 256}, {V_SPREAD128_K128, 256}, {V_SPREAD128_K64, 1}, {V_PIPE64, 1}};

int select_variant(int dtype, int M, int N, int K, const void *A, const void *B, const void *C) {
    const Variant *t = table(dtype);
    const Pref *prefs = dtype == F16 ? kPrefF16 : (dtype == S8 ? kPrefS8 : kPrefS4);
    for (int i = 0; i < 4; ++i) {
        const Variant &v = t[prefs[i].variant];
        if (!supports(dtype, v, M, N, K, A, B, C)) continue;
        const long tm = (M + v.bm - 1) / v.bm, tn = (N + v.bn - 1) / v.bn;
        // skip a tile that would mostly compute padding
        if (4 * (long)M * N < 3 * tm * v.bm * tn * v.bn && i + 1 < 4) continue;
        if (tm * tn >= prefs[i].min_tiles) return prefs[i].variant;
    }
    return 0;
}

hipError_t launch(int dtype, const Variant &v, int M, int N, int K, const void *A, const void *B,
                  void *C, hipStream_t stream) {
    const uint8_t *a = static_cast<const uint8_t *>(A);
    const uint8_t *b = static_cast<const uint8_t *>(B);
    if (v.kind == GENERIC) {
        int tiles_n = (N + 31) / 32;
        int tiles = ((M + 31) / 32) * tiles_n;
        void *args[] = {&a, &b, &C, &M, &N, &K, &tiles_n};
        return hipLaunchKernel(v.fn, dim3(tiles), dim3(v.threads), args, 0, stream);
    }
    int kb = (int)row_bytes(dtype, K);
    int tiles_m = (M + v.bm - 1) / v.bm, tiles_n = (N + v.bn - 1) / v.bn;
    void *args[] = {&a, &b, &C, &M, &N, &kb, &tiles_m, &tiles_n};
    return hipLaunchKernel(v.fn, dim3(tiles_m * tiles_n), dim3(v.threads), args, 0, stream);
}

hipError_t run(int dtype, int variant, int M, int N, int K, const void *A, const void *B, void *C,
               hipStream_t stream) {
    if (!valid_args(dtype, M, N, K, A, B, C)) return hipErrorInvalidValue;
    if (M == 0 || N == 0) return hipSuccess;
    const Variant *t = table(dtype);
    if (variant < 0) variant = select_variant(dtype, M, N, K, A, B, C);
    if (variant >= kNumVariants) return hipErrorInvalidValue;
    if (!supports(dtype, t[variant], M, N, K, A, B, C)) return hipErrorInvalidValue;
    return launch(dtype, t[variant], M, N, K, A, B, C, stream);
}

}  // namespace

extern "C" {

hipError_t gemm_f16_f32(int M, int N, int K, const void *A, const void *B, float *C,
                        hipStream_t stream) {
    return run(F16, -1, M, N, K, A, B, C, stream);
}

hipError_t gemm_s8_s32(int M, int N, int K, const int8_t *A, const int8_t *B, int32_t *C,
                       hipStream_t stream) {
    return run(S8, -1, M, N, K, A, B, C, stream);
}

hipError_t gemm_s4_s32(int M, int N, int K, const uint8_t *A, const uint8_t *B, int32_t *C,
                       hipStream_t stream) {
    return run(S4, -1, M, N, K, A, B, C, stream);
}

int mpgemm_num_variants(int dtype) { return table(dtype) ? kNumVariants : -1; }

const char *mpgemm_variant_name(int dtype, int variant) {
    const Variant *t = table(dtype);
    if (!t || variant < 0 || variant >= kNumVariants) return "";
    return t[variant].name;
}

int mpgemm_select_variant(int dtype, int M, int N, int K, const void *A, const void *B,
                          const void *C) {
    if (!valid_args(dtype, M, N, K, A, B, C)) return -1;
    return select_variant(dtype, M, N, K, A, B, C);
}

int mpgemm_variant_supports(int dtype, int variant, int M, int N, int K, const void *A,
                            const void *B, const void *C) {
    const Variant *t = table(dtype);
    if (!t) return -1;
    if (variant < 0 || variant >= kNumVariants) return 0;
    if (!valid_args(dtype, M, N, K, A, B, C)) return 0;
    return supports(dtype, t[variant], M, N, K, A, B, C) ? 1 : 0;
}

hipError_t mpgemm_run_variant(int dtype, int variant, int M, int N, int K, const void *A,
                              const void *B, void *C, hipStream_t stream) {
    if (variant < 0) return hipErrorInvalidValue;
    return run(dtype, variant, M, N, K, A, B, C, stream);
}

}  // extern "C"
