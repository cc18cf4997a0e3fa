// variants.hpp - the kernel variant table: tile configurations, the record
// the host code launches from, and the list of variants every precision
// carries. Each precision's table is built in its own translation unit
// (variants_f16.hip, variants_s8.hip, variants_s4.hip) so the kernels of the
// three precisions compile in parallel; mpgemm.hip selects and launches.
#pragma once

#include <stdint.h>

#include "generic_gemm.hpp"
#include "tiled_gemm.hpp"
#include "f6_gemm.hpp"
#include "deep_gemm.hpp"
#include "skinny_gemm.hpp"
#include "wide_gemm.hpp"
#include "wide_f6.hpp"
#include "wide_i4.hpp"
#include "stream_k.hpp"

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
// eight waves of 64 x 32 on a 128 x 128 tile (mid sizes)
typedef TileCfg<128, 128, 2, 4, 128, 4, 4> T128x128_w8_s4;
typedef TileCfg<128, 128, 2, 4, 64, 4, 4> T128x128_w8_k64_s4;
typedef TileCfg<64, 64, 1, 1, 128, 4, 4> T64x64_w1_s4;
typedef TileCfg<256, 256, 2, 4, 64, 4, 4> T256x256_w8_k64_s4;
typedef TileCfg<256, 256, 2, 4, 64, 3, 4> T256x256_w8_k64_s3;
typedef TileCfg<256, 256, 2, 2, 64, 5, 4> T256x256_w4_k64_s5;
// narrow tiles for 17..256 rows on one side (A side first, then mirrored)
typedef TileCfg<32, 64, 1, 2, 128, 4, 4, 16> T32x64_w2_m16;
typedef TileCfg<32, 128, 1, 4, 128, 4, 4, 16> T32x128_w4_m16;
typedef TileCfg<64, 128, 2, 2, 128, 4, 4> T64x128_w4;
typedef TileCfg<64, 32, 2, 1, 128, 4, 4, 16> T64x32_w2_m16;
typedef TileCfg<128, 32, 4, 1, 128, 4, 4, 16> T128x32_w4_m16;
typedef TileCfg<128, 64, 2, 2, 128, 4, 4> T128x64_w4;
// more waves on the narrow tiles: 64 x 64 (four of 32 x 32, 16x16 MFMAs),
// 64 x 128 and its mirror (eight of 32 x 32)
typedef TileCfg<64, 64, 2, 2, 128, 4, 4, 16> T64x64_w4_m16;
typedef TileCfg<64, 128, 2, 4, 128, 4, 4> T64x128_w8;
typedef TileCfg<128, 64, 4, 2, 128, 4, 4> T128x64_w8;
// narrow tiles with an eight-slice ring (160 KiB of LDS for 32 x 128): the
// unsplit kernel keeps seven slices of its rows in flight, what split K
// bought the four-slice ring by running more workgroups
typedef TileCfg<32, 64, 1, 2, 128, 8, 4, 16> T32x64_w2_m16_s8;
typedef TileCfg<32, 128, 1, 4, 128, 8, 4, 16> T32x128_w4_m16_s8;
typedef TileCfg<64, 32, 2, 1, 128, 8, 4, 16> T64x32_w2_m16_s8;
typedef TileCfg<128, 32, 4, 1, 128, 8, 4, 16> T128x32_w4_m16_s8;
typedef TileCfg<64, 64, 2, 2, 128, 8, 4, 16> T64x64_w4_m16_s8;

//             BM   BN  WGM WGN  J STG GROUP_M    (J runs of 32 k per stage)
typedef F6Cfg<256, 256, 2, 4, 4, 3, 4> F6_256x256_w8_s3;
typedef F6Cfg<256, 256, 2, 4, 4, 2, 4> F6_256x256_w8_s2;
typedef F6Cfg<256, 256, 2, 2, 4, 3, 4> F6_256x256_w4_s3;
typedef F6Cfg<256, 256, 4, 2, 4, 3, 4> F6_256x256_w8t_s3;
typedef F6Cfg<256, 128, 2, 2, 4, 4, 4> F6_256x128_w4_s4;
typedef F6Cfg<128, 128, 2, 2, 4, 4, 4> F6_128x128_w4_s4;
typedef F6Cfg<128, 128, 2, 2, 4, 6, 4> F6_128x128_w4_s6;
typedef F6Cfg<128, 128, 2, 2, 8, 3, 4> F6_128x128_w4_k256_s3;

}  // namespace mpg

namespace mpg {

enum Kind { GENERIC = 0, TILED = 1, FP6 = 2, SKINNY = 3, WIDE = 4, FP6WIDE = 5, I4WIDE = 6, TILED_SK = 7, WIDE_SK = 8, FP6WIDE_SK = 9 };

struct Variant {
    const char *name;
    int kind;
    int bm, bn, bkb;  // tile; bkb: bytes per row per K-slice (TILED), runs per stage (FP6);
                      // SKINNY: bm = most rows of the small operand, bn = rows of the
                      // large one per workgroup, bkb = bytes per K-step
    int threads;
    const void *fn;
    bool splitk;      // kernel takes (splits, counters, partials): the pipelined kernels
    const void *fn_epi = nullptr;  // WIDE(_SK), FP6WIDE(_SK), I4WIDE: the instantiation with the
                                   // shared epilogue (ragged edges, scaled outputs); fn
                                   // stores raw sums of whole tiles
};

typedef void (*kernel_fn)(const uint8_t *, const uint8_t *, void *, int, int, int, int, int,
                          EpiParams);
typedef void (*splitk_fn)(const uint8_t *, const uint8_t *, void *, int, int, int, int, int, int,
                          int *, uint32_t *, EpiParams);
typedef void (*sk_fn)(const uint8_t *, const uint8_t *, void *, int, int, int, int, int, SkArgs,
                      EpiParams);
typedef void (*generic_fn)(const uint8_t *, const uint8_t *, void *, int, int, int, int,
                           EpiParams);

template <int DT, class T>
Variant tiled(const char *name) {
    kernel_fn f = &tiled_gemm<DT, T>;
    return Variant{name, TILED, T::BM, T::BN, T::BKB, T::NTHREADS, reinterpret_cast<const void *>(f),
                   false};
}

template <int DT, class T, bool SPREAD = false>
Variant pipelined(const char *name) {
    splitk_fn f = &tiled_gemm_pf<DT, T, SPREAD>;
    return Variant{name, TILED, T::BM, T::BN, T::BKB, T::NTHREADS, reinterpret_cast<const void *>(f),
                   true};
}

// Stream-K schedule of the pipelined kernel (stream_k.hpp).
template <int DT, class T, bool SPREAD>
Variant pipelined_sk(const char *name) {
    sk_fn f = &tiled_gemm_sk<DT, T, SPREAD>;
    return Variant{name, TILED_SK, T::BM, T::BN, T::BKB, T::NTHREADS, reinterpret_cast<const void *>(f),
                   false};
}

template <int DT, class T, int NSETS>
Variant staged(const char *name) {
    kernel_fn f = &tiled_gemm_rs<DT, T, NSETS>;
    return Variant{name, TILED, T::BM, T::BN, T::BKB, T::NTHREADS, reinterpret_cast<const void *>(f),
                   false};
}

template <int DT, class T, int LEFT>
Variant pingpong(const char *name) {
    kernel_fn f = &tiled_gemm_pp<DT, T, LEFT>;
    return Variant{name, TILED, T::BM, T::BN, T::BKB, T::NTHREADS, reinterpret_cast<const void *>(f),
                   false};
}

template <int DT, class T>
Variant deep(const char *name) {
    kernel_fn f = &tiled_gemm_deep<DT, T>;
    return Variant{name, TILED, T::BM, T::BN, T::BKB, T::NTHREADS, reinterpret_cast<const void *>(f),
                   false};
}

template <int DT, int MB, int NB, int D = SKINNY_DEPTH>
Variant skinny(const char *name) {
    typedef void (*skinny_fn)(const uint8_t *, const uint8_t *, void *, int, int, int, int, int,
                              EpiParams);
    skinny_fn f = &skinny_gemm<DT, MB, NB, D>;
    return Variant{name, SKINNY, 16 * MB, 16 * NB, 64, 64 * SKINNY_WAVES, reinterpret_cast<const void *>(f),
                   false};
}

// One wave per SIMD, 256 x 256 tiles only (wide_gemm.hpp); FP16 and INT8 (no
// kernel for INT4: fn is null and the variant supports nothing). AUX: cache
// policy of the copy loads.
template <int DT, int AUX = CP_DEFAULT>
Variant wide(const char *name) {
    const void *f = nullptr, *fe = nullptr;
    if constexpr (DT == F16 || DT == S8) {
        kernel_fn k = &wide_gemm<DT, true, AUX>, ke = &wide_gemm<DT, false, AUX>;
        f = reinterpret_cast<const void *>(k);
        fe = reinterpret_cast<const void *>(ke);
    }
    return Variant{name, WIDE, WideCfg::BM, WideCfg::BN, WideCfg::BKB, WideCfg::NTHREADS, f, false, fe};
}

// Stream-K schedule of the one-wave-per-SIMD kernel (stream_k.hpp); FP16
// and INT8 only, like wide().
template <int DT>
Variant wide_sk(const char *name) {
    const void *f = nullptr, *fe = nullptr;
    if constexpr (DT == F16 || DT == S8) {
        sk_fn k = &wide_gemm_sk<DT, true>, ke = &wide_gemm_sk<DT, false>;
        f = reinterpret_cast<const void *>(k);
        fe = reinterpret_cast<const void *>(ke);
    }
    return Variant{name, WIDE_SK, WideCfg::BM, WideCfg::BN, WideCfg::BKB, WideCfg::NTHREADS, f, false, fe};
}

// INT4 on the FP6 cores with the conversion inside the GEMM (wide_i4.hpp);
// bkb holds the K multiple it needs (in elements). AUX: cache policy of the
// operand loads.
template <int AUX = CP_DEFAULT>
Variant i4wide(const char *name) {
    kernel_fn k = &wide_i4_gemm<true, AUX>, ke = &wide_i4_gemm<false, AUX>;
    return Variant{name, I4WIDE, WideI4Cfg::BM, WideI4Cfg::BN, 256, WideI4Cfg::NTHREADS,
                   reinterpret_cast<const void *>(k), false, reinterpret_cast<const void *>(ke)};
}

template <class T>
Variant fp6(const char *name) {
    typedef void (*f6_fn)(const uint8_t *, const uint8_t *, const uint8_t *, const uint8_t *,
                          int32_t *, int, int, int, int, int, int, int, EpiParams);
    f6_fn f = &f6_gemm<T>;
    return Variant{name, FP6, T::BM, T::BN, T::J, T::NTHREADS, reinterpret_cast<const void *>(f),
                   false};
}

// The one-wave-per-SIMD FP6 kernel (wide_f6.hpp); the table holds its
// raw-sum instantiation, the launcher swaps in the other where needed. AUX:
// cache policy of the copy loads.
template <int AUX = CP_DEFAULT>
Variant fp6wide(const char *name) {
    typedef void (*f6_fn)(const uint8_t *, const uint8_t *, const uint8_t *, const uint8_t *,
                          int32_t *, int, int, int, int, int, int, int, EpiParams);
    f6_fn f = &wide_f6_gemm<true, AUX>, fe = &wide_f6_gemm<false, AUX>;
    return Variant{name, FP6WIDE, WideF6Cfg::BM, WideF6Cfg::BN, WideF6Cfg::J, WideF6Cfg::NTHREADS,
                   reinterpret_cast<const void *>(f), false, reinterpret_cast<const void *>(fe)};
}

// Stream-K schedule of the one-wave-per-SIMD FP6 kernel (stream_k.hpp).
template <int AUX = CP_DEFAULT>
Variant fp6wide_sk(const char *name) {
    typedef void (*f6sk_fn)(const uint8_t *, const uint8_t *, const uint8_t *, const uint8_t *, int32_t *, int,
                            int, int, int, int, int, int, SkArgs, EpiParams);
    f6sk_fn f = &wide_f6_gemm_sk<true, AUX>, fe = &wide_f6_gemm_sk<false, AUX>;
    return Variant{name, FP6WIDE_SK, WideF6Cfg::BM, WideF6Cfg::BN, WideF6Cfg::J, WideF6Cfg::NTHREADS,
                   reinterpret_cast<const void *>(f), false, reinterpret_cast<const void *>(fe)};
}

template <int DT>
Variant generic(const char *name) {
    generic_fn f = &generic_gemm<DT>;
    return Variant{name, GENERIC, 32, 32, 0, 64, reinterpret_cast<const void *>(f), false};
}

#define VARIANT_LIST(DT)                                                   \
    generic<DT>("generic_32x32"),                                          \
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
     pipelined<DT, T128x128_w4_s4_m16, true>("spread128x128_w2x2_k128_s4_m16"), \
     pipelined<DT, T256x256_w8_k64_s4>("pipe256x256_w2x4_k64_s4"),          \
     pipelined<DT, T256x256_w8_k64_s3>("pipe256x256_w2x4_k64_s3"),          \
     deep<DT, T256x256_w4_k64_s4>("deep256x256_w2x2_k64_s4"),             \
     deep<DT, T256x256_w4_k64_s5>("deep256x256_w2x2_k64_s5"),             \
     skinny<DT, 1, 1>("skinny16x16_k64"),                                 \
     skinny<DT, 1, 2>("skinny16x32_k64"),                                 \
     skinny<DT, 2, 1>("skinny32x16_k64"),                                 \
     skinny<DT, 2, 2>("skinny32x32_k64"),                                 \
     skinny<DT, 1, 2, 8>("skinny16x32_k64_d8"),                           \
     skinny<DT, 4, 2>("skinny64x32_k64"),                                 \
     pipelined<DT, T32x64_w2_m16, true>("spread32x64_w1x2_k128_s4_m16"),  \
     pipelined<DT, T32x128_w4_m16, true>("spread32x128_w1x4_k128_s4_m16"), \
     pipelined<DT, T64x128_w4, true>("spread64x128_w2x2_k128_s4"),        \
     pipelined<DT, T64x32_w2_m16, true>("spread64x32_w2x1_k128_s4_m16"),  \
     pipelined<DT, T128x32_w4_m16, true>("spread128x32_w4x1_k128_s4_m16"), \
     pipelined<DT, T128x64_w4, true>("spread128x64_w2x2_k128_s4"),        \
     wide<DT>("wide256x256_w2x2_k128_m16"),                                \
     wide<DT, CP_SC0>("wide256x256_w2x2_k128_m16_sc0"),                    \
     wide<DT, CP_SC1>("wide256x256_w2x2_k128_m16_sc1"),                    \
     wide<DT, CP_NT>("wide256x256_w2x2_k128_m16_nt"),                     \
     pipelined<DT, T128x128_w8_s4, true>("spread128x128_w2x4_k128_s4"),    \
     pipelined<DT, T128x128_w8_k64_s4, true>("spread128x128_w2x4_k64_s4"), \
     pipelined<DT, T64x64_w4_m16, true>("spread64x64_w2x2_k128_s4_m16"),   \
     pipelined<DT, T64x128_w8, true>("spread64x128_w2x4_k128_s4"),         \
     pipelined<DT, T128x64_w8, true>("spread128x64_w4x2_k128_s4"),         \
     pipelined<DT, T32x64_w2_m16_s8, true>("spread32x64_w1x2_k128_s8_m16"),   \
     pipelined<DT, T32x128_w4_m16_s8, true>("spread32x128_w1x4_k128_s8_m16"), \
     pipelined<DT, T64x32_w2_m16_s8, true>("spread64x32_w2x1_k128_s8_m16"),   \
     pipelined<DT, T128x32_w4_m16_s8, true>("spread128x32_w4x1_k128_s8_m16"), \
     pipelined<DT, T64x64_w4_m16_s8, true>("spread64x64_w2x2_k128_s8_m16"),   \
     wide_sk<DT>("wide256x256_w2x2_k128_m16_sk"),                          \
     pipelined_sk<DT, T256x256_w8_s2, false>("pipe256x256_w2x4_k128_s2_sk"), \
     pipelined_sk<DT, T128x128_w4_s4, true>("spread128x128_w2x2_k128_s4_sk"), \
     pipelined_sk<DT, T128x128_w8_s4, true>("spread128x128_w2x4_k128_s4_sk"), \
     pipelined_sk<DT, T128x128_w8_k64_s4, true>("spread128x128_w2x4_k64_s4_sk")

// Number of entries of VARIANT_LIST, and the INT4 table's FP6 variants after
// them (variants_s4.hip); each table checks its size against these.
constexpr int kNumCommon = 69;
constexpr int kNumFp6 = 17;
constexpr int kNumF16 = kNumCommon, kNumS8 = kNumCommon, kNumS4 = kNumCommon + kNumFp6;

// Kernel of the transposed-B entry point (tposeb.hip): F16 or S8, else null.
const void *tposeb_kernel(int dtype);

extern const Variant kF16[];
extern const Variant kS8[];
extern const Variant kS4[];

}  // namespace mpg
