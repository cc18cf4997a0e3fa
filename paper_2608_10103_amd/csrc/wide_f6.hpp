// wide_f6.hpp - INT4 on the FP6 matrix cores with one wave per SIMD and
// 128 x 128 wave tiles.
//
// Same operands as f6_gemm (both converted once by s4_to_e3m2 into the
// run-major E3M2 workspace: P parts of 16 bytes, then Q parts of 8 bytes,
// rows of one run contiguous) and the same lane assignment per 32x32x64
// MFMA, but the schedule of wide_gemm.hpp:
//
//  * 4 waves of 128 x 128 (4 x 4 blocks of 32 x 32, 256 FP32 accumulators
//    per lane, all AGPRs). Operand bytes read from LDS per MFMA are two
//    thirds of those of the 8-wave 128 x 64 layout, which at the FP6 rate (a
//    32x32x64 MFMA every 32 cycles per SIMD) asks the LDS for more bytes per
//    cycle than its port delivers.
//  * MFMAs as inline assembly with the accumulator tied to its AGPRs (left
//    to the compiler, full AGPRs make it shuffle accumulators every
//    iteration).
//  * K in slices of J = 4 runs (128 k, two MFMA k-chunks), three LDS stages
//    of 48 KiB. Wave w copies run w of every slice: 4 + 2 loads of A
//    (P rows 0..255 in 64-row loads, Q in 128-row loads) and 4 + 2 of B,
//    each 1 KiB of one contiguous workspace range (eight whole lines, lanes
//    in address order) into a contiguous 1 KiB of LDS. The LDS image of a
//    stage is the workspace order: reads of 32 consecutive rows are
//    contiguous, so neither copies nor reads conflict in the banks.
//
// Schedule of slice kt (buffer kt % 3; chunk c computes on fragment set c
// while the other set is read; one fragment read after every second MFMA):
//   chunk 0: read chunk 1 of slice kt; copy loads 6..11 of slice kt + 2;
//   wait: own reads done, slice kt + 1 landed (slice kt + 2 in flight);
//   barrier: every wave has read slice kt, its buffer is free;
//   chunk 1: read chunk 0 of slice kt + 1; loads 0..5 of slice kt + 3 into
//     buffer kt % 3.
// A slice's loads are issued 1.5 to 2 slices before it is read. Slices past
// the end of K are fetched as the last slice again into buffers nobody reads
// (one loop body for every slice).
#pragma once

#include "f6_gemm.hpp"
#include "wide_gemm.hpp"

namespace mpg {

struct WideF6Cfg {
    static constexpr int BM = 256, BN = 256, J = 4, NTHREADS = 256, STAGES = 3;
    static constexpr int AP = 0, AQ = J * BM * 16, BP = J * BM * 24, BQ = BP + J * BN * 16;
    static constexpr int STAGE = J * (BM + BN) * 24;  // 48 KiB
    static constexpr int LDS_BYTES = STAGES * STAGE;  // 144 KiB
    static_assert(LDS_BYTES <= 160 * 1024, "LDS capacity");
    static_assert(F6Geom::ROW_PAD % BM == 0 && F6Geom::K_PAD % (32 * J) == 0, "tiles and slices stay in the padding");
};

// 32x32x64 MFMA, E3M2 on both sides (cbsz = blgp = 3), unit scales; the
// accumulator tied to one AGPR tuple, used once per k-chunk (16 MFMAs apart).
__device__ __forceinline__ void wf6_mfma(const F6Frag &a, const F6Frag &b, f32x16 &c) {
    asm volatile("v_mfma_f32_32x32x64_f8f6f4 %0, %1, %2, %0 cbsz:3 blgp:3" : "+a"(c) : "v"(a), "v"(b));
}

// The copy loads of one wave: run w of a slice, A rows then B rows of the
// tile. Byte offsets are 32-bit (the entry point bounds each workspace part).
struct WF6Copy {
    const uint8_t *ap, *aq, *bp, *bq;  // workspace parts
    int apn, aqn, bpn, bqn;            // their bytes
    int ap0, aq0, bp0, bq0;            // offsets of run w, tile rows, slice 0
    int aps, aqs, bps, bqs;            // offset step per slice
    uint32_t voff;                     // 16 l
    uint8_t *dp, *dq;                  // lds + run w's offset in a P / Q part
};

// copy load u (0..11) of slice ks into stage s; AUX: cache policy
template <int AUX>
__device__ __forceinline__ void wf6_load(const WF6Copy &c, int u, int ks, int s) {
    typedef WideF6Cfg T;
    const int so = s * T::STAGE;
    if (u < 4) wide_copy<AUX>(c.ap, c.apn, c.dp + so + T::AP + u * 1024, c.voff, c.ap0 + ks * c.aps + u * 1024);
    else if (u < 6) wide_copy<AUX>(c.aq, c.aqn, c.dq + so + T::AQ + (u - 4) * 1024, c.voff, c.aq0 + ks * c.aqs + (u - 4) * 1024);
    else if (u < 10) wide_copy<AUX>(c.bp, c.bpn, c.dp + so + T::BP + (u - 6) * 1024, c.voff, c.bp0 + ks * c.bps + (u - 6) * 1024);
    else wide_copy<AUX>(c.bq, c.bqn, c.dq + so + T::BQ + (u - 10) * 1024, c.voff, c.bq0 + ks * c.bqs + (u - 10) * 1024);
}

// One k-chunk: 16 MFMAs on (a, b); after MFMA 2 f, fragment f of the next
// set in the order a0 b0 b1 b2 b3 a1 a2 a3 (the order the next chunk's MFMAs
// first need them); after MFMA 2 u + 1, copy load U0 + u (u < 6) of slice ks
// into stage s. pa/qa, pb/qb: LDS offsets of the P and Q parts of block 0
// of the next set (f6_frag reads them).
template <int U0, int AUX>
__device__ __forceinline__ void wf6_chunk(const F6Frag (&a)[4], const F6Frag (&b)[4], f32x16 (&acc)[4][4],
                                          F6Frag (&na)[4], F6Frag (&nb)[4], const uint8_t *lds, int pa,
                                          int qa, int pb, int qb, const WF6Copy &c, int ks, int s) {
    static_for<16>([&](auto mm) __attribute__((always_inline)) {
        constexpr int m = decltype(mm)::value;
        __builtin_amdgcn_sched_barrier(0);
        wf6_mfma(a[m / 4], b[m % 4], acc[m / 4][m % 4]);
        if constexpr (m % 2 == 0) {
            constexpr int f = m / 2;
            if constexpr (f == 0) na[0] = f6_frag(lds, pa, qa);
            else if constexpr (f <= 4) nb[f - 1] = f6_frag(lds, pb + (f - 1) * 512, qb + (f - 1) * 256);
            else na[f - 4] = f6_frag(lds, pa + (f - 4) * 512, qa + (f - 4) * 256);
        } else if constexpr (m / 2 < 6) {
            wf6_load<AUX>(c, U0 + m / 2, ks, s);
        }
        __builtin_amdgcn_sched_barrier(0);
    });
}

// Accumulate slices [kt0, kt0 + KT) of tile (tm, tn) into acc (zeroed
// here) with the schedule above; KT >= 1 (the prologue's loads of slices
// kt0 + 1 and kt0 + 2 stay inside the padded workspace or read zeros past
// it, into buffers no MFMA reads when KT is smaller). Ap/Aq, Bp/Bq: the
// converted operands, Ma / Nb their padded row counts, KTW the slices of the
// whole padded K. On return every copy has landed and the accumulators are
// safe to read; waves may still be reading LDS.
template <int AUX>
__device__ __forceinline__ void wf6_accumulate(uint8_t *lds, const uint8_t *Ap, const uint8_t *Aq,
                                               const uint8_t *Bp, const uint8_t *Bq, int Ma, int Nb, int KTW,
                                               int tm, int tn, int kt0, int KT, f32x16 (&acc)[4][4]) {
    typedef WideF6Cfg T;
    // opaque thread id (see pf_accumulate)
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 31, h = lane >> 5;
    const int wm = wave / 2, wn = wave % 2;

    // run w of slice ks is workspace run 4 (kt0 + ks) + w
    WF6Copy c;
    const int runs = KTW * T::J;
    c.ap = Ap; c.aq = Aq; c.bp = Bp; c.bq = Bq;
    c.apn = runs * Ma * 16; c.aqn = runs * Ma * 8; c.bpn = runs * Nb * 16; c.bqn = runs * Nb * 8;
    c.aps = T::J * Ma * 16; c.aqs = T::J * Ma * 8; c.bps = T::J * Nb * 16; c.bqs = T::J * Nb * 8;
    c.ap0 = (wave * Ma + tm * T::BM) * 16 + kt0 * c.aps; c.aq0 = (wave * Ma + tm * T::BM) * 8 + kt0 * c.aqs;
    c.bp0 = (wave * Nb + tn * T::BN) * 16 + kt0 * c.bps; c.bq0 = (wave * Nb + tn * T::BN) * 8 + kt0 * c.bqs;
    c.voff = (uint32_t)lane * 16;
    // stage image: each part holds runs 0..3 of 256 rows, run w at
    // w * 256 * 16 (P) or w * 256 * 8 (Q) from the part's start
    c.dp = lds + wave * 4096;
    c.dq = lds + wave * 2048;

    // lane (r, h) reads run 2 kc + h of row 32 i + r of its wave's 128 rows
    const int rowa = h * T::BM + wm * 128 + r, rowb = h * T::BN + wn * 128 + r;
    const int pa0 = T::AP + rowa * 16, qa0 = T::AQ + rowa * 8;
    const int pb0 = T::BP + rowb * 16, qb0 = T::BQ + rowb * 8;
    constexpr int KCP = 2 * T::BM * 16, KCQ = 2 * T::BM * 8;  // next k-chunk: two runs on

#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};
    // zeroed accumulators into their AGPRs in order, then wait states before
    // the first assembly MFMA reads them (the compiler does not insert them;
    // a VALU write of an MFMA's accumulator input needs 2, the nop gives 5)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) asm volatile("" : "+a"(acc[i][j]));
    asm volatile("s_nop 4" ::: "memory");

    // prologue: slices 0 and 1 whole, loads 0..5 of slice 2; wait for slice 0
#pragma unroll
    for (int u = 0; u < 12; ++u) wf6_load<AUX>(c, u, 0, 0);
#pragma unroll
    for (int u = 0; u < 12; ++u) wf6_load<AUX>(c, u, 1, 1);
#pragma unroll
    for (int u = 0; u < 6; ++u) wf6_load<AUX>(c, u, min(2, KT - 1), 2);
    asm volatile("s_waitcnt vmcnt(18)\n\ts_barrier" ::: "memory");
    // chunk 0 of slice 0; then a wait the compiler knows of (lgkmcnt(0)),
    // so that at the loop head only the reads of the previous iteration are
    // outstanding and its wait covers just the first fragments
    F6Frag ra[2][4], rb[2][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) ra[0][i] = f6_frag(lds, pa0 + i * 512, qa0 + i * 256);
#pragma unroll
    for (int j = 0; j < 4; ++j) rb[0][j] = f6_frag(lds, pb0 + j * 512, qb0 + j * 256);
    asm volatile("" ::: "memory");  // keeps the reads above the wait
    __builtin_amdgcn_s_waitcnt(0xC07F);

    for (int kt = 0; kt < KT; ++kt) {
        const int s0 = kt % 3, s1 = (kt + 1) % 3, s2 = (kt + 2) % 3;
        const int cur = s0 * T::STAGE, nxt = s1 * T::STAGE;
        wf6_chunk<6, AUX>(ra[0], rb[0], acc, ra[1], rb[1], lds, pa0 + cur + KCP, qa0 + cur + KCQ, pb0 + cur + KCP,
                     qb0 + cur + KCQ, c, min(kt + 2, KT - 1), s2);
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_waitcnt vmcnt(12)\n\ts_barrier" ::: "memory");
        wf6_chunk<0, AUX>(ra[1], rb[1], acc, ra[0], rb[0], lds, pa0 + nxt, qa0 + nxt, pb0 + nxt, qb0 + nxt, c,
                     min(kt + 3, KT - 1), s0);
    }
    // Clamped copies may still be landing. The last MFMA results: an XDL op
    // of P passes (P = 8 for the 32x32x64 FP6 MFMA, 16 for FP8) needs P + 3
    // wait states before a VALU or memory instruction reads its destination,
    // and the compiler does not count them for the assembly MFMAs; the nops
    // give 40. The empty asm statements then order every read of the
    // accumulators after the nops.
    asm volatile("s_waitcnt vmcnt(0)\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) asm volatile("" : "+a"(acc[i][j]));
}

// Accumulators of a finished tile to C: PLAIN, raw sums of a whole tile
// stored straight from the accumulators; otherwise the shared epilogue
// (ragged edges, scales).
template <bool PLAIN>
__device__ __forceinline__ void wf6_store(const EpiParams &epi, int32_t *C, const f32x16 (&acc)[4][4], int tm,
                                          int tn, int M, int N) {
    typedef WideF6Cfg T;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 31, h = lane >> 5;
    const int wm = wave / 2, wn = wave % 2;
    const long row0 = (long)tm * T::BM + wm * 128;
    const long col0 = (long)tn * T::BN + wn * 128 + r;
    if constexpr (PLAIN) {
        // element (i, j, v): row row0 + 32 i + 8 (v / 4) + 4 h + v % 4,
        // column col0 + 32 j; the sums are integers below 2^24 in magnitude
        int32_t *base = C + (row0 + 4 * h) * (long)N + col0;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                int32_t *rowp = base + (long)(32 * i + 8 * (v / 4) + v % 4) * N;
#pragma unroll
                for (int j = 0; j < 4; ++j) rowp[32 * j] = (int)acc[i][j][v];
            }
    } else {
        epi_store_tile<S4, 32, 4, 4, 16>(epi, C, acc, row0, col0, h, M, N, ConvToInt());
    }
}

// Consume the kernel arguments the epilogue reads (C, M, N and the epilogue
// parameters) at entry: a scalar load of them still in flight in the loop
// would make every LDS wait there a wait for all (scalar loads return out of
// order).
template <bool PLAIN>
__device__ __forceinline__ void wf6_entry_args(const int32_t *C, int M, int N, const EpiParams &epi) {
    asm volatile("" ::"s"(C), "s"(M), "s"(N));
    if constexpr (!PLAIN)
        asm volatile("" ::"s"(epi.scale_a), "s"(epi.scale_b), "s"(epi.zero_a), "s"(epi.zero_b), "s"(epi.sum_a),
                     "s"(epi.sum_b), "s"(epi.K), "s"(epi.out));
}

// Ap/Aq, Bp/Bq: converted operands; Ma / Nb their padded row counts; KT =
// padded K / 128 slices (at least 2: K is padded to 256). PLAIN: raw sums to
// a row-major int32 C of whole 256 x 256 tiles, stored straight from the
// accumulators; otherwise the shared epilogue (ragged edges, scales). AUX:
// cache policy of the copy loads.
template <bool PLAIN, int AUX = CP_DEFAULT>
__global__ __launch_bounds__(WideF6Cfg::NTHREADS, 1) void wide_f6_gemm(
    const uint8_t *__restrict__ Ap, const uint8_t *__restrict__ Aq, const uint8_t *__restrict__ Bp,
    const uint8_t *__restrict__ Bq, int32_t *__restrict__ C, int M, int N, int Ma, int Nb, int KT,
    int tiles_m, int tiles_n, EpiParams epi) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[WideF6Cfg::LDS_BYTES];
    wf6_entry_args<PLAIN>(C, M, N, epi);
    int tm, tn;
    tile_coords(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, 4, tm, tn);
    f32x16 acc[4][4];
    wf6_accumulate<AUX>(lds, Ap, Aq, Bp, Bq, Ma, Nb, KT, tm, tn, 0, KT, acc);
    wf6_store<PLAIN>(epi, C, acc, tm, tn, M, N);
}

}  // namespace mpg
