// wide_gemm.hpp - one wave per SIMD, 128 x 128 wave tiles, hand-ordered
// schedule (FP16 and INT8).
//
// 256 x 256 tile of C per workgroup, 2 x 2 waves of 128 x 128 on 16x16 MFMAs
// (64 accumulator blocks: 256 accumulator registers per lane), K in 128-byte
// slices (two 64-byte MFMA K-chunks) in two LDS buffers filled by
// direct-to-LDS buffer loads. Measured on MI355X, three things decide its
// speed; each shaped the design:
//
//  * Copy loads. One load moves 1 KiB; the address path takes a load of
//    eight whole 128-byte lines much faster than one touching sixteen half
//    lines, and several waves issuing loads back to back fill its queue
//    (stalling MFMA issue). So every load fetches 128 bytes of each of 8
//    rows, with the 64 lanes in address order, and a wave issues one load per
//    two MFMA groups.
//  * LDS layout. A load writes 1 KiB contiguously, so a block holds its 8
//    rows; with the rows of a block consecutive, the 16 rows one operand read
//    touches fall into only 4 bank groups. Here load j of a wave fetches rows
//    j, j + 16, ..., j + 112 of the wave's 128-row panel: the 16 rows of an
//    MFMA block sit at the same position of 16 consecutive blocks, blocks are
//    padded to 1024 + 32 bytes, and a read touches 16 bank groups. Each wave
//    copies exactly the 128 rows it (or its partner wave) reads.
//  * Registers. The 256 accumulators fill the AGPRs; left to the compiler,
//    some MFMAs get a destination other than their source and the
//    accumulators are shuffled back every iteration. The MFMAs are written as
//    inline assembly with the accumulator tied to its registers.
//
// Schedule of slice kt (chunk c uses operand register set c; reads fill the
// other set; "group" = four MFMA blocks between scheduling fences):
//   chunk 0, groups 0-5 read chunk 1 of slice kt; groups 0, 2, 4, 6 issue
//     copy loads 12-15 of slice kt + 1;
//   barrier 1: every wave has read slice kt, its buffer is free;
//   chunk 0, groups 8, 10, 12, 14 issue loads 0-3 of slice kt + 2 into it;
//   chunk 1, groups 0, 2, 4, 6: loads 4-7 of slice kt + 2;
//   barrier 2: slice kt + 1 has landed (loads of slice kt + 2 in flight);
//   chunk 1, groups 8-13 read chunk 0 of slice kt + 1; groups 8, 10, 12, 14
//     issue loads 8-11 of slice kt + 2.
// A wave's 16 loads of a slice are spread over 32 groups, and each has at
// least 16 groups to land. Past the end of K the loads fetch the last slice
// again into a buffer nobody reads (one loop body for every slice).
// M and N may be ragged: each panel's buffer bound covers only its rows
// inside the matrix (loads of rows past it return zeros and touch no
// memory), and rows and columns past M and N are not stored. K bytes must be
// a multiple of 128.
#pragma once

#include "tiled_gemm.hpp"

namespace mpg {

struct WideCfg {
    static constexpr int BM = 256, BN = 256, BKB = 128, MS = 16, NTHREADS = 256;
    static constexpr int BLK = 1024 + 32;     // LDS bytes per 8-row copy block
    static constexpr int STAGE = 64 * BLK;    // 512 rows: A 256, B 256
    static constexpr int LDS_BYTES = 2 * STAGE;
    static_assert(LDS_BYTES <= 160 * 1024, "LDS capacity");
};

// Cache policy of the copy loads (the instruction's cache-policy bits: sc0 =
// 1, nt = 2, sc1 = 16; 0 = the default policy), the CDNA4 counterpart of the
// paper's cp.async .ca / .cg choice (Run 4).
enum CachePolicy : int { CP_DEFAULT = 0, CP_SC0 = 1, CP_NT = 2, CP_SC1 = 16 };

// One wave-wide direct-to-LDS buffer load: lane l copies 16 bytes from
// base + voff + soff (voff its own, soff wave-uniform) to lds + 16 l; `bytes`
// bounds the buffer (loads past it read zeros). Device pass only.
template <int AUX = CP_DEFAULT>
__device__ __forceinline__ void wide_copy(const uint8_t *base, int bytes, uint8_t *lds, uint32_t voff, int soff) {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        __builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0, bytes, 0x00020000), (lds_void *)lds, 16,
        (int)voff, soff, 0, AUX);
#endif
}

// 16x16 MFMA with the accumulator tied to one AGPR tuple. Every accumulator
// is used once per K-chunk (64 MFMAs apart), so no MFMA waits on the one
// before it; the kernel waits for the last results before its epilogue.
template <int DT>
__device__ __forceinline__ void wide_mfma(i32x4 a, i32x4 b, typename Acc<DT, 16>::type &c) {
    if constexpr (DT == F16)
        asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
    else
        asm volatile("v_mfma_i32_16x16x64_i8 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}

struct WideCopy {
    const uint8_t *panel;  // the wave's 128-row panel of A or B
    int bytes;             // 128 rows of K bytes
    uint32_t voff;         // lane: row 16 (l / 8) of the load, bytes 16 (l % 8) ..
    int kb;                // row pitch (bytes)
    uint8_t *dst;          // this wave's first copy block in buffer 0
};

// copy load j (0..15) of slice ks into buffer b
template <int AUX>
__device__ __forceinline__ void wide_load(const WideCopy &c, int j, int ks, int b) {
    wide_copy<AUX>(c.panel, c.bytes, c.dst + b * WideCfg::STAGE + j * WideCfg::BLK, c.voff, ks * WideCfg::BKB + j * c.kb);
}

// Groups [G0, G1) of one K-chunk CH: MFMAs on (a, b); reads of the 16 runs
// of the next operands into (na, nb) in groups [R0, R0 + 6); copy loads as in
// the schedule above (slice k1 = kt + 1, k2 = kt + 2, clamped).
template <int DT, int CH, int R0, int G0, int G1, int AUX>
__device__ __forceinline__ void wide_groups(const i32x4 (&a)[8], const i32x4 (&b)[8],
                                            typename Acc<DT, 16>::type (&acc)[8][8], i32x4 (&na)[8],
                                            i32x4 (&nb)[8], const uint8_t *rab, const uint8_t *rbb,
                                            const WideCopy &c, int k1, int k2, int kt) {
    static_for<G1 - G0>([&](auto gg) __attribute__((always_inline)) {
        constexpr int g = G0 + decltype(gg)::value;
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int p = 4 * g; p < 4 * g + 4; ++p) wide_mfma<DT>(a[p / 8], b[p % 8], acc[p / 8][p % 8]);
        if constexpr (g >= R0 && g < R0 + 6) {
            static_for<3>([&](auto xx) __attribute__((always_inline)) {
                constexpr int q = 3 * (g - R0) + decltype(xx)::value;  // run: A 0..7, B 8..15
                if constexpr (q < 8) na[q] = *reinterpret_cast<const i32x4 *>(rab + q * WideCfg::BKB);
                else if constexpr (q < 16) nb[q - 8] = *reinterpret_cast<const i32x4 *>(rbb + (q - 8) * WideCfg::BKB);
            });
        }
        if constexpr (g % 2 == 0) {
            if constexpr (CH == 0 && g < 8) wide_load<AUX>(c, 12 + g / 2, k1, (kt + 1) & 1);
            if constexpr (CH == 0 && g >= 8) wide_load<AUX>(c, (g - 8) / 2, k2, kt & 1);
            if constexpr (CH == 1 && g < 8) wide_load<AUX>(c, 4 + g / 2, k2, kt & 1);
            if constexpr (CH == 1 && g >= 8) wide_load<AUX>(c, 8 + (g - 8) / 2, k2, kt & 1);
        }
        __builtin_amdgcn_sched_barrier(0);
    });
}

// Accumulate K-slices [kt0, kt0 + KT) of tile (tm, tn) into acc (zeroed
// here) with the schedule above; A has M rows, B N rows (ragged edges read
// as zeros). On return every copy has landed and the accumulators are safe
// to read; the waves may still be reading LDS, so a caller that reuses the
// buffers for another tile needs a barrier first.
template <int DT, int AUX>
__device__ __forceinline__ void wide_accumulate(uint8_t *lds, const uint8_t *A, const uint8_t *B, int M, int N,
                                                int Kb, int tm, int tn, int kt0, int KT,
                                                typename Acc<DT, 16>::type (&acc)[8][8]) {
    typedef WideCfg T;
    typedef typename Acc<DT, 16>::type acc_t;
    // opaque thread id: see pf_accumulate
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane % 16, h = lane / 16;
    const int wm = wave / 2, wn = wave % 2;

    // wave w copies panel w: A rows [128 w, 128 w + 128) of the tile for w < 2,
    // B rows [128 (w - 2), ...) otherwise, into copy blocks [16 w, 16 w + 16);
    // the panel starts at slice kt0
    WideCopy c;
    const int row0 = (wave < 2) ? tm * T::BM + wave * 128 : tn * T::BN + (wave - 2) * 128;
    c.panel = ((wave < 2) ? A : B) + (size_t)row0 * Kb + (size_t)kt0 * T::BKB;
    // the panel's rows inside the matrix (0 .. 128): the buffer bound, so
    // that copies of rows past M (N) read zeros without touching memory
    // (wave-uniform; kept in a scalar register, or every copy load becomes a
    // loop over the descriptor values of the wave's lanes)
    const int rows = min(max(((wave < 2) ? M : N) - row0, 0), 128);
    c.bytes = __builtin_amdgcn_readfirstlane(rows ? rows * Kb - kt0 * T::BKB : 0);
    c.voff = (uint32_t)((lane / 8) * 16 * Kb + (lane % 8) * 16);
    c.kb = Kb;
    c.dst = lds + wave * 16 * T::BLK;
    // run p of A (rows 128 wm + 16 p + r): position p of block 16 wm + r;
    // lane group h reads logical chunk h (chunk 0) or 4 + h (chunk 1)
    const uint8_t *ra0 = lds + (wm * 16 + r) * T::BLK + h * 16;
    const uint8_t *rb0 = lds + (32 + wn * 16 + r) * T::BLK + h * 16;

#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = acc_t{};
    // The zeroed accumulators are written to the AGPRs here (each empty asm
    // takes its block in AGPRs, in order), then wait states before the first
    // assembly MFMA reads them: the compiler does not insert them for
    // assembly it does not know is an MFMA. A VALU write of a register an
    // MFMA then reads as its accumulator needs 2 wait states; the nop gives 5.
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) asm volatile("" : "+a"(acc[i][j]));
    asm volatile("s_nop 4" ::: "memory");

    // prologue: slice 0 whole, loads 0-11 of slice 1; wait for slice 0
#pragma unroll
    for (int j = 0; j < 16; ++j) wide_load<AUX>(c, j, 0, 0);
#pragma unroll
    for (int j = 0; j < 12; ++j) wide_load<AUX>(c, j, min(1, KT - 1), 1);
    asm volatile("s_waitcnt vmcnt(12)\n\ts_barrier" ::: "memory");
    i32x4 ra[2][8], rb[2][8];
#pragma unroll
    for (int p = 0; p < 8; ++p) ra[0][p] = *reinterpret_cast<const i32x4 *>(ra0 + p * T::BKB);
#pragma unroll
    for (int p = 0; p < 8; ++p) rb[0][p] = *reinterpret_cast<const i32x4 *>(rb0 + p * T::BKB);

    for (int kt = 0; kt < KT; ++kt) {
        const int cur = (kt & 1) * T::STAGE, nxt = ((kt + 1) & 1) * T::STAGE;
        const int k1 = min(kt + 1, KT - 1), k2 = min(kt + 2, KT - 1);
        const uint8_t *r1a = ra0 + cur + 64, *r1b = rb0 + cur + 64;  // chunk 1 of slice kt
        const uint8_t *r0a = ra0 + nxt, *r0b = rb0 + nxt;            // chunk 0 of slice kt + 1
        wide_groups<DT, 0, 0, 0, 8, AUX>(ra[0], rb[0], acc, ra[1], rb[1], r1a, r1b, c, k1, k2, kt);
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        wide_groups<DT, 0, 0, 8, 16, AUX>(ra[0], rb[0], acc, ra[1], rb[1], r1a, r1b, c, k1, k2, kt);
        wide_groups<DT, 1, 8, 0, 8, AUX>(ra[1], rb[1], acc, ra[0], rb[0], r0a, r0b, c, k1, k2, kt);
        asm volatile("s_waitcnt vmcnt(8)\n\ts_barrier" ::: "memory");
        wide_groups<DT, 1, 8, 8, 16, AUX>(ra[1], rb[1], acc, ra[0], rb[0], r0a, r0b, c, k1, k2, kt);
    }
    // Clamped copies may still be landing. The last MFMA results: an XDL op
    // of P passes (P = 8 for the 16x16 FP16 and INT8 MFMAs here) needs
    // P + 3 wait states before a VALU or memory instruction reads its
    // destination, and the compiler does not count them for the assembly
    // MFMAs; the nops give 32. The empty asm statements then order every
    // read of the accumulators after the nops.
    asm volatile("s_waitcnt vmcnt(0)\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) asm volatile("" : "+a"(acc[i][j]));
}

// Accumulators of a finished tile to C. PLAIN: raw sums of a whole tile to
// the row-major output, stored straight from the accumulators; otherwise the
// shared epilogue with scales, zero points, output types and ragged edges
// (see EpiParams).
template <int DT, bool PLAIN>
__device__ __forceinline__ void wide_store(const EpiParams &epi, void *Cv,
                                           const typename Acc<DT, 16>::type (&acc)[8][8], int tm, int tn,
                                           int M, int N) {
    typedef WideCfg T;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane % 16, h = lane / 16;
    const int wm = wave / 2, wn = wave % 2;
    const long row0 = (long)tm * T::BM + wm * 128;
    const long col0 = (long)tn * T::BN + wn * 128 + r;
    if constexpr (PLAIN) {
        // whole tiles: element (i, j, v) of this lane is row row0 + 16 i +
        // 4 h + v, column col0 + 16 j
        typedef typename Acc<DT, 16>::out out_t;
        out_t *base = reinterpret_cast<out_t *>(Cv) + (row0 + 4 * h) * (long)N + col0;
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                out_t *rowp = base + (long)(16 * i + v) * N;
#pragma unroll
                for (int j = 0; j < 8; ++j) rowp[16 * j] = acc[i][j][v];
            }
    } else {
        epi_store_tile<DT, 16, 8, 8, 4>(epi, Cv, acc, row0, col0, h, M, N, ConvSame());
    }
}

// PLAIN: see wide_store. AUX: cache policy of the copy loads.
template <int DT, bool PLAIN = true, int AUX = CP_DEFAULT>
__global__ __launch_bounds__(WideCfg::NTHREADS, 1) void wide_gemm(const uint8_t *__restrict__ A,
                                                                 const uint8_t *__restrict__ B,
                                                                 void *__restrict__ Cv, int M, int N, int Kb,
                                                                 int tiles_m, int tiles_n, EpiParams epi) {
    static_assert(DT == F16 || DT == S8, "FP16 and INT8");
    __shared__ __attribute__((aligned(1024))) uint8_t lds[WideCfg::LDS_BYTES];
    int tm, tn;
    tile_coords(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, 4, tm, tn);
    typename Acc<DT, 16>::type acc[8][8];
    wide_accumulate<DT, AUX>(lds, A, B, M, N, Kb, tm, tn, 0, Kb / WideCfg::BKB, acc);
    wide_store<DT, PLAIN>(epi, Cv, acc, tm, tn, M, N);
}

}  // namespace mpg
