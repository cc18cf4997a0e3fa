// wide_i4.hpp - INT4 GEMM on the FP6 matrix cores with the conversion done
// inside the GEMM: no pre-pass, no workspace.
//
// gfx950 has no 4-bit integer MFMA; its f8f6f4 MFMA multiplies FP6 at twice
// the INT8 rate. Each signed nibble v (-8..7) is fed as the FP6 E2M3 code
// u = v + 8 (the nibble with its top bit flipped, 0..15). E2M3 (1 sign, 2
// exponent bits with bias 1, 3 fraction bits) represents code u, 0 <= u < 16,
// as exactly u / 8: codes 0..7 are the subnormals u / 8, codes 8..15 the
// first binade (8 + f) / 8. The MFMA therefore accumulates
//     acc = sum_k u_a u_b / 64 = (sum_k a b + 8 Sa + 8 Sb + 64 K) / 64
// with Sa = sum_k a(i, k) and Sb = sum_k b(k, j), and the exact product sum
// is 64 acc - 8 Sa - 8 Sb - 64 K. Every partial sum of the MFMA is a multiple
// of 1/64 of magnitude at most 225 K / 64, exact in FP32 while 225 K < 2^24:
// the kernel takes K <= 65536. Sa and Sb are summed while converting, with
// the signed 4-bit dot product against all ones (v_dot8_i32_i4).
//
// The conversion is pure bit movement, because a code is just the biased
// nibble placed in a 6-bit field with its two top bits clear. The MFMA
// operand of a lane is a 192-bit string of 32 six-bit fields; any fixed
// assignment of the 32 k of a run to fields works, since A and B use the
// same one. s4_e2m3_16 maps two 32-bit words of nibbles (x, y) to three
// words: x keeps its nibbles 0, 3, 6 / 1, 4, 7 / 2, 5 in place (they already
// sit at 6-bit field offsets 0, 12, 24 / 4, 16, 28 / 8, 20 of the output
// words) and y, rotated left by 2, supplies the fields at offsets 6, 18, 30 /
// 10, 22 (and the two bits of field 5 that cross into the next word) /
// 2, 14, 26. Nine bit operations per 16 values, no table lookups.
//
// Kernel (one wave per SIMD, the schedule of wide_f6.hpp): 256 x 256 tile of
// C per workgroup, 2 x 2 waves of 128 x 128 (4 x 4 blocks of 32 x 32, the
// 256 FP32 accumulators of a lane in its AGPRs, MFMAs as inline assembly
// with the accumulator tied), K in slices of 4 runs (128 k). A slice is
// staged in the run-major E2M3 layout of wide_f6.hpp (P parts of 16 bytes,
// then Q parts of 8 bytes; rows of one run contiguous), 48 KiB, in two LDS
// buffers. Staging: waves 0 and 1 stage A rows 0..127 / 128..255 of the
// tile, waves 2 and 3 the B rows. Lane l stages run l / 16 of panel rows
// 16 i + l % 16 (items i = 0..7): a 16-byte global load (buffer load into
// registers, two slices ahead), the row-sum update, the conversion and one
// 16-byte plus one 8-byte LDS write. Items 4..7 of slice kt + 1 are staged
// during chunk 0 of slice kt, items 0..3 of slice kt + 2 during chunk 1, one
// item per four MFMAs.
//
// Slice kt (buffer kt % 2; chunk c computes on fragment set c):
//   chunk 0: read chunk 1 of slice kt; stage items 4..7 of slice kt + 1 into
//            buffer (kt + 1) % 2 and reload their registers with slice kt + 3;
//   wait for own LDS accesses; barrier (slice kt + 1 complete in LDS, every
//            wave done reading slice kt);
//   chunk 1: read chunk 0 of slice kt + 1; stage items 0..3 of slice kt + 2
//            into buffer kt % 2 and reload their registers with slice kt + 4.
// One barrier per slice. Loads past the end of K re-read the last slice;
// what they stage lands in a buffer nobody reads again, and they do not
// count in the row sums. Needs K a multiple of 256 (an even slice count: the
// loop body covers two slices, whose register sets alternate), 16-byte
// aligned rows; M and N may be ragged (rows past the operands load as zeros
// and their results are not stored).
#pragma once

#include "f6_gemm.hpp"
#include "wide_gemm.hpp"

namespace mpg {

// Biased E2M3 codes of 16 nibbles: x, y hold nibbles 0..7 (low nibble of
// byte 0 first) of two words; o0, o1, o2 receive 16 six-bit fields, field f
// at bits [6 f, 6 f + 6) of the 96-bit string o2:o1:o0. Field f holds the
// code of nibble kI4FieldNibble[f] (0..7: nibble of x, 8..15: nibble - 8 of y).
__host__ __device__ inline void s4_e2m3_16(uint32_t x, uint32_t y, uint32_t &o0, uint32_t &o1, uint32_t &o2) {
    const uint32_t xb = x ^ 0x88888888u, yb = y ^ 0x88888888u;
#if defined(__HIP_DEVICE_COMPILE__)
    const uint32_t yr = __builtin_amdgcn_alignbit(yb, yb, 30);  // rotate left by 2
#else
    const uint32_t yr = (yb << 2) | (yb >> 30);
#endif
    o0 = (xb & 0x0F00F00Fu) | (yr & 0xC03C03C0u);
    o1 = (xb & 0xF00F00F0u) | (yr & 0x03C03C03u);
    o2 = (xb & 0x00F00F00u) | (yr & 0x3C03C03Cu);
}

// Source nibble of each field of s4_e2m3_16 (for the host-side check).
constexpr int kI4FieldNibble[16] = {0, 9, 3, 12, 6, 15, 1, 10, 4, 13, 7, 8, 2, 11, 5, 14};

// One run (16 bytes = 32 nibbles, words w[0..3]) -> the six words of its
// MFMA operand: words 0..3 are the P part, 4..5 the Q part.
__host__ __device__ inline void s4_run_to_e2m3(const uint32_t (&w)[4], uint32_t (&out)[6]) {
    s4_e2m3_16(w[0], w[1], out[0], out[1], out[2]);
    s4_e2m3_16(w[2], w[3], out[3], out[4], out[5]);
}

struct WideI4Cfg {
    static constexpr int BM = 256, BN = 256, J = 4, NTHREADS = 256;
    static constexpr int AP = 0, AQ = J * BM * 16, BP = J * BM * 24, BQ = BP + J * BN * 16;
    static constexpr int STAGE = J * (BM + BN) * 24;  // 48 KiB
    static constexpr int SUMS = 2 * STAGE;            // 512 row sums (A rows, then B rows)
    static constexpr int LDS_BYTES = SUMS + (BM + BN) * 4;
    static constexpr int SLICE_BYTES = J * 16;        // packed bytes of one row per slice
    static constexpr int MAX_K = 65536;               // 225 K < 2^24
    static_assert(LDS_BYTES <= 160 * 1024, "LDS capacity");
};

// 32x32x64 MFMA, E2M3 on both sides (cbsz = blgp = 2), unit scales.
__device__ __forceinline__ void wi4_mfma(const F6Frag &a, const F6Frag &b, f32x16 &c) {
    asm volatile("v_mfma_f32_32x32x64_f8f6f4 %0, %1, %2, %0 cbsz:2 blgp:2" : "+a"(c) : "v"(a), "v"(b));
}

#if defined(__HIP_DEVICE_COMPILE__)
typedef __amdgpu_buffer_rsrc_t wi4_rsrc_t;
#else
typedef i32x4 wi4_rsrc_t;  // the host pass never runs the kernel
#endif

// Staging state of one lane.
struct WI4Stage {
    wi4_rsrc_t rsrc;              // the wave's 128-row panel (rows past the operand: zeros)
    uint32_t voff;                // (l % 16) * pitch + (l / 16) * 16
    int item_step;                // 16 rows: 16 * pitch
    int pw, qw;                   // LDS offsets of item 0 in buffer 0: P and Q parts
};

template <int AUX>
__device__ __forceinline__ i32x4 wi4_gload(const WI4Stage &g, int item, int slice) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_raw_buffer_load_b128(g.rsrc, (int)g.voff,
                                                 item * g.item_step + slice * WideI4Cfg::SLICE_BYTES, AUX);
#else
    return i32x4{};
#endif
}

// Row sum, conversion and LDS writes of one staged item into buffer `buf`.
// `ones` is 0x11111111 for a slice inside K, 0 for a clamped one.
__device__ __forceinline__ void wi4_stage(uint8_t *lds, const WI4Stage &g, int item, int buf, const i32x4 &x,
                                          int &sum, int ones) {
#pragma unroll
    for (int d = 0; d < 4; ++d) sum = __builtin_amdgcn_sdot8(x[d], ones, sum, false);
    uint32_t w[4] = {(uint32_t)x[0], (uint32_t)x[1], (uint32_t)x[2], (uint32_t)x[3]}, o[6];
    s4_run_to_e2m3(w, o);
    uint8_t *b = lds + buf * WideI4Cfg::STAGE;
    *reinterpret_cast<i32x4 *>(b + g.pw + item * 256) = i32x4{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
    *reinterpret_cast<i32x2 *>(b + g.qw + item * 128) = i32x2{(int)o[4], (int)o[5]};
}

// One k-chunk: 16 MFMAs on (a, b); after MFMA 2 f, fragment f of the next set
// (a0 b0 b1 b2 b3 a1 a2 a3); after MFMA 4 q + 3, item I0 + q of the register
// set `regs` (slice s_stage) is staged into buffer `buf` and reloaded with
// slice s_load. The staging waits until at most 15 loads of this wave are
// in flight: the loads are issued in the order they are consumed, four
// items per half slice, and 15 later loads are always outstanding.
template <int I0, int AUX>
__device__ __forceinline__ void wi4_chunk(const F6Frag (&a)[4], const F6Frag (&b)[4], f32x16 (&acc)[4][4],
                                          F6Frag (&na)[4], F6Frag (&nb)[4], uint8_t *lds, int pa, int qa, int pb,
                                          int qb, const WI4Stage &g, i32x4 (&regs)[8], int (&sums)[8], int buf,
                                          int ones, int s_load) {
    static_for<16>([&](auto mm) __attribute__((always_inline)) {
        constexpr int m = decltype(mm)::value;
        __builtin_amdgcn_sched_barrier(0);
        wi4_mfma(a[m / 4], b[m % 4], acc[m / 4][m % 4]);
        if constexpr (m % 2 == 0) {
            constexpr int f = m / 2;
            if constexpr (f == 0) na[0] = f6_frag(lds, pa, qa);
            else if constexpr (f <= 4) nb[f - 1] = f6_frag(lds, pb + (f - 1) * 512, qb + (f - 1) * 256);
            else na[f - 4] = f6_frag(lds, pa + (f - 4) * 512, qa + (f - 4) * 256);
        }
        if constexpr (m % 4 == 3) {
            constexpr int it = I0 + m / 4;
            asm volatile("s_waitcnt vmcnt(15)" ::: "memory");
            wi4_stage(lds, g, it, buf, regs[it], sums[it], ones);
            regs[it] = wi4_gload<AUX>(g, it, s_load);
        }
        __builtin_amdgcn_sched_barrier(0);
    });
}

// A, B: packed INT4 (M rows and N rows of K / 2 bytes), Kb = K / 2. KT = K /
// 128 slices (even, >= 2). PLAIN: raw sums to a row-major int32 C of whole
// 256 x 256 tiles, stored straight from the accumulators; otherwise the
// shared epilogue (ragged edges, scales, zero points).
template <bool PLAIN, int AUX = 0>
__global__ __launch_bounds__(WideI4Cfg::NTHREADS, 1) void wide_i4_gemm(const uint8_t *__restrict__ A,
                                                                      const uint8_t *__restrict__ B,
                                                                      void *__restrict__ Cv, int M, int N, int Kb,
                                                                      int tiles_m, int tiles_n, EpiParams epi) {
    typedef WideI4Cfg T;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[T::LDS_BYTES];
    // consume the epilogue's arguments now: a scalar load still in flight in
    // the loop would turn every LDS wait there into a wait for all
    asm volatile("" ::"s"(Cv), "s"(M), "s"(N));
    if constexpr (!PLAIN)
        asm volatile("" ::"s"(epi.scale_a), "s"(epi.scale_b), "s"(epi.zero_a), "s"(epi.zero_b), "s"(epi.sum_a),
                     "s"(epi.sum_b), "s"(epi.K), "s"(epi.out));
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 31, h = lane >> 5;
    const int wm = wave / 2, wn = wave % 2;
    int tm, tn;
    tile_coords(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, 4, tm, tn);
    const int KT = Kb / T::SLICE_BYTES;

    // staging: wave w < 2 stages A rows [128 w, 128 w + 128) of the tile,
    // w >= 2 the B rows [128 (w - 2), ...)
    WI4Stage g;
    {
        const bool isa = wave < 2;
        const long row0 = isa ? (long)tm * T::BM + wave * 128 : (long)tn * T::BN + (wave - 2) * 128;
        const long rows = isa ? M : N;
        // rows of the panel inside the operand (none for a panel past a ragged edge)
        const long avail = rows - row0 < 0 ? 0 : (rows - row0 < 128 ? rows - row0 : 128);
        const uint8_t *base = (isa ? A : B) + (avail > 0 ? row0 : 0) * Kb;
#if defined(__HIP_DEVICE_COMPILE__)
        g.rsrc = __builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0, (int)(avail * Kb), 0x00020000);
#else
        (void)base;
        g.rsrc = i32x4{};
#endif
        g.voff = (uint32_t)((lane & 15) * Kb + (lane >> 4) * 16);
        g.item_step = 16 * Kb;
        const int prow = (wave & 1) * 128 + (lane & 15), run = lane >> 4;
        g.pw = (isa ? T::AP : T::BP) + (run * 256 + prow) * 16;
        g.qw = (isa ? T::AQ : T::BQ) + (run * 256 + prow) * 8;
    }

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};
    // zeroed accumulators into their AGPRs in order; then the wait a VALU
    // write of a register needs before an MFMA reads it (the compiler does
    // not insert it for the assembly MFMAs)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) asm volatile("" : "+a"(acc[i][j]));
    asm volatile("s_nop 4" ::: "memory");

    // Prologue: loads of slices 0 and 1; stage slice 0 and items 0..3 of
    // slice 1; then the loads that make the steady state: slice 2, items
    // 0..3 of slice 3 (register set = slice parity).
    i32x4 regs[2][8];
    int sums[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    constexpr int ONES = 0x11111111;
#pragma unroll
    for (int i = 0; i < 8; ++i) regs[0][i] = wi4_gload<AUX>(g, i, 0);
#pragma unroll
    for (int i = 0; i < 8; ++i) regs[1][i] = wi4_gload<AUX>(g, i, 1);
    asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
#pragma unroll
    for (int i = 0; i < 8; ++i) wi4_stage(lds, g, i, 0, regs[0][i], sums[i], ONES);
#pragma unroll
    for (int i = 0; i < 4; ++i) wi4_stage(lds, g, i, 1, regs[1][i], sums[i], ONES);
#pragma unroll
    for (int i = 0; i < 8; ++i) regs[0][i] = wi4_gload<AUX>(g, i, min(2, KT - 1));
#pragma unroll
    for (int i = 0; i < 4; ++i) regs[1][i] = wi4_gload<AUX>(g, i, min(3, KT - 1));

    // lane (r, h) reads run 2 kc + h of row 32 i + r of its wave's 128 rows
    const int rowa = h * T::BM + wm * 128 + r, rowb = h * T::BN + wn * 128 + r;
    const int pa0 = T::AP + rowa * 16, qa0 = T::AQ + rowa * 8;
    const int pb0 = T::BP + rowb * 16, qb0 = T::BQ + rowb * 8;
    constexpr int KCP = 2 * T::BM * 16, KCQ = 2 * T::BM * 8;  // next k-chunk: two runs on

    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    F6Frag ra[2][4], rb[2][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) ra[0][i] = f6_frag(lds, pa0 + i * 512, qa0 + i * 256);
#pragma unroll
    for (int j = 0; j < 4; ++j) rb[0][j] = f6_frag(lds, pb0 + j * 512, qb0 + j * 256);
    asm volatile("" ::: "memory");  // keeps the reads above the wait
    __builtin_amdgcn_s_waitcnt(0xC07F);

    // Two slices per iteration (register sets alternate with slice parity).
    for (int kt = 0; kt < KT; kt += 2) {
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const int s = kt + p;
            const int cur = p * T::STAGE, nxt = (1 - p) * T::STAGE;
            // items 4..7 of slice s + 1 (register set 1 - p)
            const int ones1 = s + 1 < KT ? ONES : 0;
            wi4_chunk<4, AUX>(ra[0], rb[0], acc, ra[1], rb[1], lds, pa0 + cur + KCP, qa0 + cur + KCQ,
                              pb0 + cur + KCP, qb0 + cur + KCQ, g, regs[1 - p], sums, 1 - p, ones1,
                              min(s + 3, KT - 1));
            asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
            // items 0..3 of slice s + 2 (register set p)
            const int ones2 = s + 2 < KT ? ONES : 0;
            wi4_chunk<0, AUX>(ra[1], rb[1], acc, ra[0], rb[0], lds, pa0 + nxt, qa0 + nxt, pb0 + nxt, qb0 + nxt, g,
                              regs[p], sums, p, ones2, min(s + 4, KT - 1));
        }
    }
    // Clamped loads may still be in flight. The last MFMA results: an XDL
    // op of P passes (P = 8 for 32x32x64 FP6) needs P + 3 wait states before
    // a VALU or memory instruction reads its destination; the nops give 40.
    // The empty asm statements then order every read of the accumulators
    // after the nops.
    asm volatile("s_waitcnt vmcnt(0)\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) asm volatile("" : "+a"(acc[i][j]));

    // Row sums: the four lanes l % 16 + 16 c of an item cover its row's four
    // runs; then lanes 0..15 publish their eight rows.
    int *sum_lds = reinterpret_cast<int *>(lds + T::SUMS);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        sums[i] += __shfl_xor(sums[i], 16, 64);
        sums[i] += __shfl_xor(sums[i], 32, 64);
    }
    if (lane < 16) {
        const int base = (wave < 2 ? 0 : T::BM) + (wave & 1) * 128 + lane;
#pragma unroll
        for (int i = 0; i < 8; ++i) sum_lds[base + 16 * i] = sums[i];
    }
    __syncthreads();

    // exact sum = 64 acc - 8 Sa - 8 Sb - 64 K: with ta = 8 Sa + 64 K (per row)
    // and tb = 8 Sb (per column), fma(acc, 64, -ta) - tb in FP32 is exact
    // (every term and result is an integer of magnitude below 2^24)
    const int K = Kb * 2;
    float tb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) tb[j] = (float)(8 * sum_lds[T::BM + wn * 128 + 32 * j + r]);
    const long row0 = (long)tm * T::BM + wm * 128;
    const long col0 = (long)tn * T::BN + wn * 128 + r;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            // rows 32 i + 8 q + 4 h + (0..3) of the wave's 128: four consecutive sums
            const i32x4 sa = *reinterpret_cast<const i32x4 *>(sum_lds + wm * 128 + 32 * i + 8 * q + 4 * h);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float nta = -(float)(8 * sa[e] + 64 * K);
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j][4 * q + e] = __builtin_fmaf(acc[i][j][4 * q + e], 64.0f, nta) - tb[j];
            }
        }
    if constexpr (PLAIN) {
        // element (i, j, v): row row0 + 32 i + 8 (v / 4) + 4 h + v % 4, column col0 + 32 j
        int32_t *base = reinterpret_cast<int32_t *>(Cv) + (row0 + 4 * h) * (long)N + col0;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                int32_t *rowp = base + (long)(32 * i + 8 * (v / 4) + v % 4) * N;
#pragma unroll
                for (int j = 0; j < 4; ++j) rowp[32 * j] = (int)acc[i][j][v];
            }
    } else {
        epi_store_tile<S4, 32, 4, 4, 16>(epi, Cv, acc, row0, col0, h, M, N, ConvToInt());
    }
}

}  // namespace mpg
