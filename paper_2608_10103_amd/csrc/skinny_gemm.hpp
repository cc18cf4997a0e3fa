// skinny_gemm.hpp - GEMMs with at most 16 * MB rows on one side (LLM
// decoding: a few tokens times a weight matrix).
//
// Such a product is bound by streaming the large operand once from HBM; the
// tiled kernels pad the small side to a 128-row tile and finish each tile's
// K range too quickly for their pipeline to reach full bandwidth. This kernel
// streams instead:
//
//  * The small operand ("X": R <= 16 MB rows of K, K-contiguous) is padded to
//    16-row blocks, read from L2 straight into registers.
//  * The large operand ("W": Q rows of K, K-contiguous) is split into groups
//    of 16 * NB rows, one workgroup per group; the 8 waves of a workgroup split
//    K eight ways. A wave loads its W rows from global memory into registers,
//    DEPTH 64-byte K-steps ahead of the MFMAs (no LDS staging: every W byte is
//    used by exactly one wave), so each CU keeps 8 x DEPTH x NB KiB of W in
//    flight.
//  * 16x16 MFMAs (v_mfma_f32_16x16x32_f16, v_mfma_i32_16x16x64_i8; INT4
//    decoded to int8 in registers as in the tiled kernels) consume one
//    64-byte K-step of every row per instruction.
//  * The eight partial blocks are summed in LDS in wave order (the result
//    does not depend on timing) and stored through the shared epilogue.
//
// Both operands are K-contiguous, so the kernel serves either side: X = A
// (rows of C) when M is small, or X = B (columns of C) when N is small, with
// the output transposed on store.
#pragma once

#include "device_common.hpp"

namespace mpg {

template <int DT>
struct SkinnyAcc {
    typedef typename Acc<DT, 16>::type type;
    typedef typename Acc<DT, 16>::out out;
};

// 16x16 MFMA step on one 16-byte run per lane of each operand (INT4: 32
// nibbles, two MFMAs, sums carried times 256).
template <int DT>
__device__ __forceinline__ void skinny_mma(i32x4 x, i32x4 w, typename SkinnyAcc<DT>::type &acc) {
    if constexpr (DT == F16) {
        acc = mfma_f16(x, w, acc);
    } else if constexpr (DT == S8) {
        acc = mfma_i8(x, w, acc);
    } else {
        acc = mfma_i8(s4_lo_x16(x), s4_lo_x16(w), acc);
        acc = mfma_i8(s4_hi_x16(x), s4_hi_x16(w), acc);
    }
}

constexpr int SKINNY_WAVES = 8;
constexpr int SKINNY_DEPTH = 4;  // default K-steps loaded ahead of the MFMAs

// X: R rows (R <= 16 * MB), W: Q rows, both of Kb bytes (Kb a multiple of
// 64). Workgroup g covers W rows [16 NB g, 16 NB (g + 1)). Output element
// (x-row r, w-row q) goes to C(r, q) if trans == 0, C(q, r) otherwise, C
// being row-major with `ldc` columns.
template <int DT, int MB, int NB, int D = SKINNY_DEPTH>
__global__ __launch_bounds__(64 * SKINNY_WAVES, 1) void skinny_gemm(const uint8_t *__restrict__ X,
                                                                   const uint8_t *__restrict__ W,
                                                                   void *__restrict__ Cv, int R, int Q,
                                                                   int Kb, int ldc, int trans,
                                                                   EpiParams epi) {
    typedef typename SkinnyAcc<DT>::type acc_t;
    typedef typename SkinnyAcc<DT>::out out_t;
    constexpr int NV = 4;  // accumulator values per lane of a 16x16 block
    __shared__ __attribute__((aligned(16))) out_t part[SKINNY_WAVES][MB * NB][NV * 64];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r16 = lane & 15, kg = lane >> 4;  // row within a block, 16-byte group of the step
    const int q0 = blockIdx.x * 16 * NB;

    // this wave's K-steps [s0, s1) of 64 bytes
    const int steps = Kb >> 6;
    const int s0 = (int)((long)steps * wave / SKINNY_WAVES);
    const int s1 = (int)((long)steps * (wave + 1) / SKINNY_WAVES);

    // Row pointers (rows past the data clamped to the last one: their
    // results are never stored) at this lane's 16-byte group of step s0.
    const uint8_t *xp[MB], *wp[NB];
#pragma unroll
    for (int i = 0; i < MB; ++i) xp[i] = X + (size_t)min(16 * i + r16, R - 1) * Kb + (size_t)s0 * 64 + kg * 16;
#pragma unroll
    for (int j = 0; j < NB; ++j) wp[j] = W + (size_t)min(q0 + 16 * j + r16, Q - 1) * Kb + (size_t)s0 * 64 + kg * 16;

    acc_t acc[MB][NB];
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) acc[i][j] = acc_t{};

    // Groups of D steps, double-buffered; loads past s1 re-read the wave's
    // last step (in bounds) and their MFMAs are skipped.
    const int n = s1 - s0;
    if (n > 0) {
        i32x4 xb[2][D][MB], wb[2][D][NB];
        auto load = [&](int buf, int g) __attribute__((always_inline)) {
#pragma unroll
            for (int d = 0; d < D; ++d) {
                const size_t off = (size_t)min(g * D + d, n - 1) * 64;
#pragma unroll
                for (int j = 0; j < NB; ++j) wb[buf][d][j] = *reinterpret_cast<const i32x4 *>(wp[j] + off);
#pragma unroll
                for (int i = 0; i < MB; ++i) xb[buf][d][i] = *reinterpret_cast<const i32x4 *>(xp[i] + off);
            }
        };
        auto compute = [&](int buf, int g) __attribute__((always_inline)) {
#pragma unroll
            for (int d = 0; d < D; ++d) {
                if (g * D + d < n) {
#pragma unroll
                    for (int i = 0; i < MB; ++i)
#pragma unroll
                        for (int j = 0; j < NB; ++j) skinny_mma<DT>(xb[buf][d][i], wb[buf][d][j], acc[i][j]);
                }
            }
        };
        const int G = (n + D - 1) / D;
        load(0, 0);
        int g = 0;
        for (; g + 2 <= G; g += 2) {
            load(1, g + 1);
            compute(0, g);
            load(0, min(g + 2, G - 1));
            compute(1, g + 1);
        }
        if (g < G) compute(0, g);
    }

    // Partial blocks to LDS, summed in wave order by the workgroup.
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int v = 0; v < NV; ++v) part[wave][i * NB + j][v * 64 + lane] = (out_t)acc[i][j][v];
    __syncthreads();
    // Element e of the workgroup's (16 MB) x (16 NB) block: block b = e / 256,
    // accumulator value v and lane l inside it.
    for (int e = tid; e < MB * NB * 256; e += 64 * SKINNY_WAVES) {
        const int b = e >> 8, v = (e >> 6) & 3, l = e & 63;
        out_t s = part[0][b][v * 64 + l];
#pragma unroll
        for (int w = 1; w < SKINNY_WAVES; ++w) s += part[w][b][v * 64 + l];
        if constexpr (DT == S4) s >>= 8;  // INT4 sums carried times 256
        const int i = b / NB, j = b % NB;
        const int r = 16 * i + acc_row<16>(l >> 4, v);  // x-row
        const int q = q0 + 16 * j + (l & 15);           // w-row
        if (r < R && q < Q) {
            if (trans) epi_store_one<DT>(epi, Cv, q, r, ldc, s);
            else epi_store_one<DT>(epi, Cv, r, q, ldc, s);
        }
    }
}

}  // namespace mpg
