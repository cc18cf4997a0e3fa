// generic_gemm.hpp - bounds-checked MFMA kernel for any M, N, K and any
// element-aligned pointers.
//
// One wave computes one 32x32 block of C. Each K-step every lane gathers its
// operand run straight from global memory with per-element bounds checks
// (out-of-range elements read as zero, which adds nothing to the sums), then
// issues one MFMA (FP16, INT8) or one MFMA on exactly sign-extended INT4
// values. Stores are bounds-checked too. This kernel carries the ragged edges
// and unaligned operands the tiled kernels do not accept; it also serves K = 0
// (no K-steps: C is written with zeros).
#pragma once

#include "device_common.hpp"

namespace mpg {

template <int DT>
__global__ __launch_bounds__(64) void generic_gemm(const uint8_t *__restrict__ A,
                                                   const uint8_t *__restrict__ B,
                                                   void *__restrict__ Cv, int M, int N, int K,
                                                   int tiles_n, EpiParams epi) {
    typedef typename Acc<DT>::type acc_t;
    const int lane = threadIdx.x;
    const int r = lane & 31, h = lane >> 5;
    const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
    const long row = (long)tm * 32 + r;  // A row this lane feeds
    const long col = (long)tn * 32 + r;  // B column this lane feeds
    const bool row_ok = row < M, col_ok = col < N;
    acc_t acc = {};

    if constexpr (DT == F16) {
        const _Float16 *a = reinterpret_cast<const _Float16 *>(A) + (row_ok ? row : 0) * K;
        const _Float16 *b = reinterpret_cast<const _Float16 *>(B) + (col_ok ? col : 0) * K;
        for (int k0 = 0; k0 < K; k0 += 16) {
            half8 av, bv;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int k = k0 + 8 * h + e;
                av[e] = (row_ok && k < K) ? a[k] : (_Float16)0;
                bv[e] = (col_ok && k < K) ? b[k] : (_Float16)0;
            }
            acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, bv, acc, 0, 0, 0);
        }
    } else {
        const long pitch = (DT == S8) ? (long)K : (long)K / 2;
        const uint8_t *a = A + (row_ok ? row : 0) * pitch;
        const uint8_t *b = B + (col_ok ? col : 0) * pitch;
        for (int k0 = 0; k0 < K; k0 += 32) {
            i32x4 av = {0, 0, 0, 0}, bv = {0, 0, 0, 0};
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int k = k0 + 16 * h + e;
                int va = 0, vb = 0;
                if (k < K) {
                    if constexpr (DT == S8) {
                        va = row_ok ? (int)(int8_t)a[k] : 0;
                        vb = col_ok ? (int)(int8_t)b[k] : 0;
                    } else {
                        va = row_ok ? s4_nibble(a[k >> 1], k & 1) : 0;
                        vb = col_ok ? s4_nibble(b[k >> 1], k & 1) : 0;
                    }
                }
                av[e >> 2] |= (int)((uint32_t)(va & 0xFF) << (8 * (e & 3)));
                bv[e >> 2] |= (int)((uint32_t)(vb & 0xFF) << (8 * (e & 3)));
            }
            acc = mfma_i8(av, bv, acc);
        }
    }

    const long ccol = (long)tn * 32 + r;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const long crow = (long)tm * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
        if (crow < M && ccol < N) epi_store_one<DT>(epi, Cv, crow, ccol, N, acc[v]);
    }
}

}  // namespace mpg
