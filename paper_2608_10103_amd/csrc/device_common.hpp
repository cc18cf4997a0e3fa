// device_common.hpp - types and per-precision MFMA steps shared by the kernels.
//
// All three precisions feed 32x32 MFMA blocks from 16-byte operand runs: each
// lane supplies one 16-byte run of one A row and one B column (both
// K-contiguous, the paper's ".row.col" operand order). Lane l of a wave owns
// row/column (l % 32) of the block and K-half (l / 32) of the run pair:
//   FP16: v_mfma_f32_32x32x16_f16, 8 binary16 values per lane per operand;
//   INT8: v_mfma_i32_32x32x32_i8, 16 int8 values per lane per operand;
//   INT4: 16 packed bytes per lane = 32 nibbles, decoded to two int8 runs that
//         feed two v_mfma_i32_32x32x32_i8 (gfx950 has no 4-bit integer MFMA).
// The hardware pairs element e of A-lane (i + 32h) with element e of B-lane
// (j + 32h); as long as A and B put the same k at the same (h, e), the MFMA
// computes sum_k A(i,k) B(k,j) whatever the k order, exactly for integers.
//
// Accumulator layout of a 32x32 block (16 values per lane): value v of lane l
// holds C[8*(v/4) + 4*(l/32) + (v%4)][l % 32].
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mpg {

enum Dtype : int { F16 = 0, S8 = 1, S4 = 2 };

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

// Accumulator of one MS x MS MFMA block (MS = 32: 16 values per lane, MS =
// 16: 4 values per lane) and the output element type.
template <int DT, int MS = 32> struct Acc;
template <> struct Acc<F16, 32> { typedef f32x16 type; typedef float out; };
template <> struct Acc<S8, 32> { typedef i32x16 type; typedef int32_t out; };
template <> struct Acc<S4, 32> { typedef i32x16 type; typedef int32_t out; };
template <> struct Acc<F16, 16> { typedef f32x4 type; typedef float out; };
template <> struct Acc<S8, 16> { typedef i32x4 type; typedef int32_t out; };
template <> struct Acc<S4, 16> { typedef i32x4 type; typedef int32_t out; };

// Row within an MS x MS block of accumulator value v of a lane in lane group
// h (= lane / MS); the column is lane % MS. 32x32: value v covers row
// 8 (v / 4) + 4 h + v % 4; 16x16: row 4 h + v.
template <int MS>
__device__ __forceinline__ constexpr int acc_row(int h, int v) {
    return MS == 32 ? 8 * (v >> 2) + 4 * h + (v & 3) : 4 * h + v;
}

// Bytes of one element in storage: FP16 2, INT8 1; INT4 is handled as bytes of
// two nibbles, so the row pitch in bytes is K/2.
__host__ __device__ constexpr long row_bytes(int dt, long K) {
    return dt == F16 ? 2 * K : (dt == S8 ? K : K / 2);
}

__device__ __forceinline__ f32x16 mfma_f16(i32x4 a, i32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, a),
                                                   __builtin_bit_cast(half8, b), c, 0, 0, 0);
}

__device__ __forceinline__ i32x16 mfma_i8(i32x4 a, i32x4 b, i32x16 c) {
    return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}

// 16x16 blocks: v_mfma_f32_16x16x32_f16 and v_mfma_i32_16x16x64_i8 take the
// same 16-byte operand run per lane; lane l owns row/column l % 16 and K-group
// l / 16 of four.
__device__ __forceinline__ f32x4 mfma_f16(i32x4 a, i32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8, a),
                                                   __builtin_bit_cast(half8, b), c, 0, 0, 0);
}

__device__ __forceinline__ i32x4 mfma_i8(i32x4 a, i32x4 b, i32x4 c) {
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// INT4 decode for the tiled kernels, four bytes (eight nibbles) per 32-bit
// word. The low nibble of each byte is moved to the byte's top half and the
// high nibble kept there, the other half cleared: the resulting int8 is 16*v
// for the nibble's two's-complement value v, exactly. Both operands are
// scaled the same way, so the MFMA sums 256 * a * b and the epilogue shifts
// right by 8 (exact: the sum is a multiple of 256 and |256 * C| < 2^31 while
// K < 131072).
__device__ __forceinline__ i32x4 s4_lo_x16(i32x4 x) {
    i32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = (int)(((uint32_t)x[e] << 4) & 0xF0F0F0F0u);
    return r;
}
__device__ __forceinline__ i32x4 s4_hi_x16(i32x4 x) {
    i32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = (int)((uint32_t)x[e] & 0xF0F0F0F0u);
    return r;
}

// Exact signed value of nibble `which` (0 low, 1 high) of a byte, for the
// bounds-checked kernel: (n ^ 8) - 8 maps 0..7 to 0..7 and 8..15 to -8..-1.
__device__ __forceinline__ int s4_nibble(uint32_t byte, int which) {
    uint32_t n = which ? (byte >> 4) : (byte & 0xFu);
    return (int)(n ^ 8u) - 8;
}

// LDS swizzle: in a tile of rows of CH 16-byte chunks, chunk c of row q is
// stored at slot c ^ swz(q). Chosen so that the 16-byte reads of 32
// consecutive rows at one chunk index (what one MFMA operand fetch does) hit
// distinct bank groups both in 8-lane (128-byte) and 16-lane (256-byte)
// service groups.
template <int CH> __host__ __device__ constexpr int swz(int q) {
    if constexpr (CH == 8) return (q ^ (q >> 3)) & 7;
    else if constexpr (CH == 4) return ((q >> 1) ^ (q >> 3)) & 3;
    else return 0;
}

// Workgroup id -> (tile row, tile column). Workgroups are dispatched
// round-robin over the 8 XCDs, each with its own L2; ids are first regrouped
// so each XCD owns a contiguous run of the ordering, and the ordering walks
// group_m tile rows at a time so concurrently running tiles share A row
// panels and B column panels.
__device__ __forceinline__ void tile_coords(int pid, int ntiles, int tiles_m, int tiles_n,
                                            int group_m, int &tm, int &tn) {
    if ((ntiles & 7) == 0) pid = (pid & 7) * (ntiles >> 3) + (pid >> 3);
    const int width = group_m * tiles_n;
    const int group = pid / width;
    const int first_m = group * group_m;
    const int gsize = min(tiles_m - first_m, group_m);
    const int in_group = pid - group * width;
    tm = first_m + in_group % gsize;
    tn = in_group / gsize;
}

}  // namespace mpg
