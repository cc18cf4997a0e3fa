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

#include <type_traits>
#include <utility>

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
// stored at slot c ^ swz(q). An MFMA operand fetch reads one chunk index of 32
// consecutive rows (16 bytes per lane). 128-byte rows: rows 8 apart get
// different slots, which keeps every 8 consecutive lanes on distinct 16-byte
// bank groups (no bank conflicts counted by SQ_LDS_BANK_CONFLICT). 64-byte
// rows: the swizzle was chosen by measurement on MI355X among the functions
// ((q >> a) ^ (q >> b)) & 3: this one reads at the conflict-free rate of the
// 128-byte layout, while ((q >> 1) ^ (q >> 3)) & 3, conflict-free for 16
// consecutive lanes on paper, reads 1.75x slower.
template <int CH> __host__ __device__ constexpr int swz(int q) {
    if constexpr (CH == 8) return (q ^ (q >> 3)) & 7;
    else if constexpr (CH == 4) return ((q >> 3) ^ (q >> 4)) & 3;
    else return 0;
}

// ---------------------------------------------------------------------------
// Output stage shared by every GEMM kernel. OUT_PLAIN stores the raw sum (FP32
// for FP16 inputs, INT32 otherwise). The scaled outputs compute, per element,
//   sa[i] * sb[j] * sum_k (A(i,k) - za[i]) (B(k,j) - zb[j])
// (absent scales are 1, absent zero points 0; zero points only for integer
// inputs) and store it as FP32, FP16 or BF16, rounded to nearest even. The
// zero-point terms use the row sums of A and column sums of B:
//   sum (a - za)(b - zb) = sum ab - zb * rowsum_a - za * colsum_b + K za zb,
// evaluated exactly in 64-bit integers, then converted to FP32 once and
// multiplied by the scales in FP32.
enum Out : int { OUT_PLAIN = 0, OUT_F32 = 1, OUT_F16 = 2, OUT_BF16 = 3 };

struct EpiParams {
    const float *scale_a;  // M values or null
    const float *scale_b;  // N values or null
    const int *zero_a;     // M values or null
    const int *zero_b;     // N values or null
    const int *sum_a;      // row sums of A (used with zero_b)
    const int *sum_b;      // column sums of B (used with zero_a)
    int K;
    int out;
};

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __builtin_bit_cast(uint32_t, f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);  // NaN stays NaN
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ void store_out(const EpiParams &e, void *C, long idx, float v) {
    if (e.out == OUT_F32) reinterpret_cast<float *>(C)[idx] = v;
    else if (e.out == OUT_F16) reinterpret_cast<_Float16 *>(C)[idx] = (_Float16)v;
    else reinterpret_cast<uint16_t *>(C)[idx] = f32_to_bf16_rne(v);
}

// Scaled value of one raw sum x (float for FP16 inputs, int otherwise) at
// row i, column j, with the column terms of j preloaded.
template <int DT, class V>
__device__ __forceinline__ float epi_value(const EpiParams &e, V x, long i, float sb, long long zb,
                                           long long cs) {
    float v;
    if constexpr (DT == F16) {
        v = x;
    } else {
        long long c = x;
        const long long za = e.zero_a ? e.zero_a[i] : 0;
        if (e.zero_b) c -= zb * (long long)e.sum_a[i];
        if (e.zero_a) c -= za * cs - (long long)e.K * za * zb;
        v = (float)c;
    }
    if (e.scale_a) v *= e.scale_a[i];
    return v * sb;
}

// One element (the bounds-checked kernel).
template <int DT, class V>
__device__ __forceinline__ void epi_store_one(const EpiParams &e, void *C, long i, long j, long N, V x) {
    if (e.out == OUT_PLAIN) {
        reinterpret_cast<V *>(C)[i * N + j] = x;
        return;
    }
    const float sb = e.scale_b ? e.scale_b[j] : 1.0f;
    const long long zb = e.zero_b ? e.zero_b[j] : 0, cs = e.zero_a ? e.sum_b[j] : 0;
    store_out(e, C, i * N + j, epi_value<DT>(e, x, i, sb, zb, cs));
}

// Calls f(integral_constant<int, I>) for I = 0 .. N-1, unrolled by
// construction. The epilogue indexes the accumulator arrays only through
// such compile-time indices: a loop the unroller declines (it does for the
// scaled path of a 128 x 128 wave tile) would index them at run time and
// move every accumulator to scratch memory.
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F &&f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// A wave's MS x MS blocks (FM x FN of them): block (i, j) value v of lane
// group h sits at row row0 + i MS + acc_row(h, v), column col0 + j MS (col0
// includes the lane's column). conv maps an accumulator element to the raw
// sum. Rows >= M and columns >= N are not stored.
template <int DT, int MS, int FM, int FN, int NV, class AccT, class Conv>
__device__ __forceinline__ void epi_store_tile(const EpiParams &e, void *C, const AccT (&acc)[FM][FN],
                                               long row0, long col0, int h, int M, int N, Conv conv) {
    typedef typename Acc<DT, MS>::out out_t;
    if (e.out == OUT_PLAIN) {
        out_t *Co = reinterpret_cast<out_t *>(C);
        static_for<FM>([&](auto i) __attribute__((always_inline)) {
            static_for<FN>([&](auto j) __attribute__((always_inline)) {
                static_for<NV>([&](auto v) __attribute__((always_inline)) {
                    const long row = row0 + i * MS + acc_row<MS>(h, v), col = col0 + j * MS;
                    if (row < M && col < N) Co[row * N + col] = conv(acc[i][j][v.value]);
                });
            });
        });
        return;
    }
    float sb[FN];
    long long zb[FN], cs[FN];
    static_for<FN>([&](auto j) __attribute__((always_inline)) {
        const long col = col0 + j * MS;
        const bool ok = col < N;
        sb[j] = (e.scale_b && ok) ? e.scale_b[col] : 1.0f;
        zb[j] = (e.zero_b && ok) ? e.zero_b[col] : 0;
        cs[j] = (e.zero_a && ok) ? e.sum_b[col] : 0;
    });
    static_for<FM>([&](auto i) __attribute__((always_inline)) {
        static_for<NV>([&](auto v) __attribute__((always_inline)) {
            const long row = row0 + i * MS + acc_row<MS>(h, v);
            if (row < M) {
                static_for<FN>([&](auto j) __attribute__((always_inline)) {
                    const long col = col0 + j * MS;
                    if (col < N)
                        store_out(e, C, row * N + col,
                                  epi_value<DT>(e, conv(acc[i][j][v.value]), row, sb[j], zb[j], cs[j]));
                });
            }
        });
    });
}

// Accumulator element -> raw sum.
struct ConvSame {
    template <class X> __device__ __forceinline__ X operator()(X x) const { return x; }
};
struct ConvShift8 {  // INT4 on the INT8 MFMA: the sums are carried times 256
    __device__ __forceinline__ int operator()(int x) const { return x >> 8; }
};
struct ConvToInt {  // INT4 on the FP6 MFMA: exact integers held in FP32
    __device__ __forceinline__ int operator()(float x) const { return (int)x; }
};

// Row sums of an integer operand stored as R rows of K values (int8 bytes or
// packed INT4 nibbles), one block per row; used by the zero-point terms.
template <int DT>
__global__ __launch_bounds__(256) void row_sums(const uint8_t *__restrict__ X, int R, int K,
                                                int *__restrict__ out) {
    __shared__ int part[4];
    const long kb = row_bytes(DT, K);
    const uint8_t *row = X + (size_t)blockIdx.x * kb;
    int s = 0;
    for (long b = threadIdx.x; b < kb; b += 256) {
        const uint32_t byte = row[b];
        if constexpr (DT == S8) s += (int)(int8_t)byte;
        else s += s4_nibble(byte, 0) + s4_nibble(byte, 1);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) out[blockIdx.x] = part[0] + part[1] + part[2] + part[3];
}

// Rank of workgroup `id` of `n` in an order where each XCD owns a
// contiguous run: workgroups are dispatched round-robin over the 8 XCDs,
// each with its own L2, so ids id, id + 8, ... share one. XCD x runs
// n / 8 workgroups, one more when x < n % 8; its run starts after the runs
// of XCDs 0 .. x - 1 (a bijection on 0 .. n - 1).
__device__ __forceinline__ int xcd_rank(int id, int n) {
    const int x = id & 7, j = id >> 3, q = n >> 3, r = n & 7;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
}

// Linear tile index -> (tile row, tile column), walking group_m tile rows
// at a time so that consecutive indices share A row panels and B column
// panels.
__device__ __forceinline__ void grouped_tile(int t, int tiles_m, int tiles_n, int group_m, int &tm, int &tn) {
    const int width = group_m * tiles_n;
    const int group = t / width;
    const int first_m = group * group_m;
    const int gsize = min(tiles_m - first_m, group_m);
    const int in_group = t - group * width;
    tm = first_m + in_group % gsize;
    tn = in_group / gsize;
}

// Workgroup id -> (tile row, tile column): XCD-contiguous ranks in grouped
// order, so the workgroups that run together on one XCD share panels.
__device__ __forceinline__ void tile_coords(int pid, int ntiles, int tiles_m, int tiles_n,
                                            int group_m, int &tm, int &tn) {
    grouped_tile(xcd_rank(pid, ntiles), tiles_m, tiles_n, group_m, tm, tn);
}

}  // namespace mpg
