// tposeb_gemm.hpp - B stored K x N row-major (N-contiguous): the paper's
// "transposed B" operand layout (its INT4 ablation, Table XII), on CDNA4.
//
// On the paper's GPU this layout made every B load uncoalesced and cost 3x.
// Here B is copied into LDS exactly as it lies in memory (whole K-rows of
// N-contiguous bytes, the same 16-byte direct-to-LDS loads as A), and the
// MFMA operand, which wants K-contiguous runs per column, is assembled by the
// LDS transpose reads of gfx950 (ds_read_b64_tr_b16 / _b8 / _b4). Measured
// lane layout of those reads, per group of 16 lanes: lanes 4e..4e+3 (b16),
// 2e, 2e+1 (b8) or e (b4) supply row e (16 consecutive elements, 8 bytes per
// lane); output lane i receives element i of every row, i.e. 4 (b16), 8 (b8)
// or 16 (b4, row e in nibble e) elements of column i along the row index.
// With the rows being consecutive k of one 16-column slice, each lane gets
// consecutive k of its own column: the MFMA operand run, two reads per
// 32-column block per K-chunk. For INT4 (B's nibbles packed along N, the
// low nibble holding the even column) the two reads give 32 consecutive k
// packed two per byte with the low nibble holding the even k, the layout of
// a column-major INT4 run, so the decode and MFMAs are the column-major
// kernel's.
//
// Everything else is the 8-wave pipelined kernel of tiled_gemm.hpp: 256 x 256
// tile, 2 x 4 waves of 128 x 64, 128-byte K-slices of A (BKB / es k-rows of
// B) in a 2-stage ring, operand runs double-buffered in registers, the
// barrier inside the last K-chunk. FP16, INT8 and INT4. N must fill whole
// tiles (the copy takes whole B rows of the tile), K whole slices; M may be
// ragged.
#pragma once

#include "tiled_gemm.hpp"

namespace mpg {

template <int DT, class T>
struct TB {
    static_assert(T::MS == 32 && T::BKB == 128 && T::STAGES == 2, "the 128-byte 2-stage pipelined tile");
    static constexpr int EPB2 = DT == F16 ? 1 : (DT == S8 ? 2 : 4);  // elements per 2 bytes
    static constexpr int BK = T::BKB * EPB2 / 2;         // k per slice = B rows per stage
    static constexpr int RB = T::BN * 2 / EPB2;          // bytes of one B row in the tile
    static constexpr int CHB = RB / 16;                  // 16-byte chunks per B row
    static constexpr int ROWS_PER_UNIT = 1024 / RB;      // B rows one 1 KiB copy fills
    static constexpr int A_UNITS = T::BM * T::BKB / 1024;
    static constexpr int RR = 4 * EPB2;                  // B rows per transpose read: 4, 8, 16
    static constexpr int LPR = 16 / RR;                  // lanes per row in a 16-lane group
    // byte offset of column j within a B row
    static __host__ __device__ constexpr long col_bytes(long j) { return j * 2 / EPB2; }
    static_assert(A_UNITS % T::DMA_PER_WAVE == 0, "a wave copies only A or only B");
    static_assert(BK * RB == T::BN * T::BKB, "B part of a stage is as large as the column-major one");
};

// Slot of 16-byte chunk c of B row r (row r of the stage's B part). The 16
// lanes of a transpose read take RR consecutive rows of one 16-column slice
// (32 bytes per row for FP16, 16 for INT8); rows of 512 (FP16) or 256 (INT8)
// bytes all start on the same bank, so the chunks are spread by row: the two
// 16-lane groups that read one 32-column block hit 16 distinct 16-byte bank
// groups.
// INT4: rows of 128 bytes, a read's 16 lanes take 16 consecutive rows of one
// 8-byte column group; rows r and r + 1 start on opposite halves of the
// 256-byte bank row, so slot (r / 2) % 8 spreads the 16 rows over 16 distinct
// 8-byte bank pairs.
template <int DT>
__host__ __device__ constexpr int tb_swz(int r) {
    return DT == F16 ? 4 * (r & 3) : (DT == S8 ? 2 * (r & 7) : (r >> 1) & 7);
}

// Copy unit d of a stage for lane `lane`: A units as in the pipelined kernel;
// B unit u (d = A_UNITS + u) takes B rows kt * BK + u * ROWS_PER_UNIT + ...,
// chunk slot lane % CHB holding logical chunk slot ^ tb_swz(row). Returns the
// source at slice 0; the per-slice advance is tb_stride().
template <int DT, class T>
__device__ __forceinline__ const uint8_t *tb_src(const uint8_t *A, const uint8_t *B, int M, int N,
                                                 int Kb, int tm, int tn, int d, int lane) {
    typedef TB<DT, T> P;
    if (d < P::A_UNITS) return stage_src<T>(A, B, M, N, Kb, tm, tn, d, lane);
    const int u = d - P::A_UNITS;
    const int r = u * P::ROWS_PER_UNIT + lane / P::CHB;  // B row within the stage
    const int c = (lane % P::CHB) ^ tb_swz<DT>(r);
    return B + (size_t)r * P::col_bytes(N) + (size_t)tn * P::RB + c * 16;
}

// One K-chunk's operand runs: A by ds_read_b128 (as load_runs), B by two
// transpose reads per 32-column block.
template <int DT, class T>
__device__ __forceinline__ void tb_load_runs(const uint8_t *st, int kc, int wm, int wn, int lane,
                                             i32x4 (&a)[T::FM], i32x4 (&b)[T::FN]) {
    typedef TB<DT, T> P;
    const int r = lane % T::MS, h = lane / T::MS;
#pragma unroll
    for (int i = 0; i < T::FM; ++i) {
        const int q = wm * T::WTM + i * T::MS + r;
        a[i] = *reinterpret_cast<const i32x4 *>(st + q * T::BKB + (((T::G * kc + h) ^ swz<T::CH>(q)) << 4));
    }
    const uint8_t *sb = st + T::BM * T::BKB;  // B part of the stage
    const int g = lane >> 4, j16 = lane & 15;
#pragma unroll
    for (int j = 0; j < T::FN; ++j) {
        const int col = wn * T::WTN + j * T::MS + 16 * (g & 1);  // first column of the group
        const int byte = (int)P::col_bytes(col) + (j16 % P::LPR) * 8;  // this lane's 8 bytes in the row
        i32x4 v;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            // k rows of this read: chunk kc's 16 (FP16) / 32 (INT8) / 64 (INT4) k, half g / 2, part t
            const int row = kc * (2 * 2 * P::RR) + (g >> 1) * (2 * P::RR) + t * P::RR + j16 / P::LPR;
            const uint8_t *p = sb + row * P::RB + ((((byte >> 4) ^ tb_swz<DT>(row))) << 4) + (byte & 15);
            typedef __attribute__((address_space(3))) void lds_void_t;
            if constexpr (DT == F16) {
                typedef short v4s __attribute__((ext_vector_type(4)));
                typedef __attribute__((address_space(3))) v4s lds_v4s;
                const v4s x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s *)(lds_void_t *)p);
                const uint64_t u = __builtin_bit_cast(uint64_t, x);
                v[2 * t] = (int)(uint32_t)u;
                v[2 * t + 1] = (int)(uint32_t)(u >> 32);
            } else if constexpr (DT == S8) {
                typedef int v2i __attribute__((ext_vector_type(2)));
                typedef __attribute__((address_space(3))) v2i lds_v2i;
                const v2i x = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_v2i *)(lds_void_t *)p);
                v[2 * t] = x[0];
                v[2 * t + 1] = x[1];
            } else {
                typedef int v2i __attribute__((ext_vector_type(2)));
                typedef __attribute__((address_space(3))) v2i lds_v2i;
                const v2i x = __builtin_amdgcn_ds_read_tr4_b64_v2i32((lds_v2i *)(lds_void_t *)p);
                v[2 * t] = x[0];
                v[2 * t + 1] = x[1];
            }
        }
        b[j] = v;
    }
}

// This wave's copies of slice kt into buffer `stage`: A waves advance by the
// slice's bytes, B waves by its BK rows.
template <int DT, class T>
__device__ __forceinline__ void tb_issue(uint8_t *lds, const uint8_t *const *src, int wave, int stage,
                                         int kt, long stride) {
#pragma unroll
    for (int j = 0; j < T::DMA_PER_WAVE; ++j) {
        const int d = wave * T::DMA_PER_WAVE + j;
        dma16(src[j] + (size_t)kt * stride, lds + stage * T::STAGE_BYTES + d * 1024);
    }
}

template <int DT, class T, bool ISSUE>
__device__ __forceinline__ void tb_slice(uint8_t *lds, const uint8_t *const *src, long stride, int wave,
                                         int kt, int wm, int wn, int lane, i32x4 (&ra)[2][T::FM],
                                         i32x4 (&rb)[2][T::FN], typename Acc<DT, 32>::type (&acc)[T::FM][T::FN]) {
    constexpr int NB = T::FM * T::FN;
    constexpr int NRD = T::FM + 2 * T::FN;  // LDS reads per K-chunk
    constexpr int S = T::STAGES;
    const uint8_t *st = lds + (kt % S) * T::STAGE_BYTES;
#pragma unroll
    for (int kc = 0; kc < T::KCH - 1; ++kc) {
        const int cur = kc & 1;
        __builtin_amdgcn_sched_barrier(0);
        tb_load_runs<DT, T>(st, kc + 1, wm, wn, lane, ra[cur ^ 1], rb[cur ^ 1]);
        mma_runs<DT, T, 0, NB>(ra[cur], rb[cur], acc);
        chunk_hint<NB, NRD < NB ? NRD : NB, 0>();
        __builtin_amdgcn_sched_barrier(0);
    }
    constexpr int last = (T::KCH - 1) & 1;
    constexpr int PRE = NB / 4;
    mma_runs<DT, T, 0, PRE>(ra[last], rb[last], acc);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (ISSUE) wait_vm_barrier<(S - 2) * T::DMA_PER_WAVE>();
    else wait_vm_barrier<0>();
    if constexpr (ISSUE) tb_issue<DT, T>(lds, src, wave, kt % S, kt + S, stride);
    tb_load_runs<DT, T>(lds + ((kt + 1) % S) * T::STAGE_BYTES, 0, wm, wn, lane, ra[0], rb[0]);
    mma_runs<DT, T, PRE, NB>(ra[last], rb[last], acc);
    chunk_hint<NB - PRE, NRD < NB - PRE ? NRD : NB - PRE, ISSUE ? T::DMA_PER_WAVE : 0>();
    __builtin_amdgcn_sched_barrier(0);
}

// C = A * B with B(k, j) at element k * N + j. N a multiple of BN; K bytes
// per A row (Kb) a multiple of BKB.
template <int DT, class T>
__global__ __launch_bounds__(T::NTHREADS, 1) void tiled_gemm_tb(const uint8_t *__restrict__ A,
                                                               const uint8_t *__restrict__ B,
                                                               void *__restrict__ Cv, int M, int N,
                                                               int Kb, int tiles_m, int tiles_n,
                                                               EpiParams epi) {
    typedef TB<DT, T> P;
    typedef typename Acc<DT, 32>::type acc_t;
    constexpr int S = T::STAGES;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[T::LDS_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / T::WGN, wn = wave % T::WGN;
    int tm, tn;
    tile_coords(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, T::GROUP_M, tm, tn);

    const uint8_t *src[T::DMA_PER_WAVE];
#pragma unroll
    for (int j = 0; j < T::DMA_PER_WAVE; ++j)
        src[j] = tb_src<DT, T>(A, B, M, N, Kb, tm, tn, wave * T::DMA_PER_WAVE + j, lane);
    // per-slice advance: A waves by the slice's bytes, B waves by BK rows of B
    const long stride = (wave * T::DMA_PER_WAVE < P::A_UNITS) ? (long)T::BKB : (long)P::BK * P::col_bytes(N);

    acc_t acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j) acc[i][j] = acc_t{};

    const int KT = Kb / T::BKB;
#pragma unroll
    for (int s = 0; s < S; ++s)
        if (s < KT) tb_issue<DT, T>(lds, src, wave, s, s, stride);
    if (KT >= S) wait_vm_barrier<(S - 1) * T::DMA_PER_WAVE>();
    else wait_vm_barrier<0>();

    i32x4 ra[2][T::FM], rb[2][T::FN];
    tb_load_runs<DT, T>(lds, 0, wm, wn, lane, ra[0], rb[0]);
    int kt = 0;
    for (; kt + S < KT; ++kt) tb_slice<DT, T, true>(lds, src, stride, wave, kt, wm, wn, lane, ra, rb, acc);
    for (; kt < KT; ++kt) tb_slice<DT, T, false>(lds, src, stride, wave, kt, wm, wn, lane, ra, rb, acc);

    const long row0 = (long)tm * T::BM + wm * T::WTM;
    const long col0 = (long)tn * T::BN + wn * T::WTN + (lane % 32);
    if constexpr (DT == S4)  // INT4 sums are carried times 256 (s4_lo_x16)
        epi_store_tile<DT, 32, T::FM, T::FN, T::NV>(epi, Cv, acc, row0, col0, lane / 32, M, N, ConvShift8());
    else
        epi_store_tile<DT, 32, T::FM, T::FN, T::NV>(epi, Cv, acc, row0, col0, lane / 32, M, N, ConvSame());
}

}  // namespace mpg
