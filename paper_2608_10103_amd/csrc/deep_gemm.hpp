// deep_gemm.hpp - one wave per SIMD, operand runs read two K-chunks ahead.
//
// Measured on MI355X: every LDS write instruction (a 1 KiB direct-to-LDS
// load or a ds_write_b128) holds the LDS for about as long as three 1 KiB
// operand reads, and the 256 x 256 kernels with 128 x 64 wave tiles keep the
// LDS about three quarters busy at full MFMA rate; the queueing shows up as
// operand waits. A 128 x 128 wave tile reads a third less per MFMA, but with
// one wave per SIMD nothing covers a wait. This kernel removes the waits by
// construction:
//
//  * 256 x 256 tile, 2 x 2 waves of 128 x 128 (16 MFMA blocks, accumulators in
//    AGPRs), 64-byte K-slices (two 32-byte K-chunks) in a STAGES-deep ring.
//  * Three operand register sets: the runs of chunk c + 2 are read from LDS
//    while the MFMAs of chunk c run, so a read has a whole chunk of MFMAs
//    (16 on FP16/INT8) to return before anything depends on it.
//  * One barrier per slice, at its start. By then this wave has read all of
//    the slice (into registers, a slice ahead), so after the barrier the
//    slice's buffer is free for the copy of slice kt + STAGES, and the copy of
//    slice kt + 1 (waited for by vmcnt before the barrier) is visible to the
//    reads of the next two chunks. The first MFMAs after the barrier use
//    registers loaded a slice earlier, so the barrier is never followed by an
//    operand wait.
//  * The slice's direct-to-LDS loads are spread one per few MFMAs (a burst of
//    them stalls the in-order issue of MFMAs behind them), and have
//    STAGES - 1 slices to land.
#pragma once

#include "tiled_gemm.hpp"

namespace mpg {

// Scheduling hint for one K-chunk: NR LDS reads, one after each of the first
// NR MFMAs, then ND direct-to-LDS loads spread evenly over the other MFMAs.
template <int NM, int NR, int ND>
__device__ __forceinline__ void deep_hint() {
    static_assert(NM > NR, "more MFMAs than reads per chunk");
    static_for<NR>([&](auto) __attribute__((always_inline)) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
    });
    constexpr int REST = NM - NR;
    if constexpr (ND > 0) {
        constexpr int SP = REST / ND > 0 ? REST / ND : 1;
        static_for<ND>([&](auto) __attribute__((always_inline)) {
            __builtin_amdgcn_sched_group_barrier(0x008, SP, 0);  // SP MFMAs
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // one DMA
        });
        if constexpr (REST > SP * ND) __builtin_amdgcn_sched_group_barrier(0x008, REST - SP * ND, 0);
    } else {
        __builtin_amdgcn_sched_group_barrier(0x008, REST, 0);
    }
}

// One K-slice kt of the deep kernel. P = kt mod 3 names the register sets:
// chunk c of slice kt lives in set (2 kt + c) mod 3. The slice copies slice
// kt + STAGES into the buffer it frees; past the end of K the copy re-reads
// the last slice into a buffer nobody reads again, so every slice has the same
// code and the same count of copies in flight.
template <int DT, class T, int P>
__device__ __forceinline__ void deep_slice(uint8_t *lds, const uint8_t *const *src, int wave,
                                           int kt, int KT, int wm, int wn, int r, int h,
                                           i32x4 (&ra)[3][T::FM], i32x4 (&rb)[3][T::FN],
                                           typename Acc<DT, T::MS>::type (&acc)[T::FM][T::FN]) {
    constexpr int S = T::STAGES;
    constexpr int NB = T::FM * T::FN;
    constexpr int MPB = (DT == S4) ? 2 : 1;
    constexpr int NRD = T::FM + T::FN;
    constexpr int DPW = T::DMA_PER_WAVE;
    constexpr int C0 = (2 * P) % 3, C1 = (2 * P + 1) % 3;  // this slice's chunks
    constexpr int N0 = (2 * P + 2) % 3, N1 = (2 * P) % 3;  // next slice's chunks
    // This wave's reads of slice kt are done (lgkmcnt) and its copies of slice
    // kt + 1 have landed (vmcnt: the copies of slices kt + 2 .. kt + S - 1 may
    // still be in flight); the barrier extends both to the workgroup.
    wait_vm_barrier<(S - 2) * DPW>();
    // the next slice's buffer (after the last slice: one nobody uses again)
    const uint8_t *nxt = lds + ((kt + 1) % S) * T::STAGE_BYTES;
    const int ck = min(kt + S, KT - 1);  // slice copied into this slice's buffer
    const int cs = kt % S;
    __builtin_amdgcn_sched_barrier(0);
    load_runs<T>(nxt, 0, wm, wn, r, h, ra[N0], rb[N0]);
    issue_part<T, 0, DPW / 2>(lds, src, wave, cs, ck);
    mma_runs<DT, T, 0, NB>(ra[C0], rb[C0], acc);
    deep_hint<NB * MPB, NRD, DPW / 2>();
    __builtin_amdgcn_sched_barrier(0);
    load_runs<T>(nxt, 1, wm, wn, r, h, ra[N1], rb[N1]);
    issue_part<T, DPW / 2, DPW>(lds, src, wave, cs, ck);
    mma_runs<DT, T, 0, NB>(ra[C1], rb[C1], acc);
    deep_hint<NB * MPB, NRD, DPW - DPW / 2>();
    __builtin_amdgcn_sched_barrier(0);
}

// C tile = A rows x B columns of one workgroup. M and N need not be multiples
// of the tile (edge rows are clamped in the copy and masked in the stores);
// the K bytes per row must be a multiple of the 64-byte slice.
template <int DT, class T>
__global__ __launch_bounds__(T::NTHREADS, 1) void tiled_gemm_deep(const uint8_t *__restrict__ A,
                                                                 const uint8_t *__restrict__ B,
                                                                 void *__restrict__ Cv, int M,
                                                                 int N, int Kb, int tiles_m,
                                                                 int tiles_n, EpiParams epi) {
    static_assert(T::KCH == 2, "two K-chunks per slice");
    static_assert(T::DMA_PER_WAVE % 2 == 0, "copies split over the two chunks");
    static_assert((T::STAGES - 1) * T::DMA_PER_WAVE <= 63, "vmcnt range");
    typedef typename Acc<DT, T::MS>::type acc_t;
    constexpr int S = T::STAGES;
    constexpr int DPW = T::DMA_PER_WAVE;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[T::LDS_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane % T::MS, h = lane / T::MS;
    const int wm = wave / T::WGN, wn = wave % T::WGN;
    int tm, tn;
    tile_coords(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, T::GROUP_M, tm, tn);

    const uint8_t *src[DPW];
#pragma unroll
    for (int j = 0; j < DPW; ++j) src[j] = stage_src<T>(A, B, M, N, Kb, tm, tn, wave * DPW + j, lane);

    acc_t acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j) acc[i][j] = acc_t{};

    const int KT = Kb / T::BKB;
    // Prologue: copy slices 0 .. S - 1 (clamped to the last slice), wait for
    // slice 0, read both its chunks.
#pragma unroll
    for (int s = 0; s < S; ++s) issue_stage<T>(lds, src, wave, s, min(s, KT - 1));
    wait_vm_barrier<(S - 1) * DPW>();
    i32x4 ra[3][T::FM], rb[3][T::FN];
    load_runs<T>(lds, 0, wm, wn, r, h, ra[0], rb[0]);
    load_runs<T>(lds, 1, wm, wn, r, h, ra[1], rb[1]);

    // Three slices per iteration, so the register sets are fixed at compile
    // time; then at most two more.
    int kt = 0;
    for (; kt + 3 <= KT; kt += 3) {
        deep_slice<DT, T, 0>(lds, src, wave, kt, KT, wm, wn, r, h, ra, rb, acc);
        deep_slice<DT, T, 1>(lds, src, wave, kt + 1, KT, wm, wn, r, h, ra, rb, acc);
        deep_slice<DT, T, 2>(lds, src, wave, kt + 2, KT, wm, wn, r, h, ra, rb, acc);
    }
    if (kt < KT) deep_slice<DT, T, 0>(lds, src, wave, kt, KT, wm, wn, r, h, ra, rb, acc);
    if (kt + 1 < KT) deep_slice<DT, T, 1>(lds, src, wave, kt + 1, KT, wm, wn, r, h, ra, rb, acc);
    // the clamped copies of the last slices may still be landing
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

    const long row0 = (long)tm * T::BM + wm * T::WTM;
    const long col0 = (long)tn * T::BN + wn * T::WTN + r;
    if constexpr (DT == S4)
        epi_store_tile<DT, T::MS, T::FM, T::FN, T::NV>(epi, Cv, acc, row0, col0, h, M, N, ConvShift8());
    else
        epi_store_tile<DT, T::MS, T::FM, T::FN, T::NV>(epi, Cv, acc, row0, col0, h, M, N, ConvSame());
}

}  // namespace mpg
