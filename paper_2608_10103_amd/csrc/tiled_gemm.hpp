// tiled_gemm.hpp - LDS-tiled MFMA kernel for tile-aligned problems.
//
// Structure (the paper's tiled, software-pipelined GEMM - Methodology, Kernel
// design space, and Listings "lst:int4-double-buffer" / "lst:int4-three-stage"
// - re-designed for CDNA4):
//
//  * Each workgroup owns a BM x BN tile of C; the workgroup -> tile order is
//    XCD-aware and grouped (tile_coords).
//  * K advances in stages of BKB bytes per row. A stage holds the BM A-rows
//    and BN B-columns of that K-slice, all K-contiguous, in one LDS block of
//    (BM + BN) rows of BKB bytes. Rows are XOR-swizzled in 16-byte chunks
//    (swz) so MFMA operand reads are free of bank conflicts.
//  * Global -> LDS copies are direct 16-byte-per-lane DMA loads
//    (global_load_lds_dwordx4, the CDNA4 counterpart of a 16-byte cp.async):
//    no registers, no VALU. One wave-wide load fills 1 KiB of LDS, i.e.
//    1024 / BKB whole rows; each row is read as full 64/128-byte lines.
//  * STAGES LDS buffers form a ring; STAGES - 1 K-slices are in flight while
//    one is consumed. One wait + barrier per K-slice: wait until this wave's
//    copies of the slice about to be read have landed (vmcnt), make every wave
//    reach the barrier, then refill the buffer that was consumed one
//    iteration earlier and compute on the current one.
//  * The waves form a WGM x WGN grid; each computes a (BM/WGM) x (BN/WGN)
//    sub-tile as FM x FN blocks of 32x32 MFMAs, reading 16-byte operand runs
//    from LDS (ds_read_b128). INT4 runs are decoded to int8 in registers.
//  * Epilogue: accumulators straight to C (INT4: shifted right by 8, see
//    s4_lo_x16), each store instruction writing two 128-byte row segments.
#pragma once

#include "device_common.hpp"

namespace mpg {

template <int BM_, int BN_, int WGM_, int WGN_, int BKB_, int STAGES_, int GROUP_M_>
struct TileCfg {
    static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_, BKB = BKB_;
    static constexpr int STAGES = STAGES_, GROUP_M = GROUP_M_;
    static constexpr int NWAVES = WGM * WGN;
    static constexpr int NTHREADS = 64 * NWAVES;
    static constexpr int WTM = BM / WGM, WTN = BN / WGN;  // wave sub-tile
    static constexpr int FM = WTM / 32, FN = WTN / 32;    // MFMA blocks per wave
    static constexpr int CH = BKB / 16;                   // 16-byte chunks per LDS row
    static constexpr int ROWS = BM + BN;                  // LDS rows per stage
    static constexpr int STAGE_BYTES = ROWS * BKB;
    static constexpr int LDS_BYTES = STAGES * STAGE_BYTES;
    static constexpr int ROWS_PER_DMA = 1024 / BKB;       // rows one wave-wide DMA fills
    static constexpr int NDMA = ROWS / ROWS_PER_DMA;      // DMAs per stage per workgroup
    static constexpr int DMA_PER_WAVE = NDMA / NWAVES;
    static constexpr int KCH = BKB / 32;                  // 32-byte K-chunks per stage
    static_assert(BKB == 64 || BKB == 128, "LDS rows are 64 or 128 bytes");
    static_assert(WTM % 32 == 0 && WTN % 32 == 0 && FM >= 1 && FN >= 1, "wave tile");
    static_assert(NDMA % NWAVES == 0, "DMAs split evenly over waves");
    static_assert(BM % ROWS_PER_DMA == 0, "a DMA never straddles the A and B parts");
    static_assert(STAGES >= 2 && (STAGES - 2) * DMA_PER_WAVE <= 63, "vmcnt range");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS capacity");
};

// Wait until at most N of this wave's vector-memory operations are pending
// and all its LDS operations are done, then barrier the workgroup. The memory
// clobber keeps the compiler from moving LDS accesses across it.
template <int N>
__device__ __forceinline__ void wait_vm_barrier() {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

typedef __attribute__((address_space(3))) void lds_void;

// One wave-wide direct global -> LDS load: lane l copies 16 bytes from g (its
// own address) to lds_base + 16 * l. lds_base must be wave-uniform. The
// builtin needs the gfx950 target, so only the device pass sees it.
__device__ __forceinline__ void dma16(const uint8_t *g, uint8_t *lds_base) {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_global_load_lds(g, (lds_void *)lds_base, 16, 0, 0);
#endif
}

// Issue this wave's DMA loads of K-slice kt into LDS buffer `stage`.
template <class T>
__device__ __forceinline__ void issue_stage(uint8_t *lds, const uint8_t *const *src,
                                            int wave, int stage, int kt) {
#pragma unroll
    for (int j = 0; j < T::DMA_PER_WAVE; ++j) {
        const int d = wave * T::DMA_PER_WAVE + j;
        dma16(src[j] + (size_t)kt * T::BKB, lds + stage * T::STAGE_BYTES + d * 1024);
    }
}

// All MFMAs of one LDS buffer for this wave's sub-tile.
template <int DT, class T>
__device__ __forceinline__ void compute_stage(const uint8_t *st, int wm, int wn, int r, int h,
                                              typename Acc<DT>::type (&acc)[T::FM][T::FN]) {
#pragma unroll
    for (int kc = 0; kc < T::KCH; ++kc) {
        i32x4 a[T::FM], b[T::FN];
#pragma unroll
        for (int i = 0; i < T::FM; ++i) {
            const int q = wm * T::WTM + i * 32 + r;
            a[i] = *reinterpret_cast<const i32x4 *>(
                st + q * T::BKB + (((2 * kc + h) ^ swz<T::CH>(q)) << 4));
        }
#pragma unroll
        for (int j = 0; j < T::FN; ++j) {
            const int q = T::BM + wn * T::WTN + j * 32 + r;
            b[j] = *reinterpret_cast<const i32x4 *>(
                st + q * T::BKB + (((2 * kc + h) ^ swz<T::CH>(q)) << 4));
        }
        if constexpr (DT == F16) {
#pragma unroll
            for (int i = 0; i < T::FM; ++i)
#pragma unroll
                for (int j = 0; j < T::FN; ++j) acc[i][j] = mfma_f16(a[i], b[j], acc[i][j]);
        } else if constexpr (DT == S8) {
#pragma unroll
            for (int i = 0; i < T::FM; ++i)
#pragma unroll
                for (int j = 0; j < T::FN; ++j) acc[i][j] = mfma_i8(a[i], b[j], acc[i][j]);
        } else {
            i32x4 alo[T::FM], ahi[T::FM], blo[T::FN], bhi[T::FN];
#pragma unroll
            for (int i = 0; i < T::FM; ++i) { alo[i] = s4_lo_x16(a[i]); ahi[i] = s4_hi_x16(a[i]); }
#pragma unroll
            for (int j = 0; j < T::FN; ++j) { blo[j] = s4_lo_x16(b[j]); bhi[j] = s4_hi_x16(b[j]); }
#pragma unroll
            for (int i = 0; i < T::FM; ++i)
#pragma unroll
                for (int j = 0; j < T::FN; ++j) {
                    acc[i][j] = mfma_i8(alo[i], blo[j], acc[i][j]);
                    acc[i][j] = mfma_i8(ahi[i], bhi[j], acc[i][j]);
                }
        }
    }
}

template <int DT, class T>
__global__ __launch_bounds__(T::NTHREADS, 1) void tiled_gemm(const uint8_t *__restrict__ A,
                                                            const uint8_t *__restrict__ B,
                                                            void *__restrict__ Cv, int M, int N,
                                                            int Kb, int tiles_m, int tiles_n) {
    typedef typename Acc<DT>::type acc_t;
    typedef typename Acc<DT>::out out_t;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[T::LDS_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 31, h = lane >> 5;
    const int wm = wave / T::WGN, wn = wave % T::WGN;
    int tm, tn;
    tile_coords(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, T::GROUP_M, tm, tn);

    // Source of each of this wave's DMA loads (stage-independent part).
    const uint8_t *src[T::DMA_PER_WAVE];
#pragma unroll
    for (int j = 0; j < T::DMA_PER_WAVE; ++j) {
        const int d = wave * T::DMA_PER_WAVE + j;
        const int q = d * T::ROWS_PER_DMA + lane / T::CH;  // LDS row
        const int c = (lane % T::CH) ^ swz<T::CH>(q);       // logical chunk for this slot
        const uint8_t *rowp = (q < T::BM) ? A + (size_t)(tm * T::BM + q) * Kb
                                          : B + (size_t)(tn * T::BN + (q - T::BM)) * Kb;
        src[j] = rowp + c * 16;
    }

    acc_t acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j) acc[i][j] = acc_t{};

    const int KT = Kb / T::BKB;
#pragma unroll
    for (int s = 0; s < T::STAGES - 1; ++s)
        if (s < KT) issue_stage<T>(lds, src, wave, s, s);

    for (int kt = 0; kt < KT; ++kt) {
        if (kt + T::STAGES - 2 < KT) wait_vm_barrier<(T::STAGES - 2) * T::DMA_PER_WAVE>();
        else wait_vm_barrier<0>();
        if (kt + T::STAGES - 1 < KT)
            issue_stage<T>(lds, src, wave, (kt + T::STAGES - 1) % T::STAGES, kt + T::STAGES - 1);
        compute_stage<DT, T>(lds + (kt % T::STAGES) * T::STAGE_BYTES, wm, wn, r, h, acc);
    }

    out_t *C = reinterpret_cast<out_t *>(Cv);
    const long row0 = (long)tm * T::BM + wm * T::WTM + 4 * h;
    const long col0 = (long)tn * T::BN + wn * T::WTN + r;
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const long row = row0 + i * 32 + 8 * (v >> 2) + (v & 3);
                const long col = col0 + j * 32;
                if constexpr (DT == S4) C[row * N + col] = acc[i][j][v] >> 8;
                else C[row * N + col] = acc[i][j][v];
            }
}

}  // namespace mpg
