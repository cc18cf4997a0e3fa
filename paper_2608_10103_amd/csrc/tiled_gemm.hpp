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
//  * M and N need not be multiples of the tile: edge tiles clamp their
//    copy rows (stage_src) and mask their stores. K must fill whole slices.
#pragma once

#include "device_common.hpp"

namespace mpg {

template <int BM_, int BN_, int WGM_, int WGN_, int BKB_, int STAGES_, int GROUP_M_, int MS_ = 32>
struct TileCfg {
    static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_, BKB = BKB_;
    static constexpr int STAGES = STAGES_, GROUP_M = GROUP_M_;
    static constexpr int MS = MS_;                        // MFMA block: 32x32 or 16x16
    static constexpr int G = 64 / MS;                     // lane groups along K
    static constexpr int NV = MS * MS / 64;               // accumulator values per lane
    static constexpr int NWAVES = WGM * WGN;
    static constexpr int NTHREADS = 64 * NWAVES;
    static constexpr int WTM = BM / WGM, WTN = BN / WGN;  // wave sub-tile
    static constexpr int FM = WTM / MS, FN = WTN / MS;    // MFMA blocks per wave
    static constexpr int CH = BKB / 16;                   // 16-byte chunks per LDS row
    static constexpr int ROWS = BM + BN;                  // LDS rows per stage
    static constexpr int STAGE_BYTES = ROWS * BKB;
    static constexpr int LDS_BYTES = STAGES * STAGE_BYTES;
    static constexpr int ROWS_PER_DMA = 1024 / BKB;       // rows one wave-wide DMA fills
    static constexpr int NDMA = ROWS / ROWS_PER_DMA;      // DMAs per stage per workgroup
    static constexpr int DMA_PER_WAVE = NDMA / NWAVES;
    static constexpr int KCH = BKB / (16 * G);            // MFMA K-steps per stage
    static_assert(BKB == 64 || BKB == 128, "LDS rows are 64 or 128 bytes");
    static_assert(MS == 32 || MS == 16, "MFMA block");
    static_assert(WTM % MS == 0 && WTN % MS == 0 && FM >= 1 && FN >= 1 && KCH >= 1, "wave tile");
    static_assert(NDMA % NWAVES == 0, "DMAs split evenly over waves");
    static_assert(BM % ROWS_PER_DMA == 0, "a DMA never straddles the A and B parts");
    static_assert(STAGES >= 2 && (STAGES - 2) * DMA_PER_WAVE <= 63, "vmcnt range");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS capacity");
};

// Source of lane `lane` for the copy unit d (1 KiB of LDS) of a stage:
// LDS row q = d * ROWS_PER_DMA + lane / CH takes A row tm*BM + q or B row
// tn*BN + q - BM; slot lane % CH of that row holds logical chunk
// slot ^ swz(q). Rows past M (or N) are clamped to the last one: the tile's
// edge rows then compute values nobody stores, and every load stays inside
// the operands.
template <class T>
__device__ __forceinline__ const uint8_t *stage_src(const uint8_t *A, const uint8_t *B, int M,
                                                    int N, int Kb, int tm, int tn, int d,
                                                    int lane) {
    const int q = d * T::ROWS_PER_DMA + lane / T::CH;
    const int c = (lane % T::CH) ^ swz<T::CH>(q);
    const uint8_t *rowp = (q < T::BM) ? A + (size_t)min(tm * T::BM + q, M - 1) * Kb
                                      : B + (size_t)min(tn * T::BN + (q - T::BM), N - 1) * Kb;
    return rowp + c * 16;
}

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
                                              typename Acc<DT, T::MS>::type (&acc)[T::FM][T::FN]) {
#pragma unroll
    for (int kc = 0; kc < T::KCH; ++kc) {
        i32x4 a[T::FM], b[T::FN];
#pragma unroll
        for (int i = 0; i < T::FM; ++i) {
            const int q = wm * T::WTM + i * T::MS + r;
            a[i] = *reinterpret_cast<const i32x4 *>(
                st + q * T::BKB + (((T::G * kc + h) ^ swz<T::CH>(q)) << 4));
        }
#pragma unroll
        for (int j = 0; j < T::FN; ++j) {
            const int q = T::BM + wn * T::WTN + j * T::MS + r;
            b[j] = *reinterpret_cast<const i32x4 *>(
                st + q * T::BKB + (((T::G * kc + h) ^ swz<T::CH>(q)) << 4));
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

// ---------------------------------------------------------------------------
// Software-pipelined variant. Same tiles, LDS layout and DMA as tiled_gemm, but
//  * operand runs are double-buffered in registers: the ds_reads of K-chunk
//    kc+1 are issued between the MFMAs of chunk kc (sched_group_barrier
//    interleaves one read per MFMA), so LDS latency hides under the MFMAs;
//  * the per-slice wait + barrier sits inside the last K-chunk: half of its
//    MFMAs run, then the barrier, then the next slice's DMA is issued and its
//    first runs are read while the other half of the MFMAs run;
//  * all STAGES buffers are filled up front, so each slice's copy has
//    STAGES - 1 slices of compute to land.
// Needs an even number of 32-byte K-chunks per slice (KCH), so chunk 0 of
// every slice uses register set 0.

template <class T>
__device__ __forceinline__ void load_runs(const uint8_t *st, int kc, int wm, int wn, int r, int h,
                                          i32x4 (&a)[T::FM], i32x4 (&b)[T::FN]) {
#pragma unroll
    for (int i = 0; i < T::FM; ++i) {
        const int q = wm * T::WTM + i * T::MS + r;
        a[i] = *reinterpret_cast<const i32x4 *>(st + q * T::BKB +
                                                 (((T::G * kc + h) ^ swz<T::CH>(q)) << 4));
    }
#pragma unroll
    for (int j = 0; j < T::FN; ++j) {
        const int q = T::BM + wn * T::WTN + j * T::MS + r;
        b[j] = *reinterpret_cast<const i32x4 *>(st + q * T::BKB +
                                                 (((T::G * kc + h) ^ swz<T::CH>(q)) << 4));
    }
}

// MFMAs of blocks p in [P0, P1) (p = i * FN + j) on one register set.
template <int DT, class T, int P0, int P1>
__device__ __forceinline__ void mma_runs(const i32x4 (&a)[T::FM], const i32x4 (&b)[T::FN],
                                         typename Acc<DT, T::MS>::type (&acc)[T::FM][T::FN]) {
#pragma unroll
    for (int p = P0; p < P1; ++p) {
        const int i = p / T::FN, j = p % T::FN;
        if constexpr (DT == F16) {
            acc[i][j] = mfma_f16(a[i], b[j], acc[i][j]);
        } else if constexpr (DT == S8) {
            acc[i][j] = mfma_i8(a[i], b[j], acc[i][j]);
        } else {
            acc[i][j] = mfma_i8(s4_lo_x16(a[i]), s4_lo_x16(b[j]), acc[i][j]);
            acc[i][j] = mfma_i8(s4_hi_x16(a[i]), s4_hi_x16(b[j]), acc[i][j]);
        }
    }
}

// Scheduling hint: interleave NR LDS reads one-for-one with the first NR of
// NM MFMAs, then the remaining MFMAs.
template <int NM, int NR>
__device__ __forceinline__ void interleave_hint() {
#pragma unroll
    for (int x = 0; x < NR && x < NM; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
    }
    if constexpr (NM > NR) __builtin_amdgcn_sched_group_barrier(0x008, NM - NR, 0);
}

// Issue DMA loads j in [J0, J1) of this wave for K-slice kt into buffer `stage`.
template <class T, int J0, int J1>
__device__ __forceinline__ void issue_part(uint8_t *lds, const uint8_t *const *src, int wave,
                                           int stage, int kt) {
#pragma unroll
    for (int j = J0; j < J1; ++j) {
        const int d = wave * T::DMA_PER_WAVE + j;
        dma16(src[j] + (size_t)kt * T::BKB, lds + stage * T::STAGE_BYTES + d * 1024);
    }
}

// Scheduling hint for one K-chunk: NR LDS reads and NV DMA loads, each placed
// after one of the first NR + NV of the chunk's NM MFMAs, then the rest.
template <int NM, int NR, int NV>
__device__ __forceinline__ void chunk_hint() {
#pragma unroll
    for (int x = 0; x < NR; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
    }
#pragma unroll
    for (int x = 0; x < NV; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // one global load (DMA)
    }
    if constexpr (NM > NR + NV) __builtin_amdgcn_sched_group_barrier(0x008, NM - NR - NV, 0);
}

// DMA loads of one slice handed out over KCH issue slots: chunks 0..KCH-2
// and the first half of the last chunk (before its barrier).
template <class T, int C>
struct DmaSlot {
    static constexpr int J0 = T::DMA_PER_WAVE * C / T::KCH;
    static constexpr int J1 = T::DMA_PER_WAVE * (C + 1) / T::KCH;
};

// DMA slot C of a slice (no-op when the slice has fewer chunks).
template <class T, int C>
__device__ __forceinline__ void issue_slot(uint8_t *lds, const uint8_t *const *src, int wave,
                                           int stage, int kt) {
    if constexpr (C < T::KCH)
        issue_part<T, DmaSlot<T, C>::J0, DmaSlot<T, C>::J1>(lds, src, wave, stage, kt);
}

// One K-slice of the pipelined kernel (buffer kt % STAGES holds slice kt).
// ISSUE: this slice also starts a copy. SPREAD selects where:
//  * SPREAD: the copy of slice kt + S - 1 into the buffer freed at the
//    previous slice's barrier, its DMA loads spread over the slice's chunks
//    between the MFMAs (the wave's in-order issue never stalls on a burst of
//    vector-memory instructions);
//  * otherwise: the copy of slice kt + S, all DMA loads issued right after
//    this slice's barrier, into the buffer that barrier frees.
// Branch-free, so the reads, copies and MFMAs of a chunk share one
// scheduling region.
template <int DT, class T, bool ISSUE, bool SPREAD>
__device__ __forceinline__ void pf_slice(uint8_t *lds, const uint8_t *const *src, int wave, int kt,
                                         int wm, int wn, int r, int h, i32x4 (&ra)[2][T::FM],
                                         i32x4 (&rb)[2][T::FN],
                                         typename Acc<DT, T::MS>::type (&acc)[T::FM][T::FN]) {
    constexpr int NB = T::FM * T::FN;        // MFMA blocks per wave
    constexpr int MPB = (DT == S4) ? 2 : 1;  // MFMAs per block per K-chunk
    constexpr int NRD = T::FM + T::FN;       // LDS reads per K-chunk
    constexpr int S = T::STAGES;
    constexpr bool SP = ISSUE && SPREAD;
    const uint8_t *st = lds + (kt % S) * T::STAGE_BYTES;
    const int sp_stage = (kt + S - 1) % S, sp_kt = kt + S - 1;
#pragma unroll
    for (int kc = 0; kc < T::KCH - 1; ++kc) {
        const int cur = kc & 1;
        __builtin_amdgcn_sched_barrier(0);
        load_runs<T>(st, kc + 1, wm, wn, r, h, ra[cur ^ 1], rb[cur ^ 1]);
        if constexpr (SP) {
            // kc is a compile-time constant after unrolling
            static_assert(T::KCH <= 4, "DMA slots are handed out for at most 4 chunks");
            if (kc == 0) issue_slot<T, 0>(lds, src, wave, sp_stage, sp_kt);
            if (kc == 1) issue_slot<T, 1>(lds, src, wave, sp_stage, sp_kt);
            if (kc == 2) issue_slot<T, 2>(lds, src, wave, sp_stage, sp_kt);
        }
        mma_runs<DT, T, 0, NB>(ra[cur], rb[cur], acc);
        if constexpr (SP) {
            constexpr int nv = T::DMA_PER_WAVE / T::KCH + 1;
            chunk_hint<NB * MPB, NRD, nv>();
        } else {
            chunk_hint<NB * MPB, NRD, 0>();
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    // Last K-chunk: a quarter of its MFMAs (with the slice's last DMA loads),
    // the barrier that publishes slice kt + 1 and frees this slice's buffer,
    // then the next slice's first runs under the other MFMAs.
    constexpr int last = (T::KCH - 1) & 1;
    constexpr int PRE = NB / 4;
    if constexpr (SP) issue_slot<T, T::KCH - 1>(lds, src, wave, sp_stage, sp_kt);
    mma_runs<DT, T, 0, PRE>(ra[last], rb[last], acc);
    if constexpr (SP) {
        constexpr int nv = DmaSlot<T, T::KCH - 1>::J1 - DmaSlot<T, T::KCH - 1>::J0;
        chunk_hint<PRE * MPB, 0, nv>();
    }
    __builtin_amdgcn_sched_barrier(0);
    // slices issued so far: 0 .. kt + S - 1 (steady state); those after
    // slice kt + 1 may stay in flight
    if constexpr (ISSUE) wait_vm_barrier<(S - 2) * T::DMA_PER_WAVE>();
    else wait_vm_barrier<0>();
    if constexpr (ISSUE && !SPREAD) issue_stage<T>(lds, src, wave, kt % S, kt + S);
    // for the final slice this reads a buffer nobody uses again; harmless
    load_runs<T>(lds + ((kt + 1) % S) * T::STAGE_BYTES, 0, wm, wn, r, h, ra[0], rb[0]);
    mma_runs<DT, T, PRE, NB>(ra[last], rb[last], acc);
    chunk_hint<(NB - PRE) * MPB, NRD, (ISSUE && !SPREAD) ? T::DMA_PER_WAVE : 0>();
    __builtin_amdgcn_sched_barrier(0);
}

// Split-K fixup of one workgroup (see tiled_gemm_pf). Returns true in the
// workgroup that must write C, with acc holding the sum of all splits.
// Partial slot layout: value v of block (i, j) of thread t at word
// ((i * FN + j) * NV + v) * NTHREADS + t of the slot, so every store and load
// instruction covers NTHREADS consecutive words.
template <int DT, class T>
__device__ __forceinline__ bool splitk_fixup(typename Acc<DT, T::MS>::type (&acc)[T::FM][T::FN],
                                             int pid, int split, int splits, int *counters,
                                             uint32_t *partials, uint8_t *lds) {
    typedef typename Acc<DT, T::MS>::out out_t;
    constexpr int SLOT = T::BM * T::BN;
    const int tid = threadIdx.x;
    uint32_t *mine = partials + ((size_t)pid * splits + split) * SLOT;
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j)
#pragma unroll
            for (int v = 0; v < T::NV; ++v)
                mine[((i * T::FN + j) * T::NV + v) * T::NTHREADS + tid] =
                    __builtin_bit_cast(uint32_t, (out_t)acc[i][j][v]);
    // Each wave waits until its stores have reached L2 (stores write through
    // L1); after the barrier one thread makes them visible device-wide (the
    // agent-scope release writes back the L2, whatever wave wrote the lines)
    // and counts the split. Fencing in one thread instead of every wave keeps
    // the L2 write-back / invalidate to one per workgroup.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    int *flag = reinterpret_cast<int *>(lds);
    if (tid == 0) {
        __threadfence();
        const int last = atomicAdd(&counters[pid], 1) == splits - 1;
        if (last) __threadfence();  // acquire: later loads see the other splits' partials
        flag[0] = last;
    }
    __syncthreads();
    if (!flag[0]) return false;
    const uint32_t *tile = partials + (size_t)pid * splits * SLOT;
    // One chunk of accumulators at a time: a block row (or, when the wave
    // holds 256 accumulators and registers are short, one block); the loads
    // of a chunk for one split are independent, so each split costs one memory
    // round trip per chunk. Every element is still summed in split order.
    constexpr int JW = (T::FM * T::FN * T::NV >= 256) ? 1 : T::FN;
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j0 = 0; j0 < T::FN; j0 += JW) {
#pragma unroll
            for (int j = j0; j < j0 + JW; ++j)
#pragma unroll
                for (int v = 0; v < T::NV; ++v)
                    acc[i][j][v] = __builtin_bit_cast(out_t, tile[((i * T::FN + j) * T::NV + v) * T::NTHREADS + tid]);
            for (int s = 1; s < splits; ++s) {
                const uint32_t *part = tile + (size_t)s * SLOT;
                out_t add[JW][T::NV];
#pragma unroll
                for (int j = 0; j < JW; ++j)
#pragma unroll
                    for (int v = 0; v < T::NV; ++v)
                        add[j][v] = __builtin_bit_cast(
                            out_t, part[((i * T::FN + j0 + j) * T::NV + v) * T::NTHREADS + tid]);
#pragma unroll
                for (int j = 0; j < JW; ++j)
#pragma unroll
                    for (int v = 0; v < T::NV; ++v) acc[i][j0 + j][v] += add[j][v];
            }
        }
    if (tid == 0) counters[pid] = 0;  // ready for the next call on this workspace
    return true;
}

//
// Split-K (splits > 1): workgroup x computes K-range x / ntiles of tile
// x % ntiles (the K bytes divided evenly, whole slices each), stores its
// accumulators to its slot of `partials` in register order, and counts itself
// in counters[tile]. The workgroup that brings the count to `splits` sums the
// tile's partials in split order 0, 1, ... (so the result does not depend on
// which workgroup finishes last), writes C and resets the counter to zero for
// the next call. No workgroup waits for another. The counters must be zero
// before the first call.
// Accumulate K-slices [kt0, kt0 + KT) of tile (tm, tn) into acc (zeroed
// here) with the pipelined schedule above. On return every copy has landed;
// the waves may still be reading LDS, so a caller that reuses the buffers
// for another tile needs a barrier first.
template <int DT, class T, bool SPREAD>
__device__ __forceinline__ void pf_accumulate(uint8_t *lds, const uint8_t *A, const uint8_t *B, int M,
                                              int N, int Kb, int tm, int tn, int kt0, int KT,
                                              typename Acc<DT, T::MS>::type (&acc)[T::FM][T::FN]) {
    typedef typename Acc<DT, T::MS>::type acc_t;
    constexpr int S = T::STAGES;
    // the lane's addresses derive from an opaque copy of the thread id, so a
    // caller that accumulates several tiles in a loop recomputes them per
    // tile instead of keeping them live through its epilogues
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane % T::MS, h = lane / T::MS;
    const int wm = wave / T::WGN, wn = wave % T::WGN;
    A += (size_t)kt0 * T::BKB;
    B += (size_t)kt0 * T::BKB;

    const uint8_t *src[T::DMA_PER_WAVE];
#pragma unroll
    for (int j = 0; j < T::DMA_PER_WAVE; ++j) {
        const int d = wave * T::DMA_PER_WAVE + j;
        src[j] = stage_src<T>(A, B, M, N, Kb, tm, tn, d, lane);
    }

#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j) acc[i][j] = acc_t{};

    // Fill the ring (all S buffers; S - 1 when later copies are spread over
    // the slices), then wait for slice 0.
    constexpr int PRE = SPREAD ? S - 1 : S;
#pragma unroll
    for (int s = 0; s < PRE; ++s)
        if (s < KT) issue_stage<T>(lds, src, wave, s, s);
    if (KT >= PRE) wait_vm_barrier<(PRE - 1) * T::DMA_PER_WAVE>();
    else wait_vm_barrier<0>();

    i32x4 ra[2][T::FM], rb[2][T::FN];
    load_runs<T>(lds, 0, wm, wn, r, h, ra[0], rb[0]);

    // Steady state: every slice issues one copy. Tail: the last PRE slices
    // issue nothing and wait for all outstanding copies.
    int kt = 0;
    for (; kt + PRE < KT; ++kt)
        pf_slice<DT, T, true, SPREAD>(lds, src, wave, kt, wm, wn, r, h, ra, rb, acc);
    for (; kt < KT; ++kt)
        pf_slice<DT, T, false, SPREAD>(lds, src, wave, kt, wm, wn, r, h, ra, rb, acc);
}

// Accumulators of a finished tile to C (INT4: the sums carried times 256
// shifted back).
template <int DT, class T>
__device__ __forceinline__ void pf_store(const EpiParams &epi, void *Cv,
                                         const typename Acc<DT, T::MS>::type (&acc)[T::FM][T::FN], int tm,
                                         int tn, int M, int N) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int r = lane % T::MS, h = lane / T::MS;
    const int wm = wave / T::WGN, wn = wave % T::WGN;
    const long row0 = (long)tm * T::BM + wm * T::WTM;
    const long col0 = (long)tn * T::BN + wn * T::WTN + r;
    if constexpr (DT == S4)
        epi_store_tile<DT, T::MS, T::FM, T::FN, T::NV>(epi, Cv, acc, row0, col0, h, M, N, ConvShift8());
    else
        epi_store_tile<DT, T::MS, T::FM, T::FN, T::NV>(epi, Cv, acc, row0, col0, h, M, N, ConvSame());
}

//
// Split-K (splits > 1): workgroup x computes K-range x / ntiles of tile
// x % ntiles (the K bytes divided evenly, whole slices each), stores its
// accumulators to its slot of `partials` in register order, and counts itself
// in counters[tile]. The workgroup that brings the count to `splits` sums the
// tile's partials in split order 0, 1, ... (so the result does not depend on
// which workgroup finishes last), writes C and resets the counter to zero for
// the next call. No workgroup waits for another. The counters must be zero
// before the first call.
template <int DT, class T, bool SPREAD>
__global__ __launch_bounds__(T::NTHREADS, 1) void tiled_gemm_pf(const uint8_t *__restrict__ A,
                                                               const uint8_t *__restrict__ B,
                                                               void *__restrict__ Cv, int M,
                                                               int N, int Kb, int tiles_m,
                                                               int tiles_n, int splits,
                                                               int *__restrict__ counters,
                                                               uint32_t *__restrict__ partials,
                                                               EpiParams epi) {
    static_assert(T::KCH % 2 == 0, "even number of K-chunks per slice");
    typedef typename Acc<DT, T::MS>::type acc_t;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[T::LDS_BYTES];

    const int ntiles = tiles_m * tiles_n;
    const int split = blockIdx.x / ntiles, pid = blockIdx.x - split * ntiles;
    int tm, tn;
    tile_coords(pid, ntiles, tiles_m, tiles_n, T::GROUP_M, tm, tn);
    const int KT = Kb / splits / T::BKB;  // slices of this workgroup's K-range

    acc_t acc[T::FM][T::FN];
    pf_accumulate<DT, T, SPREAD>(lds, A, B, M, N, Kb, tm, tn, split * KT, KT, acc);

    if (splits > 1 && !splitk_fixup<DT, T>(acc, pid, split, splits, counters, partials, lds))
        return;
    pf_store<DT, T>(epi, Cv, acc, tm, tn, M, N);
}

// ---------------------------------------------------------------------------
// Register-staged variant. Same tiles, LDS layout and operand reads as the
// pipelined kernel, but the global -> LDS copy goes through registers: each
// lane loads its 16-byte chunks with ordinary global loads (NSETS slices in
// flight, so a load has NSETS slices of compute to return) and later writes
// them with ds_write_b128 to exactly the place the DMA would have filled. Two
// LDS buffers; during slice kt the waves write slice kt + 1 (from register
// set (kt + 1) % NSETS) into the buffer slice kt - 1 used, then refill that
// register set with slice kt + 1 + NSETS. The writes go in the first half of
// the slice's chunks, the refill loads in the second half, both interleaved
// with MFMAs; one barrier per slice publishes the written buffer. Index
// arithmetic near the end of K is clamped instead of branched (the surplus
// loads re-read the last slice, the surplus writes land in a buffer no one
// reads again), so every slice body is one scheduling region.

template <class T, int J0, int J1>
__device__ __forceinline__ void gload_part(i32x4 (&reg)[T::DMA_PER_WAVE], const uint8_t *const *src,
                                           int kt) {
#pragma unroll
    for (int j = J0; j < J1; ++j)
        reg[j] = *reinterpret_cast<const i32x4 *>(src[j] + (size_t)kt * T::BKB);
}

template <class T, int J0, int J1>
__device__ __forceinline__ void swrite_part(uint8_t *lds, const i32x4 (&reg)[T::DMA_PER_WAVE],
                                            int wave, int lane, int stage) {
#pragma unroll
    for (int j = J0; j < J1; ++j) {
        const int d = wave * T::DMA_PER_WAVE + j;
        *reinterpret_cast<i32x4 *>(lds + stage * T::STAGE_BYTES + d * 1024 + lane * 16) = reg[j];
    }
}

// Scheduling hint: NR LDS reads, NW LDS writes and NV global loads, each after
// one MFMA, then the remaining MFMAs.
template <int NM, int NR, int NW, int NV>
__device__ __forceinline__ void chunk_hint_rs() {
#pragma unroll
    for (int x = 0; x < NR; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
#pragma unroll
    for (int x = 0; x < NW; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
    }
#pragma unroll
    for (int x = 0; x < NV; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
    if constexpr (NM > NR + NW + NV)
        __builtin_amdgcn_sched_group_barrier(0x008, NM - NR - NW - NV, 0);
}

// Part P of NP equal parts of this wave's DMA_PER_WAVE chunks.
template <class T, int P, int NP>
struct Part {
    static constexpr int J0 = T::DMA_PER_WAVE * P / NP;
    static constexpr int J1 = T::DMA_PER_WAVE * (P + 1) / NP;
};

// Chunk kc of a slice: its share of the register -> LDS writes (chunks in the
// first half) or of the refill loads (chunks in the second half, the last
// chunk excluded).
template <class T, int KC>
__device__ __forceinline__ void rs_chunk_copy(uint8_t *lds, i32x4 (&reg)[T::DMA_PER_WAVE],
                                              const uint8_t *const *src, int wave, int lane,
                                              int wstage, int lkt) {
    constexpr int HALF = T::KCH / 2;
    if constexpr (KC < HALF) {
        swrite_part<T, Part<T, KC, HALF>::J0, Part<T, KC, HALF>::J1>(lds, reg, wave, lane, wstage);
    } else if constexpr (KC < T::KCH - 1) {
        constexpr int NPL = T::KCH - 1 - HALF;  // load slots
        gload_part<T, Part<T, KC - HALF, NPL>::J0, Part<T, KC - HALF, NPL>::J1>(reg, src, lkt);
    }
}

template <int DT, class T, int SET, int NSETS>
__device__ __forceinline__ void rs_slice(uint8_t *lds, const uint8_t *const *src, int wave, int lane,
                                         int kt, int KT, int wm, int wn, int r, int h,
                                         i32x4 (&stg)[NSETS][T::DMA_PER_WAVE], i32x4 (&ra)[2][T::FM],
                                         i32x4 (&rb)[2][T::FN],
                                         typename Acc<DT, T::MS>::type (&acc)[T::FM][T::FN]) {
    static_assert(T::STAGES == 2, "two LDS buffers");
    constexpr int NB = T::FM * T::FN;
    constexpr int MPB = (DT == S4) ? 2 : 1;
    constexpr int NRD = T::FM + T::FN;
    constexpr int HALF = T::KCH / 2;
    constexpr int NPL = T::KCH - 1 - HALF;
    const uint8_t *st = lds + (kt & 1) * T::STAGE_BYTES;
    const int wstage = (kt + 1) & 1;
    const int lkt = min(kt + 1 + NSETS, KT - 1);
    // chunk bodies 0 .. KCH-2, each with compile-time chunk index
#define MPG_RS_CHUNK(KC)                                                                       \
    if constexpr ((KC) < T::KCH - 1) {                                                         \
        constexpr int cur = (KC) & 1;                                                          \
        __builtin_amdgcn_sched_barrier(0);                                                     \
        load_runs<T>(st, (KC) + 1, wm, wn, r, h, ra[cur ^ 1], rb[cur ^ 1]);                   \
        rs_chunk_copy<T, (KC)>(lds, stg[SET], src, wave, lane, wstage, lkt);                    \
        mma_runs<DT, T, 0, NB>(ra[cur], rb[cur], acc);                                         \
        if constexpr ((KC) < HALF)                                                             \
            chunk_hint_rs<NB * MPB, NRD, Part<T, (KC), HALF>::J1 - Part<T, (KC), HALF>::J0, 0>(); \
        else                                                                                   \
            chunk_hint_rs<NB * MPB, NRD, 0,                                                    \
                          Part<T, (KC) - HALF, (NPL > 0 ? NPL : 1)>::J1 -                      \
                              Part<T, (KC) - HALF, (NPL > 0 ? NPL : 1)>::J0>();                \
        __builtin_amdgcn_sched_barrier(0);                                                     \
    }
    MPG_RS_CHUNK(0)
    MPG_RS_CHUNK(1)
    MPG_RS_CHUNK(2)
#undef MPG_RS_CHUNK
    static_assert(T::KCH <= 4, "at most 4 chunks per slice");
    // With two chunks per slice there is no load slot before the last chunk:
    // the refill loads go with the last chunk's first MFMAs.
    constexpr int last = (T::KCH - 1) & 1;
    constexpr int PRE = NB / 4;
    if constexpr (NPL == 0) gload_part<T, 0, T::DMA_PER_WAVE>(stg[SET], src, lkt);
    mma_runs<DT, T, 0, PRE>(ra[last], rb[last], acc);
    if constexpr (NPL == 0) chunk_hint_rs<PRE * MPB, 0, 0, T::DMA_PER_WAVE>();
    __builtin_amdgcn_sched_barrier(0);
    wait_vm_barrier<63>();  // LDS writes and reads done; register loads are tracked by the compiler
    load_runs<T>(lds + wstage * T::STAGE_BYTES, 0, wm, wn, r, h, ra[0], rb[0]);
    mma_runs<DT, T, PRE, NB>(ra[last], rb[last], acc);
    chunk_hint_rs<(NB - PRE) * MPB, NRD, 0, 0>();
    __builtin_amdgcn_sched_barrier(0);
}

template <int DT, class T, int NSETS>
__global__ __launch_bounds__(T::NTHREADS, 1) void tiled_gemm_rs(const uint8_t *__restrict__ A,
                                                               const uint8_t *__restrict__ B,
                                                               void *__restrict__ Cv, int M,
                                                               int N, int Kb, int tiles_m,
                                                               int tiles_n, EpiParams epi) {
    static_assert(T::KCH % 2 == 0, "even number of K-chunks per slice");
    static_assert(NSETS == 1 || NSETS == 2, "one or two register sets in flight");
    typedef typename Acc<DT, T::MS>::type acc_t;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[T::LDS_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane % T::MS, h = lane / T::MS;
    const int wm = wave / T::WGN, wn = wave % T::WGN;
    int tm, tn;
    tile_coords(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, T::GROUP_M, tm, tn);

    const uint8_t *src[T::DMA_PER_WAVE];
#pragma unroll
    for (int j = 0; j < T::DMA_PER_WAVE; ++j) {
        const int d = wave * T::DMA_PER_WAVE + j;
        src[j] = stage_src<T>(A, B, M, N, Kb, tm, tn, d, lane);
    }

    acc_t acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j) acc[i][j] = acc_t{};

    const int KT = Kb / T::BKB;
    // Prologue: slice 0 into LDS buffer 0; slices 1 .. NSETS into register
    // set s % NSETS (indices clamped to the last slice).
    i32x4 stg[NSETS][T::DMA_PER_WAVE];
    gload_part<T, 0, T::DMA_PER_WAVE>(stg[0], src, 0);
    swrite_part<T, 0, T::DMA_PER_WAVE>(lds, stg[0], wave, lane, 0);
    gload_part<T, 0, T::DMA_PER_WAVE>(stg[1 % NSETS], src, min(1, KT - 1));
    if constexpr (NSETS == 2) gload_part<T, 0, T::DMA_PER_WAVE>(stg[0], src, min(2, KT - 1));
    wait_vm_barrier<63>();

    i32x4 ra[2][T::FM], rb[2][T::FN];
    load_runs<T>(lds, 0, wm, wn, r, h, ra[0], rb[0]);

    // slice kt writes register set (kt + 1) % NSETS
    int kt = 0;
    if constexpr (NSETS == 1) {
        for (; kt < KT; ++kt)
            rs_slice<DT, T, 0, 1>(lds, src, wave, lane, kt, KT, wm, wn, r, h, stg, ra, rb, acc);
    } else {
        for (; kt + 1 < KT; kt += 2) {
            rs_slice<DT, T, 1, 2>(lds, src, wave, lane, kt, KT, wm, wn, r, h, stg, ra, rb, acc);
            rs_slice<DT, T, 0, 2>(lds, src, wave, lane, kt + 1, KT, wm, wn, r, h, stg, ra, rb, acc);
        }
        if (kt < KT)
            rs_slice<DT, T, 1, 2>(lds, src, wave, lane, kt, KT, wm, wn, r, h, stg, ra, rb, acc);
    }

    const long row0 = (long)tm * T::BM + wm * T::WTM;
    const long col0 = (long)tn * T::BN + wn * T::WTN + r;
    if constexpr (DT == S4)
        epi_store_tile<DT, T::MS, T::FM, T::FN, T::NV>(epi, Cv, acc, row0, col0, h, M, N, ConvShift8());
    else
        epi_store_tile<DT, T::MS, T::FM, T::FN, T::NV>(epi, Cv, acc, row0, col0, h, M, N, ConvSame());
}

// ---------------------------------------------------------------------------
// Ping-pong variant: 8 waves in two groups of 4, group g computing rows
// [128 g, 128 g + 128) of a 256 x 256 tile (wave tiles 128 x 64), the groups
// offset by one phase. Each K-slice takes two phases separated by workgroup
// barriers; in every phase one group runs the slice's MFMAs from LDS while
// the other writes its share of later slices from registers to LDS and
// issues its next global loads, so the MFMA pipe of each SIMD is fed by one
// wave while the other does the memory work, and a barrier never drains it:
// each group issues the last LEFT MFMA blocks of a slice after the barrier
// that ends its compute phase, while the other group's first LDS reads are in
// flight.
//
// Copy duties (two LDS buffers, buffer k % 2 holds slice k):
//   group 0, phase 2k+1: A rows 0..127 and B rows 0..127 of slice k+1;
//   group 1, phase 2k:   A rows 128..255 of slice k and B rows 128..255 of
//                        slice k+1.
// Group 0 computes slice k in phase 2k, group 1 in phase 2k+1. Every write
// lands in a buffer region whose last reader finished at least one barrier
// earlier, and every slice is complete one barrier before its first reader.
// Register loads run one copy phase (two phases) ahead of their writes.

template <class T>
struct PingPong {
    static constexpr int NA = T::BM * T::BKB / 1024;  // 1 KiB units of the A part
    static constexpr int NB = T::BN * T::BKB / 1024;  // units of the B part
    static constexpr int UA = NA / 8, UB = NB / 8;    // per wave
    static constexpr int U = UA + UB;
    static_assert(T::BM == 256 && T::BN == 256 && T::WGM == 2 && T::WGN == 4 && T::STAGES == 2,
                  "ping-pong needs 256 x 256 tiles, 2 x 4 waves, two buffers");
    static_assert(NA % 8 == 0 && NB % 8 == 0, "units split over the waves");
};

// Unit index (LDS 1 KiB block of a stage) of this wave's copy slot j.
template <class T>
__device__ __forceinline__ int pp_unit(int g, int w4, int j) {
    typedef PingPong<T> P;
    return (j < P::UA) ? g * (P::NA / 2) + w4 * P::UA + j
                       : P::NA + g * (P::NB / 2) + w4 * P::UB + (j - P::UA);
}

template <int DT, class T, int LEFT>
__device__ __forceinline__ void pp_compute(const uint8_t *st, int wm, int wn, int r, int h,
                                           i32x4 (&ra)[2][T::FM], i32x4 (&rb)[2][T::FN],
                                           typename Acc<DT, T::MS>::type (&acc)[T::FM][T::FN]) {
    constexpr int NBK = T::FM * T::FN;
    constexpr int MPB = (DT == S4) ? 2 : 1;
    constexpr int NRD = T::FM + T::FN;
    constexpr int last = (T::KCH - 1) & 1;
    __builtin_amdgcn_sched_barrier(0);
    load_runs<T>(st, 0, wm, wn, r, h, ra[0], rb[0]);
#pragma unroll
    for (int kc = 0; kc < T::KCH - 1; ++kc) {
        const int cur = kc & 1;
        __builtin_amdgcn_sched_barrier(0);
        load_runs<T>(st, kc + 1, wm, wn, r, h, ra[cur ^ 1], rb[cur ^ 1]);
        mma_runs<DT, T, 0, NBK>(ra[cur], rb[cur], acc);
        chunk_hint<NBK * MPB, NRD, 0>();
        __builtin_amdgcn_sched_barrier(0);
    }
    mma_runs<DT, T, 0, NBK - LEFT>(ra[last], rb[last], acc);
    __builtin_amdgcn_sched_barrier(0);
    wait_vm_barrier<63>();
}

// Copy phase: the LEFT MFMA blocks the group carried over (if any), the
// register -> LDS writes of this wave's slots, then the refill loads.
// Slots j < UA go to buffer `sa` (A part), the others to buffer `sb`.
template <int DT, class T, int LEFT, bool CARRY>
__device__ __forceinline__ void pp_copy(uint8_t *lds, const uint8_t *const *src,
                                        i32x4 (&stg)[PingPong<T>::U], int g, int w4, int lane,
                                        int sa, int sb, int lka, int lkb, i32x4 (&ra)[2][T::FM],
                                        i32x4 (&rb)[2][T::FN],
                                        typename Acc<DT, T::MS>::type (&acc)[T::FM][T::FN]) {
    typedef PingPong<T> P;
    constexpr int NBK = T::FM * T::FN;
    constexpr int MPB = (DT == S4) ? 2 : 1;
    constexpr int last = (T::KCH - 1) & 1;
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (CARRY) mma_runs<DT, T, NBK - LEFT, NBK>(ra[last], rb[last], acc);
#pragma unroll
    for (int j = 0; j < P::U; ++j) {
        const int d = pp_unit<T>(g, w4, j);
        const int stage = (j < P::UA) ? sa : sb;
        *reinterpret_cast<i32x4 *>(lds + stage * T::STAGE_BYTES + d * 1024 + lane * 16) = stg[j];
    }
#pragma unroll
    for (int j = 0; j < P::U; ++j) {
        const int kt = (j < P::UA) ? lka : lkb;
        stg[j] = *reinterpret_cast<const i32x4 *>(src[j] + (size_t)kt * T::BKB);
    }
    if constexpr (CARRY) chunk_hint_rs<LEFT * MPB, 0, P::U, P::U>();
    __builtin_amdgcn_sched_barrier(0);
    wait_vm_barrier<63>();
}

template <int DT, class T, int LEFT>
__global__ __launch_bounds__(512, 1) void tiled_gemm_pp(const uint8_t *__restrict__ A,
                                                       const uint8_t *__restrict__ B,
                                                       void *__restrict__ Cv, int M, int N, int Kb,
                                                       int tiles_m, int tiles_n, EpiParams epi) {
    typedef PingPong<T> P;
    static_assert(T::NTHREADS == 512, "8 waves");
    static_assert(LEFT >= 1 && LEFT < T::FM * T::FN, "carried MFMA blocks");
    typedef typename Acc<DT, T::MS>::type acc_t;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[T::LDS_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane % T::MS, h = lane / T::MS;
    const int g = wave / T::WGN, w4 = wave % T::WGN;  // group = wave row
    int tm, tn;
    tile_coords(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, T::GROUP_M, tm, tn);

    const uint8_t *src[P::U];
#pragma unroll
    for (int j = 0; j < P::U; ++j) {
        const int d = pp_unit<T>(g, w4, j);
        src[j] = stage_src<T>(A, B, M, N, Kb, tm, tn, d, lane);
    }

    acc_t acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j) acc[i][j] = acc_t{};

    const int KT = Kb / T::BKB;
    i32x4 stg[P::U];
    i32x4 ra[2][T::FM], rb[2][T::FN];
    // Prologue: group 0 writes its A and B parts of slice 0 and loads slice 1;
    // group 1 writes its B part of slice 0 and loads its A part of slice 0 and
    // its B part of slice 1 (indices clamped to the last slice).
#pragma unroll
    for (int j = 0; j < P::U; ++j) stg[j] = *reinterpret_cast<const i32x4 *>(src[j]);
#pragma unroll
    for (int j = 0; j < P::U; ++j) {
        if (g == 1 && j < P::UA) continue;
        const int d = pp_unit<T>(g, w4, j);
        *reinterpret_cast<i32x4 *>(lds + d * 1024 + lane * 16) = stg[j];
    }
    const int k1 = min(1, KT - 1);
#pragma unroll
    for (int j = 0; j < P::U; ++j) {
        const int kt = (g == 1 && j < P::UA) ? 0 : k1;
        stg[j] = *reinterpret_cast<const i32x4 *>(src[j] + (size_t)kt * T::BKB);
    }
    wait_vm_barrier<63>();

    // Phase sequence (one barrier per phase):
    //   group 0: C(0) M(0) C(1) M(1) ... C(KT-1) [carry]
    //   group 1: M'(0) C(0) M'(1) C(1) ... M'(KT-1) C(KT-1) [carry]
    // with C(k) = MFMAs of slice k from buffer k % 2, M(k) = write A0, B0 of
    // slice k+1 and load slice k+2, M'(k) = write A1 of slice k and B1 of
    // slice k+1, load A1 of slice k+1 and B1 of slice k+2. Both groups run
    // the same loop body "C(k), copy"; group 1 enters it one phase later.
    if (g == 1)
        pp_copy<DT, T, LEFT, false>(lds, src, stg, g, w4, lane, 0, min(1, KT - 1) & 1,
                                    min(1, KT - 1), min(2, KT - 1), ra, rb, acc);
    for (int k = 0; k + 1 < KT; ++k) {
        pp_compute<DT, T, LEFT>(lds + (k & 1) * T::STAGE_BYTES, g, w4, r, h, ra, rb, acc);
        // group 0: M(k); group 1: M'(k + 1)
        const int sa = (k + 1) & 1;
        const int sb = (g == 0) ? (k + 1) & 1 : k & 1;
        const int lka = min(k + 2, KT - 1);
        const int lkb = min(g == 0 ? k + 2 : k + 3, KT - 1);
        pp_copy<DT, T, LEFT, true>(lds, src, stg, g, w4, lane, sa, sb, lka, lkb, ra, rb, acc);
    }
    pp_compute<DT, T, LEFT>(lds + ((KT - 1) & 1) * T::STAGE_BYTES, g, w4, r, h, ra, rb, acc);
    {
        constexpr int last = (T::KCH - 1) & 1;
        mma_runs<DT, T, T::FM * T::FN - LEFT, T::FM * T::FN>(ra[last], rb[last], acc);
    }
    // group 0's last phase, matching the barrier of group 1's last compute
    if (g == 0) wait_vm_barrier<63>();

    const long row0 = (long)tm * T::BM + g * T::WTM;
    const long col0 = (long)tn * T::BN + w4 * T::WTN + r;
    if constexpr (DT == S4)
        epi_store_tile<DT, T::MS, T::FM, T::FN, T::NV>(epi, Cv, acc, row0, col0, h, M, N, ConvShift8());
    else
        epi_store_tile<DT, T::MS, T::FM, T::FN, T::NV>(epi, Cv, acc, row0, col0, h, M, N, ConvSame());
}

template <int DT, class T>
__global__ __launch_bounds__(T::NTHREADS, 1) void tiled_gemm(const uint8_t *__restrict__ A,
                                                            const uint8_t *__restrict__ B,
                                                            void *__restrict__ Cv, int M, int N,
                                                            int Kb, int tiles_m, int tiles_n, EpiParams epi) {
    typedef typename Acc<DT, T::MS>::type acc_t;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[T::LDS_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane % T::MS, h = lane / T::MS;
    const int wm = wave / T::WGN, wn = wave % T::WGN;
    int tm, tn;
    tile_coords(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, T::GROUP_M, tm, tn);

    // Source of each of this wave's DMA loads (stage-independent part).
    const uint8_t *src[T::DMA_PER_WAVE];
#pragma unroll
    for (int j = 0; j < T::DMA_PER_WAVE; ++j) {
        const int d = wave * T::DMA_PER_WAVE + j;
        src[j] = stage_src<T>(A, B, M, N, Kb, tm, tn, d, lane);
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

    const long row0 = (long)tm * T::BM + wm * T::WTM;
    const long col0 = (long)tn * T::BN + wn * T::WTN + r;
    if constexpr (DT == S4)
        epi_store_tile<DT, T::MS, T::FM, T::FN, T::NV>(epi, Cv, acc, row0, col0, h, M, N, ConvShift8());
    else
        epi_store_tile<DT, T::MS, T::FM, T::FN, T::NV>(epi, Cv, acc, row0, col0, h, M, N, ConvSame());
}

}  // namespace mpg
