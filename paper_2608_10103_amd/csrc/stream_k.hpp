// stream_k.hpp - stream-K schedules of the pipelined and the one-wave-per-SIMD
// kernels (FP16, INT8, and INT4 on the FP6 cores), for problems whose tile count leaves the last round of workgroups
// partly idle.
//
// A problem of T tiles, each KT K-slices deep, is T * KT iterations (one
// slice of one tile). With G workgroups resident at once (one per CU for
// these kernels) and T = q G + r, 0 < r <= G / 2, plain tiling runs q + 1
// rounds, the last with r busy CUs. Here the first q G tiles stay whole, one
// workgroup each, launched first ("data-parallel" rounds); the iterations of
// the r remaining tiles are then shared out over r * s further workgroups,
// s = min(G / r, 8) contiguous K-parts per tile (whole slices each, sizes
// differing by at most one), so the last round fills up to G CUs and takes
// about 1 / s of a tile's time plus the fixup.
//
// Why not the other stream-K partitions. Giving each of G workgroups an
// equal range of the last G + r tiles' iterations (so ranges straddle tile
// boundaries) measured slower than plain tiling on MI355X at 272-688 tiles
// of 256 x 256 (1.5-1.8x with INT8, 1.2-1.4x with FP16 at K = 4096), also
// with the ranges of each XCD contiguous, and no faster with the fixup's
// fences and partial traffic removed: the ranges start at different K
// offsets, so the workgroups that run together on one XCD no longer stream
// the same panel slices through its 4 MB L2, and every tile's panels come
// from HBM again. Data-parallel rounds keep that sharing; only the
// remainder, r tiles read once each, runs split.
//
// Fixup of a split tile: every part stores its partial tile to its slot and
// counts itself in the tile's counter (stores, device-scope release, atomic
// add). The part that brings the count to s loads the s partials in part
// order 0, 1, ..., s - 1 and writes C, so the sum does not depend on which
// part finishes last; it resets the counter. No workgroup waits for another.
//
// Workspace: the caller's 64 KiB counter block (counter t belongs to tile t;
// zero before the first call, left zero by every call), then r s partial
// slots of BM x BN 32-bit words, slot u for remainder workgroup u.
#pragma once

#include "wide_f6.hpp"
#include "wide_gemm.hpp"

namespace mpg {

struct SkArgs {
    int dp_tiles;        // tiles computed whole, by workgroups 0 .. dp_tiles - 1
    int parts;           // K-parts of every remaining tile, one workgroup each
    int *counters;       // one per tile
    uint32_t *partials;  // one slot per remainder workgroup
};

// Work of workgroup b: tile t (an index in grouped order, see grouped_tile)
// and its K-slices [k0, k0 + len), part `part` of the tile. Whole tiles go
// to XCD-contiguous ranks of the first dp_tiles workgroups, so the
// workgroups that run together on one XCD share panels as in the plain
// kernels. u: the remainder workgroup's index (its slot), or -1 for a whole
// tile.
struct SkWork {
    int t, k0, len, part, u;
};

__device__ __forceinline__ SkWork sk_work(int b, const SkArgs &sk, int KT) {
    if (b < sk.dp_tiles) return SkWork{xcd_rank(b, sk.dp_tiles), 0, KT, -1, -1};
    const int u = b - sk.dp_tiles, j = u % sk.parts;
    const int k0 = (int)((long)j * KT / sk.parts), k1 = (int)((long)(j + 1) * KT / sk.parts);
    return SkWork{sk.dp_tiles + u / sk.parts, k0, k1 - k0, j, u};
}

// Fixup of a split tile (see the top of this file); acc holds this part,
// slots the tile's first slot. Returns true in the part that must write C,
// with acc replaced by the sum of all parts in part order (its own part
// taken from its registers, the others loaded). Slot layout: quad w (values
// 4w .. 4w + 3) of block (i, j) of thread t in the 16 bytes at vector index
// ((i FN + j) NQ + w) NT + t, NQ = NV / 4, so each wave's store or load
// instruction covers 1 KiB. The sum is formed a few blocks at a time (see
// below), each part's loads of them
// issued together; this keeps the registers it needs bounded. AGPR: the
// accumulators live in AGPRs (the one-wave-per-SIMD kernels); each finished
// block is put back there at once, or the compiler keeps all sums in VGPRs
// and spills.
template <class OutT, int FM, int FN, int NV, int NT, bool AGPR = false, class AccT>
__device__ __forceinline__ bool sk_fixup(AccT (&acc)[FM][FN], int *counter, uint32_t *slots, int part,
                                         int parts, int *flag) {
    typedef OutT V __attribute__((ext_vector_type(4)));
    constexpr int NQ = NV / 4;
    constexpr size_t SLOT = (size_t)FM * FN * NQ * NT;  // in 16-byte vectors
    static_assert(NV % 4 == 0, "accumulator blocks of whole quads");
    const int tid = threadIdx.x;
    V *base = reinterpret_cast<V *>(slots);
    auto quad = [&](const AccT &blk, int w) __attribute__((always_inline)) {
        return V{(OutT)blk[4 * w], (OutT)blk[4 * w + 1], (OutT)blk[4 * w + 2], (OutT)blk[4 * w + 3]};
    };
    V *mine = base + (size_t)part * SLOT;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int w = 0; w < NQ; ++w) mine[((i * FN + j) * NQ + w) * NT + tid] = quad(acc[i][j], w);
    // every wave's stores have reached L2 before thread 0 releases them
    // device-wide (the release writes back the L2, whichever wave wrote)
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0) {
        __threadfence();
        const int last = atomicAdd(counter, 1) == parts - 1;
        if (last) __threadfence();  // acquire: the other parts' partials are visible
        flag[0] = last;
    }
    __syncthreads();
    if (!flag[0]) return false;
    // blocks per step: with the accumulators in AGPRs, two block rows of
    // 16x16 blocks (64 values per lane) or one 32x32 block (16 values; more
    // spills); else a block row (the VGPRs hold the accumulators too)
    constexpr int NB = FM * FN;
    constexpr int S = AGPR ? (NV >= 16 ? 1 : 64 / NV) : FN;
    static_assert(NB % S == 0, "whole steps");
#pragma unroll
    for (int b0 = 0; b0 < NB; b0 += S) {
        V sum[S][NQ];
        for (int q = 0; q < parts; ++q) {
            V add[S][NQ];
            if (q == part) {
#pragma unroll
                for (int b = 0; b < S; ++b)
#pragma unroll
                    for (int w = 0; w < NQ; ++w) add[b][w] = quad(acc[(b0 + b) / FN][(b0 + b) % FN], w);
            } else {
                const V *p = base + (size_t)q * SLOT;
#pragma unroll
                for (int b = 0; b < S; ++b)
#pragma unroll
                    for (int w = 0; w < NQ; ++w) add[b][w] = p[((b0 + b) * NQ + w) * NT + tid];
            }
#pragma unroll
            for (int b = 0; b < S; ++b)
#pragma unroll
                for (int w = 0; w < NQ; ++w) sum[b][w] = q == 0 ? add[b][w] : sum[b][w] + add[b][w];
        }
#pragma unroll
        for (int b = 0; b < S; ++b) {
            AccT &blk = acc[(b0 + b) / FN][(b0 + b) % FN];
#pragma unroll
            for (int w = 0; w < NQ; ++w)
#pragma unroll
                for (int e = 0; e < 4; ++e) blk[4 * w + e] = sum[b][w][e];
            if constexpr (AGPR) asm volatile("" : "+a"(blk));
        }
    }
    if (tid == 0) *counter = 0;  // ready for the next call on this workspace
    return true;
}

// Stream-K schedule of the pipelined kernel (tiled_gemm_pf): grid =
// dp_tiles + (remaining tiles) * parts; M and N may be ragged.
template <int DT, class T, bool SPREAD>
__global__ __launch_bounds__(T::NTHREADS, 1) void tiled_gemm_sk(const uint8_t *__restrict__ A,
                                                               const uint8_t *__restrict__ B,
                                                               void *__restrict__ Cv, int M, int N, int Kb,
                                                               int tiles_m, int tiles_n, SkArgs sk,
                                                               EpiParams epi) {
    static_assert(T::KCH % 2 == 0, "even number of K-chunks per slice");
    typedef typename Acc<DT, T::MS>::out out_t;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[T::LDS_BYTES];
    const SkWork wk = sk_work(blockIdx.x, sk, Kb / T::BKB);
    int tm, tn;
    grouped_tile(wk.t, tiles_m, tiles_n, T::GROUP_M, tm, tn);
    typename Acc<DT, T::MS>::type acc[T::FM][T::FN];
    pf_accumulate<DT, T, SPREAD>(lds, A, B, M, N, Kb, tm, tn, wk.k0, wk.len, acc);
    // The fixup's flag lives in the copy buffers: after the last slice's
    // barrier no wave reads what it overwrites. (A separate LDS variable would
    // make the compiler wait for every copy in flight before each LDS read.)
    if (wk.u >= 0 &&
        !sk_fixup<out_t, T::FM, T::FN, T::NV, T::NTHREADS>(
            acc, sk.counters + wk.t, sk.partials + (size_t)(wk.u - wk.part) * T::BM * T::BN, wk.part, sk.parts,
            reinterpret_cast<int *>(lds)))
        return;
    pf_store<DT, T>(epi, Cv, acc, tm, tn, M, N);
}

// Stream-K schedule of the one-wave-per-SIMD kernel (wide_gemm): 256 x 256
// tiles (ragged edges as there), grid as for tiled_gemm_sk.
template <int DT, bool PLAIN = true, int AUX = CP_DEFAULT>
__global__ __launch_bounds__(WideCfg::NTHREADS, 1) void wide_gemm_sk(const uint8_t *__restrict__ A,
                                                                    const uint8_t *__restrict__ B,
                                                                    void *__restrict__ Cv, int M, int N, int Kb,
                                                                    int tiles_m, int tiles_n, SkArgs sk,
                                                                    EpiParams epi) {
    static_assert(DT == F16 || DT == S8, "FP16 and INT8");
    typedef typename Acc<DT, 16>::out out_t;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[WideCfg::LDS_BYTES];
    const SkWork wk = sk_work(blockIdx.x, sk, Kb / WideCfg::BKB);
    int tm, tn;
    grouped_tile(wk.t, tiles_m, tiles_n, 4, tm, tn);
    typename Acc<DT, 16>::type acc[8][8];
    wide_accumulate<DT, AUX>(lds, A, B, M, N, Kb, tm, tn, wk.k0, wk.len, acc);
    // flag in the copy buffers, as in tiled_gemm_sk
    if (wk.u >= 0 &&
        !sk_fixup<out_t, 8, 8, 4, WideCfg::NTHREADS, true>(
            acc, sk.counters + wk.t, sk.partials + (size_t)(wk.u - wk.part) * WideCfg::BM * WideCfg::BN, wk.part,
            sk.parts, reinterpret_cast<int *>(lds)))
        return;
    wide_store<DT, PLAIN>(epi, Cv, acc, tm, tn, M, N);
}

// Stream-K schedule of the one-wave-per-SIMD FP6 kernel (wide_f6_gemm,
// INT4 on operands converted by the pre-pass): whole 256 x 256 tiles of
// 128-k slices, grid as for tiled_gemm_sk. The parts add their FP32 sums,
// integers whose magnitudes add up to at most 64 K < 2^24, so the sum of the
// parts is exact in any order.
template <bool PLAIN, int AUX = CP_DEFAULT>
__global__ __launch_bounds__(WideF6Cfg::NTHREADS, 1) void wide_f6_gemm_sk(
    const uint8_t *__restrict__ Ap, const uint8_t *__restrict__ Aq, const uint8_t *__restrict__ Bp,
    const uint8_t *__restrict__ Bq, int32_t *__restrict__ C, int M, int N, int Ma, int Nb, int KT, int tiles_m,
    int tiles_n, SkArgs sk, EpiParams epi) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[WideF6Cfg::LDS_BYTES];
    wf6_entry_args<PLAIN>(C, M, N, epi);
    const SkWork wk = sk_work(blockIdx.x, sk, KT);
    int tm, tn;
    grouped_tile(wk.t, tiles_m, tiles_n, 4, tm, tn);
    f32x16 acc[4][4];
    wf6_accumulate<AUX>(lds, Ap, Aq, Bp, Bq, Ma, Nb, KT, tm, tn, wk.k0, wk.len, acc);
    // flag in the copy buffers, as in tiled_gemm_sk
    if (wk.u >= 0 &&
        !sk_fixup<float, 4, 4, 16, WideF6Cfg::NTHREADS, true>(
            acc, sk.counters + wk.t, sk.partials + (size_t)(wk.u - wk.part) * WideF6Cfg::BM * WideF6Cfg::BN,
            wk.part, sk.parts, reinterpret_cast<int *>(lds)))
        return;
    wf6_store<PLAIN>(epi, C, acc, tm, tn, M, N);
}

}  // namespace mpg
