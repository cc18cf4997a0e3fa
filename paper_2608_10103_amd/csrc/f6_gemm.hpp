// f6_gemm.hpp - INT4 GEMM on the FP6 matrix cores.
//
// gfx950 has no 4-bit integer MFMA, but its f8f6f4 MFMA multiplies FP6 values
// at twice the INT8 rate (32x32x64 per instruction). Every INT4 value v in
// [-8, 7] is exactly representable in FP6 E3M2 (1 sign, 3 exponent bits with
// bias 3, 2 mantissa bits: 0, 1, 2, 3, 4, 5, 6, 7 and 8 are all normal or
// zero), each product of two is an integer of magnitude <= 64, and the FP32
// accumulator holds every partial sum exactly while it stays <= 2^24, i.e.
// for K <= 2^18. The result, converted to int32, is the exact INT4 GEMM
// D = A B (the paper's MMA primitive D = AB + C, Background, started from
// zero) with the INT32 accumulation of its INT4 MMA (Listing
// "lst:int4-primitives", part (c); Results and Analysis, Run 3).
//
// Two kernels:
//  * s4_to_e3m2 converts each operand once (A: M rows, B: N columns, both
//    K-contiguous packed nibbles, low nibble = even k) into a workspace in a
//    run-major layout. A run is 32 consecutive k of one row: 32 six-bit
//    codes = 24 bytes (in the field order of s4_run_to_e3m2), split into a 16-byte part P (bits 0..127) and an
//    8-byte part Q (bits 128..191). The workspace of an operand with R rows
//    holds P[j][r] (16 bytes) for run j and row r, rows padded to R_pad
//    (multiple of 256) and runs to J_pad (K padded to a multiple of 256)
//    with zero codes, then Q[j][r] (8 bytes) in the same order. Rows of one
//    run are contiguous, so one wave-wide DMA copies 64 rows of P or 128
//    rows of Q into 1 KiB of LDS, and the MFMA operand reads of 32
//    consecutive rows are contiguous in LDS: no swizzle, no bank conflicts.
//  * f6_gemm is the pipelined tile kernel (the structure of tiled_gemm_pf,
//    non-spread form): BM x BN tile per workgroup, J runs (32 J k) per LDS
//    stage, STAGES-deep DMA ring, one wait + barrier per stage, operand
//    fragments double-buffered in registers. Lane l of a wave supplies run
//    (2 kc + l / 32) of row / column l % 32 for MFMA k-chunk kc; A and B use
//    the same assignment, so the MFMA sums over exactly the k of the chunk.
#pragma once

#include "device_common.hpp"
#include "tiled_gemm.hpp"

namespace mpg {

typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef int i32x6 __attribute__((ext_vector_type(6)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

// E3M2 code of a two's-complement nibble n (value n for n < 8, n - 16
// otherwise). Byte n & 7 of the first constant encodes 0..7, of the second
// -8..-1: magnitude m >= 1 is 2^e (1 + f / 4) with code (e + 3) << 2 | f, and
// the sign is bit 5.
constexpr uint64_t kE3M2Pos = 0x1716151412100C00ull, kE3M2Neg = 0x2C30323435363738ull;

__host__ __device__ constexpr uint32_t e3m2_code(uint32_t n) {
    return (uint32_t)(((n & 8u) ? kE3M2Neg : kE3M2Pos) >> (8u * (n & 7u))) & 0x3Fu;
}

// Byte permute: byte i of the result is byte sel_i (0..7) of the 64-bit
// value hi:lo (v_perm_b32 on the device; selectors 0..7 only).
__host__ __device__ inline uint32_t byte_perm(uint32_t hi, uint32_t lo, uint32_t sel) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_perm(hi, lo, sel);
#else
    const uint64_t v = ((uint64_t)hi << 32) | lo;
    uint32_t r = 0;
    for (int i = 0; i < 4; ++i) r |= (uint32_t)((v >> (8 * ((sel >> (8 * i)) & 7))) & 0xFF) << (8 * i);
    return r;
#endif
}

// E3M2 codes of four nibbles held one per byte (values 0..15): two 8-entry
// table lookups by byte permute, then per byte the one its bit 3 selects.
__host__ __device__ inline uint32_t e3m2_codes4(uint32_t b) {
    const uint32_t idx = b & 0x07070707u;
    const uint32_t pos = byte_perm((uint32_t)(kE3M2Pos >> 32), (uint32_t)kE3M2Pos, idx);
    const uint32_t neg = byte_perm((uint32_t)(kE3M2Neg >> 32), (uint32_t)kE3M2Neg, idx);
    const uint32_t m8 = b & 0x08080808u;
    const uint32_t mask = (m8 << 3) - (m8 >> 3);  // 0x3F in the bytes of negative nibbles
    return (neg & mask) | (pos & ~mask);
}

// Four 6-bit codes, one per byte -> 24 bits, byte i at bits [6 i, 6 i + 6).
__host__ __device__ inline uint32_t pack6x4(uint32_t c) {
    const uint32_t p = (c & 0x003F003Fu) | ((c >> 2) & 0x0FC00FC0u);
    return (p & 0xFFFu) | ((p >> 4) & 0xFFF000u);
}

// One run: 16 bytes = 32 nibbles -> 32 E3M2 codes in a 192-bit string
// out[0..5] (little-endian), code of field f at bits [6 f, 6 f + 6). Field
// f = 8 d + 4 h + i holds nibble 8 d + 2 i + h (input word d, byte i, low
// nibble h = 0 or high nibble h = 1): the low nibbles of a word come first,
// then its high nibbles. Any fixed assignment of k to fields works because A
// and B are converted alike and the MFMA sums over all 64 fields of a lane
// pair.
__host__ __device__ inline void s4_run_to_e3m2(const uint32_t (&in)[4], uint32_t (&out)[6]) {
    uint32_t q[8];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        q[2 * d] = pack6x4(e3m2_codes4(in[d] & 0x0F0F0F0Fu));
        q[2 * d + 1] = pack6x4(e3m2_codes4((in[d] >> 4) & 0x0F0F0F0Fu));
    }
#pragma unroll
    for (int g = 0; g < 2; ++g) {  // 4 chunks of 24 bits -> 3 words
        const uint32_t *c = q + 4 * g;
        out[3 * g] = c[0] | (c[1] << 24);
        out[3 * g + 1] = (c[1] >> 8) | (c[2] << 16);
        out[3 * g + 2] = (c[2] >> 16) | (c[3] << 8);
    }
}

// Workspace geometry of one operand (R rows, K columns).
struct F6Geom {
    static constexpr int ROW_PAD = 256, K_PAD = 256;
    static __host__ __device__ long rows_pad(long R) { return (R + ROW_PAD - 1) / ROW_PAD * ROW_PAD; }
    static __host__ __device__ long runs_pad(long K) { return (K + K_PAD - 1) / K_PAD * (K_PAD / 32); }
    // bytes: P part then Q part
    static __host__ __device__ uint64_t bytes(long R, long K) {
        return (uint64_t)rows_pad(R) * (uint64_t)runs_pad(K) * 24u;
    }
};

struct F6Prep {
    const uint8_t *src;  // R rows of K / 2 bytes
    uint8_t *p, *q;      // workspace parts
    int rows, rows_pad, K, runs;
};

// Conversion kernel. A block converts a tile of 32 rows x 32 runs of one
// operand (blockIdx.z: 0 = A, 1 = B) and transposes it through LDS: the
// reads are 512 contiguous bytes per row, the writes 512 contiguous bytes
// (P) or 256 (Q) per run. LDS rows of a run are padded to 33 entries so the
// transposing accesses of 16 (P) or 32 (Q) lanes hit distinct banks. Rows
// and runs past the data are written as zero codes. (Two tiles per block,
// the second's loads issued before the first is converted, measured slower:
// 13.4 against 11.7 us at 4096^3.)
constexpr int F6_PREP_ROWS = 32, F6_PREP_RUNS = 32, F6_PREP_PITCH = 33;

// The four runs of lane t in the tile at rows r0, runs j0 (rows t / 32 + 8 i,
// run t % 32): all four loads issued together where the tile lies inside
// the data and rows are 16-byte aligned, byte by byte (zeros past the data)
// otherwise.
__device__ __forceinline__ void f6_prep_load(const F6Prep &o, int r0, int j0, int t, uint32_t (&in)[4][4]) {
    const long kb = o.K / 2;
    const bool whole = r0 + F6_PREP_ROWS <= o.rows && (long)(j0 + F6_PREP_RUNS) * 16 <= kb && kb % 16 == 0 &&
                       (reinterpret_cast<uintptr_t>(o.src) & 15) == 0;
    if (whole) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const i32x4 v = *reinterpret_cast<const i32x4 *>(o.src + (size_t)(r0 + (t >> 5) + 8 * i) * kb +
                                                             (long)(j0 + (t & 31)) * 16);
#pragma unroll
            for (int e = 0; e < 4; ++e) in[i][e] = (uint32_t)v[e];
        }
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = r0 + (t >> 5) + 8 * i, j = j0 + (t & 31);
#pragma unroll
            for (int e = 0; e < 4; ++e) in[i][e] = 0;
            if (r < o.rows && j < o.runs) {
                const long b0 = (long)j * 16;
                const uint8_t *rowp = o.src + (size_t)r * kb;
                for (int e = 0; e < 16 && b0 + e < kb; ++e) in[i][e >> 2] |= (uint32_t)rowp[b0 + e] << (8 * (e & 3));
            }
        }
    }
}

inline __global__ __launch_bounds__(256) void s4_to_e3m2(F6Prep a, F6Prep b) {
    __shared__ __attribute__((aligned(16))) uint8_t lp[F6_PREP_RUNS * F6_PREP_PITCH * 16];
    __shared__ __attribute__((aligned(16))) uint8_t lq[F6_PREP_RUNS * F6_PREP_PITCH * 8];
    const F6Prep &o = blockIdx.z ? b : a;
    const int r0 = blockIdx.y * F6_PREP_ROWS, j0 = blockIdx.x * F6_PREP_RUNS;
    if (r0 >= o.rows_pad) return;  // the other operand has more rows; uniform per block
    const int t = threadIdx.x;
    uint32_t in[4][4];
    f6_prep_load(o, r0, j0, t, in);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int rl = (t >> 5) + 8 * i, jl = t & 31;
        uint32_t out[6];
        s4_run_to_e3m2(in[i], out);
        const int slot = jl * F6_PREP_PITCH + rl;
        *reinterpret_cast<i32x4 *>(lp + slot * 16) = i32x4{(int)out[0], (int)out[1], (int)out[2], (int)out[3]};
        *reinterpret_cast<i32x2 *>(lq + slot * 8) = i32x2{(int)out[4], (int)out[5]};
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {  // P: 32 runs x 32 rows x 16 bytes
        const int idx = t + 256 * i, jl = idx >> 5, rl = idx & 31;
        if (j0 + jl < o.runs)
            *reinterpret_cast<i32x4 *>(o.p + ((size_t)(j0 + jl) * o.rows_pad + r0 + rl) * 16) =
                *reinterpret_cast<const i32x4 *>(lp + (jl * F6_PREP_PITCH + rl) * 16);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {  // Q: 32 runs x 16 row pairs x 16 bytes
        const int idx = t + 256 * i, jl = idx >> 4, rl = 2 * (idx & 15);
        if (j0 + jl < o.runs) {
            const i32x2 q0 = *reinterpret_cast<const i32x2 *>(lq + (jl * F6_PREP_PITCH + rl) * 8);
            const i32x2 q1 = *reinterpret_cast<const i32x2 *>(lq + (jl * F6_PREP_PITCH + rl + 1) * 8);
            *reinterpret_cast<i32x4 *>(o.q + ((size_t)(j0 + jl) * o.rows_pad + r0 + rl) * 8) =
                i32x4{q0[0], q0[1], q1[0], q1[1]};
        }
    }
}

template <int BM_, int BN_, int WGM_, int WGN_, int J_, int STAGES_, int GROUP_M_>
struct F6Cfg {
    static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_, J = J_;
    static constexpr int STAGES = STAGES_, GROUP_M = GROUP_M_;
    static constexpr int NWAVES = WGM * WGN, NTHREADS = 64 * NWAVES;
    static constexpr int WTM = BM / WGM, WTN = BN / WGN;
    static constexpr int FM = WTM / 32, FN = WTN / 32;
    static constexpr int KCH = J / 2;                 // MFMA k-chunks (64 k) per stage
    static constexpr int BK = 32 * J;                 // k per stage
    static constexpr int AQ_OFF = J * BM * 16;        // LDS offsets inside a stage
    static constexpr int BP_OFF = J * BM * 24;
    static constexpr int BQ_OFF = BP_OFF + J * BN * 16;
    static constexpr int STAGE_BYTES = J * (BM + BN) * 24;
    static constexpr int LDS_BYTES = STAGES * STAGE_BYTES;
    static constexpr int UAP = J * BM / 64, UAQ = J * BM / 128;  // 1 KiB DMA units per stage
    static constexpr int UBP = J * BN / 64, UBQ = J * BN / 128;
    static constexpr int NDMA = UAP + UAQ + UBP + UBQ;
    static constexpr int DPW = NDMA / NWAVES;
    static_assert(NDMA * 1024 == STAGE_BYTES, "stage is whole DMA units");
    static_assert(BM % 128 == 0 && BN % 128 == 0, "a Q unit (128 rows) stays inside one run");
    static_assert(F6Geom::ROW_PAD % BM == 0 && F6Geom::ROW_PAD % BN == 0, "tiles stay in padded rows");
    static_assert((32 * J) <= F6Geom::K_PAD && F6Geom::K_PAD % (32 * J) == 0, "stages tile padded K");
    static_assert(KCH % 2 == 0, "even number of k-chunks per stage");
    static_assert(FM >= 1 && FN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile");
    static_assert(NDMA % NWAVES == 0, "DMA units split evenly over waves");
    static_assert(STAGES >= 2 && (STAGES - 2) * DPW <= 63, "vmcnt range");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS capacity");
};

// Operand fragment of one 32x32x64 MFMA: a lane's run, the P part in
// elements 0..3 and the Q part in elements 4..5 (six consecutive VGPRs).
typedef i32x6 F6Frag;

// Read a fragment from LDS at byte offsets p_off (16-byte P part) and q_off
// (8-byte Q part). The Q offset goes through an empty asm so the compiler
// cannot see that the Q parts of neighbouring fragments are a constant
// distance apart: it would merge their 8-byte reads into one ds_read2_b64,
// whose result then has to be waited for and copied into place.
__device__ __forceinline__ F6Frag f6_frag(const uint8_t *lds, int p_off, int q_off) {
    asm("" : "+v"(q_off));
    const i32x4 pv = *reinterpret_cast<const i32x4 *>(lds + p_off);
    const i32x2 qv = *reinterpret_cast<const i32x2 *>(lds + q_off);
    return __builtin_shufflevector(pv, __builtin_shufflevector(qv, qv, 0, 1, -1, -1), 0, 1, 2, 3, 4, 5);
}

__device__ __forceinline__ f32x16 mfma_e3m2(F6Frag a, F6Frag b, f32x16 c) {
    // format 3 = FP6 E3M2 for both operands (six VGPRs each); unit scales
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
        __builtin_shufflevector(a, a, 0, 1, 2, 3, 4, 5, -1, -1),
        __builtin_shufflevector(b, b, 0, 1, 2, 3, 4, 5, -1, -1), c, 3, 3, 0, 0, 0, 0);
}

// Source address of lane `lane` in DMA unit d of the stage for slice 0, and
// the byte step from one slice to the next. Units: A P, A Q, B P, B Q.
template <class T>
__device__ __forceinline__ const uint8_t *f6_unit_src(const uint8_t *Ap, const uint8_t *Aq,
                                                      const uint8_t *Bp, const uint8_t *Bq,
                                                      long Ma, long Nb, int tm, int tn, int d,
                                                      int lane, long &step) {
    if (d < T::UAP) {
        const int j = d / (T::BM / 64), q = (d % (T::BM / 64)) * 64 + lane;
        step = (long)T::J * Ma * 16;
        return Ap + ((size_t)j * Ma + (size_t)tm * T::BM + q) * 16;
    }
    d -= T::UAP;
    if (d < T::UAQ) {
        const int j = d / (T::BM / 128), q = (d % (T::BM / 128)) * 128 + 2 * lane;
        step = (long)T::J * Ma * 8;
        return Aq + ((size_t)j * Ma + (size_t)tm * T::BM + q) * 8;
    }
    d -= T::UAQ;
    if (d < T::UBP) {
        const int j = d / (T::BN / 64), q = (d % (T::BN / 64)) * 64 + lane;
        step = (long)T::J * Nb * 16;
        return Bp + ((size_t)j * Nb + (size_t)tn * T::BN + q) * 16;
    }
    d -= T::UBP;
    const int j = d / (T::BN / 128), q = (d % (T::BN / 128)) * 128 + 2 * lane;
    step = (long)T::J * Nb * 8;
    return Bq + ((size_t)j * Nb + (size_t)tn * T::BN + q) * 8;
}

template <class T>
__device__ __forceinline__ void f6_issue(uint8_t *lds, const uint8_t *const *src, const long *step,
                                         int wave, int stage, int kt) {
#pragma unroll
    for (int u = 0; u < T::DPW; ++u)
        dma16(src[u] + (size_t)kt * step[u], lds + stage * T::STAGE_BYTES + (wave * T::DPW + u) * 1024);
}

// Fragments of k-chunk kc from the stage at byte offset so of the LDS ring.
template <class T>
__device__ __forceinline__ void f6_load(const uint8_t *lds, int so, int kc, int wm, int wn, int r,
                                        int h, F6Frag (&a)[T::FM], F6Frag (&b)[T::FN]) {
    const int jj = 2 * kc + h;
#pragma unroll
    for (int i = 0; i < T::FM; ++i) {
        const int q = jj * T::BM + wm * T::WTM + i * 32 + r;
        a[i] = f6_frag(lds, so + q * 16, so + T::AQ_OFF + q * 8);
    }
#pragma unroll
    for (int j = 0; j < T::FN; ++j) {
        const int q = jj * T::BN + wn * T::WTN + j * 32 + r;
        b[j] = f6_frag(lds, so + T::BP_OFF + q * 16, so + T::BQ_OFF + q * 8);
    }
}

template <class T, int P0, int P1>
__device__ __forceinline__ void f6_mma(const F6Frag (&a)[T::FM], const F6Frag (&b)[T::FN],
                                       f32x16 (&acc)[T::FM][T::FN]) {
#pragma unroll
    for (int p = P0; p < P1; ++p) acc[p / T::FN][p % T::FN] = mfma_e3m2(a[p / T::FN], b[p % T::FN], acc[p / T::FN][p % T::FN]);
}

// Scheduling hint: NR LDS reads spread evenly over NM MFMAs, one DMA load
// after each of the first NV MFMAs.
template <int NM, int NR, int NV, int X = 0>
__device__ __forceinline__ void f6_hint() {
    if constexpr (X < NM) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        constexpr int nr = (NR * (X + 1)) / NM - (NR * X) / NM;
        if constexpr (nr > 0) __builtin_amdgcn_sched_group_barrier(0x100, nr, 0);  // LDS reads
        if constexpr (X < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // one DMA
        f6_hint<NM, NR, NV, X + 1>();
    }
}

// One stage (slice kt in buffer kt % STAGES); ISSUE: also start the copy of
// slice kt + STAGES into the buffer this stage frees at its barrier.
template <class T, bool ISSUE>
__device__ __forceinline__ void f6_slice(uint8_t *lds, const uint8_t *const *src, const long *step,
                                         int wave, int kt, int wm, int wn, int r, int h,
                                         F6Frag (&ra)[2][T::FM], F6Frag (&rb)[2][T::FN],
                                         f32x16 (&acc)[T::FM][T::FN]) {
    constexpr int NB = T::FM * T::FN;
    constexpr int NRD = 2 * (T::FM + T::FN);
    constexpr int S = T::STAGES;
    const int so = (kt % S) * T::STAGE_BYTES;
#pragma unroll
    for (int kc = 0; kc < T::KCH - 1; ++kc) {
        const int cur = kc & 1;
        __builtin_amdgcn_sched_barrier(0);
        f6_load<T>(lds, so, kc + 1, wm, wn, r, h, ra[cur ^ 1], rb[cur ^ 1]);
        f6_mma<T, 0, NB>(ra[cur], rb[cur], acc);
        f6_hint<NB, NRD, 0>();
        __builtin_amdgcn_sched_barrier(0);
    }
    constexpr int last = (T::KCH - 1) & 1;
    constexpr int PRE = NB / 4 > 0 ? NB / 4 : 1;
    f6_mma<T, 0, PRE>(ra[last], rb[last], acc);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (ISSUE) wait_vm_barrier<(S - 2) * T::DPW>();
    else wait_vm_barrier<0>();
    if constexpr (ISSUE) f6_issue<T>(lds, src, step, wave, kt % S, kt + S);
    f6_load<T>(lds, ((kt + 1) % S) * T::STAGE_BYTES, 0, wm, wn, r, h, ra[0], rb[0]);
    f6_mma<T, PRE, NB>(ra[last], rb[last], acc);
    f6_hint<NB - PRE, NRD, ISSUE ? T::DPW : 0>();
    __builtin_amdgcn_sched_barrier(0);
}

// Ap/Aq, Bp/Bq: converted operands (s4_to_e3m2), Ma / Nb their padded row
// counts; KT = padded K / (32 J) slices.
template <class T>
__global__ __launch_bounds__(T::NTHREADS, 1) void f6_gemm(const uint8_t *__restrict__ Ap,
                                                         const uint8_t *__restrict__ Aq,
                                                         const uint8_t *__restrict__ Bp,
                                                         const uint8_t *__restrict__ Bq,
                                                         int32_t *__restrict__ C, int M, int N,
                                                         int Ma, int Nb, int KT, int tiles_m,
                                                         int tiles_n, EpiParams epi) {
    constexpr int S = T::STAGES;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[T::LDS_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 31, h = lane >> 5;
    const int wm = wave / T::WGN, wn = wave % T::WGN;
    int tm, tn;
    tile_coords(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, T::GROUP_M, tm, tn);

    const uint8_t *src[T::DPW];
    long step[T::DPW];
#pragma unroll
    for (int u = 0; u < T::DPW; ++u)
        src[u] = f6_unit_src<T>(Ap, Aq, Bp, Bq, Ma, Nb, tm, tn, wave * T::DPW + u, lane, step[u]);

    f32x16 acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j) acc[i][j] = f32x16{};

#pragma unroll
    for (int s = 0; s < S; ++s)
        if (s < KT) f6_issue<T>(lds, src, step, wave, s, s);
    if (KT >= S) wait_vm_barrier<(S - 1) * T::DPW>();
    else wait_vm_barrier<0>();

    F6Frag ra[2][T::FM], rb[2][T::FN];
    f6_load<T>(lds, 0, 0, wm, wn, r, h, ra[0], rb[0]);

    int kt = 0;
    for (; kt + S < KT; ++kt) f6_slice<T, true>(lds, src, step, wave, kt, wm, wn, r, h, ra, rb, acc);
    for (; kt < KT; ++kt) f6_slice<T, false>(lds, src, step, wave, kt, wm, wn, r, h, ra, rb, acc);

    const long row0 = (long)tm * T::BM + wm * T::WTM;
    const long col0 = (long)tn * T::BN + wn * T::WTN + r;
    // the sums are integers of magnitude <= 2^24: the conversion is exact
    epi_store_tile<S4, 32, T::FM, T::FN, 16>(epi, C, acc, row0, col0, h, M, N, ConvToInt());
}

}  // namespace mpg
