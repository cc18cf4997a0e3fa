/*
 * mpgemm.h - dense C = A * B on one AMD Instinct MI355X (gfx950) in three
 * precisions, on the matrix cores (MFMA).
 *
 * Operation (all three entry points). The paper's primitive is the matrix
 * multiply-accumulate D = A*B + C (Background, "Tensor Cores, WMMA, and PTX
 * mma.sync"); a GEMM starts from zero, so each call computes
 *
 *     C[i][j] = sum_{k=0}^{K-1} A(i,k) * B(k,j),   0 <= i < M, 0 <= j < N,
 *
 * and OVERWRITES C (no alpha/beta, no accumulation into C's old contents).
 *
 * Layouts (the ".row.col" operand order of the paper's INT4 MMA, Listing
 * "lst:int4-primitives"; the layouts of the paper's tiles in Listings
 * "lst:int4-double-buffer" and "lst:int4-three-stage"): dense, no leading
 * dimensions.
 *   A  row-major M x K:     A(i,k) at element i*K + k.
 *   B  column-major K x N:  B(k,j) at element j*K + k (N rows of K).
 *   C  row-major M x N:     C[i][j] at element i*N + j.
 *
 * Memory and ownership. A, B and C are DEVICE pointers on the current HIP
 * device, owned by the caller; the library never allocates, frees, copies or
 * synchronises, keeps no pointer after the call returns and holds no state
 * between calls. C must not overlap A or B. Any alignment is accepted;
 * operands whose shapes and alignment suit a tuned tile take the fast
 * kernels, everything else a bounds-checked kernel.
 * Scratch memory: the plain entry points (gemm_f16_f32, gemm_s8_s32,
 * gemm_s4_s32, gemm_scaled) use none; they only choose kernels that need no
 * scratch. Split K, the INT4 kernels fed by an FP6 conversion pre-pass and
 * zero points take scratch from a caller-owned workspace passed to
 * mpgemm_gemm_ws / mpgemm_run_variant_ws (see "workspace" below).
 *
 * Streams. Work is enqueued on `stream` (0 = the null stream), which must
 * belong to the current device, and the call returns without synchronising.
 * Calls on different streams may run concurrently. Faults inside a kernel
 * surface at the caller's next synchronisation of the stream, not in the
 * return value.
 *
 * Errors. Each entry point returns hipSuccess or:
 *   hipErrorInvalidValue  M, N or K negative; K odd for INT4; a required
 *                         pointer NULL (A and B when M, N, K > 0; C when
 *                         M, N > 0); C overlapping A or B; a problem whose
 *                         element counts overflow 64-bit byte offsets;
 *   the launch error      if a kernel launch itself fails.
 * Nothing is enqueued when an argument error is returned.
 * Degenerate sizes: M == 0 or N == 0 is a no-op returning hipSuccess; K == 0
 * writes zeros to C (empty sums).
 */
#ifndef MPGEMM_H
#define MPGEMM_H

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* FP16 inputs, FP32 accumulation and output (paper Run 1; Table VI lists the
 * f32-accumulator FP16 kernels). A and B hold IEEE binary16 values (finite or
 * not: the hardware's IEEE arithmetic decides inf/NaN propagation); C receives
 * binary32. Products are summed in FP32 in an unspecified order, so results
 * are not bit-unique; the library's tests bound them by
 * |C - exact| <= 1e-3 * sum_k |A(i,k)| |B(k,j)|. */
hipError_t gemm_f16_f32(int M, int N, int K, const void *A, const void *B, float *C,
                        hipStream_t stream);

/* Signed INT8 inputs, INT32 accumulation and output (paper Run 2). Exact: C
 * equals the integer sum whenever every partial sum fits in int32, which
 * always holds for K < 131072 (|a*b| <= 2^14); results beyond that range are
 * not specified. */
hipError_t gemm_s8_s32(int M, int N, int K, const int8_t *A, const int8_t *B, int32_t *C,
                       hipStream_t stream);

/* Signed INT4 inputs, INT32 accumulation and output (paper Run 3: the
 * ".s4.s4.s32" MMA, no dequantisation or scaling). K must be even. Values are
 * two's-complement nibbles packed two per byte along K, the low nibble holding
 * the even k: A is M rows of K/2 bytes, B is N rows of K/2 bytes. Exact
 * whenever every partial sum fits in int32, which always holds for K < 2^25
 * (|a*b| <= 64). gfx950 has no 4-bit integer MFMA: for K a multiple of 256
 * up to 65536 the kernel feeds each value v as the FP6 E2M3 code v + 8
 * (value (v + 8) / 8, exact) to the FP6 MFMA, converting inside the GEMM,
 * and removes the bias with row and column sums it takes on the way; every
 * FP32 partial sum is then a multiple of 1/64 below 2^18, held exactly.
 * Other problems run on the INT8 MFMA (K < 131072) or the bounds-checked
 * kernel. */
hipError_t gemm_s4_s32(int M, int N, int K, const uint8_t *A, const uint8_t *B, int32_t *C,
                       hipStream_t stream);

/* ---- scaled outputs: the dequantisation step after the GEMM, fused ----
 * The paper's kernels return the raw INT32 sums, without dequantisation or
 * scaling (Scope and Generality); the next step of an inference pipeline
 * multiplies them by per-row and per-column scales, optionally removing
 * zero points first, and narrows the result. gemm_scaled does that in the
 * GEMM's own epilogue:
 *
 *   C[i][j] = round( sa[i] * sb[j] * sum_k (A(i,k) - za[i]) * (B(k,j) - zb[j]) )
 *
 * with absent scales = 1 and absent zero points = 0. Integer inputs: the sum
 * is exact (the zero-point terms are evaluated in 64-bit integers from row
 * sums of A and column sums of B), converted to binary32 once, multiplied by
 * sa[i] then sb[j] in binary32, and rounded to nearest even into the output
 * type; so the result is within 1 unit in the last place of the output type
 * of the exact value (binary32 output: within 3 ulp). FP16 inputs:
 * the binary32 sum of the plain entry point (same error bound), scaled the
 * same way; zero points are not accepted. The struct is a HOST pointer read
 * during the call; the vectors it points to are DEVICE arrays of M (for _a)
 * or N (for _b) elements, 4-byte aligned. C holds M x N elements of the
 * output type, row-major (2-byte aligned for FP16/BF16, 4-byte for FP32).
 * Zero points cost one extra pass over A and/or B (row sums, kept in a
 * workspace): gemm_scaled takes no workspace and refuses zero points; pass
 * them to mpgemm_gemm_ws. Errors as for the plain entry points, plus
 * hipErrorInvalidValue for a NULL struct, an unknown output type, zero
 * points (here) or zero points with FP16 inputs (everywhere), misaligned
 * vectors. */
enum { MPGEMM_OUT_F32 = 1, MPGEMM_OUT_F16 = 2, MPGEMM_OUT_BF16 = 3 };

typedef struct mpgemm_epilogue {
    const float *scale_a;  /* M per-row scales, or NULL */
    const float *scale_b;  /* N per-column scales, or NULL */
    const int32_t *zero_a; /* M per-row zero points (integer inputs), or NULL */
    const int32_t *zero_b; /* N per-column zero points (integer inputs), or NULL */
    int out_type;          /* MPGEMM_OUT_F32, MPGEMM_OUT_F16 or MPGEMM_OUT_BF16 */
} mpgemm_epilogue;

/* dtype as below (0 = FP16, 1 = INT8, 2 = INT4, same operand layouts as the
 * plain entry points); C receives the scaled output. */
hipError_t gemm_scaled(int dtype, int M, int N, int K, const void *A, const void *B, void *C,
                       const mpgemm_epilogue *epi, hipStream_t stream);

/* ---- workspace: scratch memory owned by the caller ----
 * Some kernels need device scratch memory besides A, B and C: split K (the
 * partial tiles of the K ranges and one counter per tile; the automatic
 * choice splits only skinny problems, see mpgemm_select_splits), the INT4
 * kernels fed by an FP6 conversion pre-pass (the converted operands, 0.75
 * byte per padded element) and zero points (row sums of A and column sums
 * of B). The library never allocates it: the caller passes a workspace.
 *
 * mpgemm_workspace_size: bytes of workspace the call with the same arguments
 * would use, into *bytes (0: none). variant < 0 and splits == 0 ask for the
 * automatic choice made with a large enough workspace; epi may be NULL.
 * Returns hipErrorInvalidValue for arguments the call would refuse (sizes,
 * epilogue, a variant that cannot run the problem, a bad split count).
 *
 * mpgemm_gemm_ws: the operation of the dtype's entry point (dtype 0 = FP16
 * -> FP32, 1 = INT8 -> INT32, 2 = INT4 -> INT32), with scaled outputs when
 * epi is not NULL (as gemm_scaled, zero points allowed), using `workspace`
 * (DEVICE memory on the current device, 256-byte aligned, not overlapping A,
 * B or C, `workspace_bytes` long) for scratch. With workspace == NULL or
 * workspace_bytes == 0 it is the plain entry point (or gemm_scaled); a
 * workspace smaller than the automatic choice wants makes it choose a kernel
 * that needs less (no split), except that zero points always need theirs.
 * Contract:
 *   - zero-fill the workspace once before its first use (hipMemset after
 *     allocating it); every completed call leaves the counter block (the
 *     first 64 KiB) zero again, so later calls need no clearing;
 *   - one call at a time per workspace: calls that may run concurrently
 *     (other streams, other threads) need workspaces of their own; calls in
 *     order on one stream may share one;
 *   - the library keeps no pointer to it after the call returns; free it
 *     once the stream's pending work that uses it has completed.
 * Errors: those of the entry points, plus hipErrorInvalidValue for a
 * misaligned or overlapping workspace, or one too small for the scratch the
 * call cannot do without (zero points; an explicit split or FP6 pre-pass
 * variant in mpgemm_run_variant_ws). Nothing is enqueued then. */
hipError_t mpgemm_workspace_size(int dtype, int variant, int splits, int M, int N, int K,
                                 const mpgemm_epilogue *epi, size_t *bytes);

hipError_t mpgemm_gemm_ws(int dtype, int M, int N, int K, const void *A, const void *B, void *C,
                          const mpgemm_epilogue *epi, void *workspace, size_t workspace_bytes,
                          hipStream_t stream);

/* For callers that cannot allocate (code under graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): mpgemm_gemm_ws with the scratch
 * taken from a 32 MiB array the library holds on each device it runs on
 * (allocated with the code object, kept until the process ends) instead of
 * a caller workspace. Allocates and frees nothing. The first call on a
 * device looks up that device's array address (hipGetSymbolAddress). The
 * automatic choice is the one mpgemm_gemm_ws makes with a 32 MiB workspace: a
 * split or stream-K schedule (or the INT4 pre-pass) that would need more is
 * not taken; zero points needing more (M + N above about 8.4 million) return
 * hipErrorInvalidValue. A split or stream-K call first clears the tile
 * counters with a small kernel on `stream`. Every
 * call on a device shares that device's array: calls that may overlap on
 * one device (other streams, other threads) race, and must be ordered by
 * the caller (one stream, or events). Other arguments, semantics and errors
 * as mpgemm_gemm_ws. */
hipError_t mpgemm_gemm_noalloc(int dtype, int M, int N, int K, const void *A, const void *B, void *C,
                               const mpgemm_epilogue *epi, hipStream_t stream);

/* B stored K x N ROW-major (B(k,j) at element k*N + j, N-contiguous): the
 * "transposed B" operand layout of the paper's INT4 ablation (Table XII),
 * which cost its kernels 3x through uncoalesced loads. Here B is copied to
 * LDS as stored and turned into MFMA operands by the LDS transpose reads of
 * gfx950. dtype 0 (FP16 -> FP32 C), 1 (INT8 -> INT32 C) or 2 (INT4 -> INT32
 * C; B's nibbles packed two per byte along N, the low nibble holding the even
 * column: B(k,j) in byte k*N/2 + j/2); A row-major M x K and C row-major
 * M x N as for the plain entry points; same semantics, ownership, stream and
 * tolerance rules.
 * Requirements (else hipErrorInvalidValue, nothing enqueued): N a multiple
 * of 256; K a multiple of 64 (FP16), 128 (INT8) or 256 (INT4, and below
 * 131072), or K == 0 (C zero-filled); A and B 16-byte aligned, C 4-byte
 * aligned; the checks of the plain entry points (sizes, NULL pointers,
 * overlap). M may be any size. No workspace. */
hipError_t mpgemm_gemm_bt(int dtype, int M, int N, int K, const void *A, const void *B, void *C,
                          hipStream_t stream);

/* ---- introspection and tuning (same operation, explicit kernel choice) ----
 * dtype: 0 = FP16->FP32, 1 = INT8->INT32, 2 = INT4->INT32. A variant is one
 * compiled kernel configuration (tile shape, wave layout, pipeline depth).
 * Variant 0 of every dtype is the bounds-checked kernel that accepts any
 * shape and alignment. */

/* Number of variants for dtype, or -1 for an unknown dtype. */
int mpgemm_num_variants(int dtype);

/* Static, NUL-terminated name of a variant ("" if out of range). */
const char *mpgemm_variant_name(int dtype, int variant);

/* The variant the dtype's entry point runs for these arguments (pointers are
 * only inspected for alignment), or -1 if the arguments are invalid. */
int mpgemm_select_variant(int dtype, int M, int N, int K, const void *A, const void *B,
                          const void *C);

/* The variant mpgemm_gemm_ws runs for these arguments with a workspace that
 * holds that variant's scratch (INT4 then takes the FP6 kernels fed by the
 * conversion pre-pass where they are faster), or -1 for invalid arguments. */
int mpgemm_select_variant_ws(int dtype, int M, int N, int K, const void *A, const void *B,
                             const void *C);

/* Whether `variant` can run these arguments: 1 yes, 0 no, -1 invalid dtype. */
int mpgemm_variant_supports(int dtype, int variant, int M, int N, int K, const void *A,
                            const void *B, const void *C);

/* Run one specific variant with the same semantics, validation and errors as
 * the dtype's entry point; hipErrorInvalidValue also when the variant does not
 * support the arguments. C is float* for dtype 0, int32_t* otherwise. */
hipError_t mpgemm_run_variant(int dtype, int variant, int M, int N, int K, const void *A,
                              const void *B, void *C, hipStream_t stream);

/* Split-K: the pipelined variants can divide K into `splits` ranges of whole
 * K-slices, one workgroup per (tile, range); the last workgroup of a tile to
 * finish adds the ranges' partial sums in range order 0, 1, ... and writes C,
 * so results do not depend on scheduling (FP16: the summation order differs
 * from the unsplit kernel's, within the same error bound; integers: exact).
 * Partials and per-tile counters live in the caller's workspace. With a
 * workspace, the automatic choice splits only problems with a small side:
 * the narrow tiles (at most 256 rows on one side, at least 1024 on the other)
 * while the grid stays within 128 workgroups, up to 4 ranges; where those do
 * not apply, the 128x128 tiles of problems with M or N at most 128 up to 256
 * workgroups, 4 ranges for FP16, 2 for the integer types. The narrow tiles
 * with an eight-slice ring ("..._s8_m16") are never split. */

/* Splits the automatic choice uses for this variant and problem when a large
 * enough workspace is given (1 = none), or -1 for an invalid dtype, variant
 * or size. */
int mpgemm_select_splits(int dtype, int variant, int M, int N, int K);

/* Stream-K: the variants named "..._sk" (the one-wave-per-SIMD FP16/INT8
 * kernel, the 256x256 and the 128x128 pipelined kernels, and the INT4
 * one-wave-per-SIMD FP6 kernel fed by the conversion pre-pass) share the
 * last, partly filled round of a problem's tiles out over more workgroups.
 * With T tiles, G workgroups resident at once (one per CU: 256 on MI355X)
 * and T = q G + r, 0 < r <= G / 2: workgroups 0 .. q G - 1 compute one whole
 * tile each; the K-slices (KT per tile: 128 bytes of K each, or 128 k of K
 * padded to 256 for the FP6 kernel) of each of the r remaining tiles are
 * then cut into s contiguous parts, one workgroup each, s =
 * round(sqrt(KT t / 5)) capped at G / r, 8 and KT / 2, where t is the time
 * of a slice in microseconds (1; 0.5 for the FP6 kernel). The last of a
 * tile's parts to finish adds the s partial tiles in part order and writes
 * C, so results do not depend on scheduling (FP16: the order of summation
 * differs from the whole-tile kernel's, within the same error bound;
 * integers: exact, the FP6 kernel's FP32 part sums included, whose
 * magnitudes add up to at most 64 K < 2^24).
 * Scratch, in the workspace: the 64 KiB counter block (one counter per
 * tile, left zero by every call), then (after the FP6 kernel's converted
 * operands) r * s partial tiles of 4 x BM x BN bytes. Every tile is computed
 * whole without a large enough workspace, when T is a multiple of G,
 * r > G / 2, T is beyond 16384 tiles, s < 2, or the expected gain,
 * KT t (1 - 1/s) - 5 (s - 1) - 13 microseconds, is at most KT t / 10 (a
 * quarter of KT t for the FP6 kernel). With a workspace the automatic
 * choice takes a stream-K variant in place of its whole-tile kernel where
 * its schedule is on and its scratch fits, else the whole-tile kernel.
 * mpgemm_sk_schedule: the schedule a stream-K variant would use for this
 * problem on the current device (G = 256 when no device is visible):
 * *dp_tiles whole tiles first, then *parts parts per remaining tile (1:
 * stream-K off), *grid workgroups in all. hipErrorInvalidValue for an
 * invalid dtype or variant, null outputs, or a problem the variant cannot
 * run; for a variant without a stream-K schedule it reports every tile
 * whole. Host only: enqueues nothing. */
hipError_t mpgemm_sk_schedule(int dtype, int variant, int M, int N, int K, int *dp_tiles, int *parts,
                              int *grid);

/* One specific variant with an explicit split count (0 = the automatic
 * choice for the variant), scaled outputs when epi is not NULL, and a
 * workspace as for mpgemm_gemm_ws. hipErrorInvalidValue also when the
 * variant cannot run the problem, splits > 1 for a variant that cannot
 * split, splits > 16, K's slices not dividing evenly into `splits`, or the
 * workspace too small for the split or the FP6 pre-pass the variant needs. */
hipError_t mpgemm_run_variant_ws(int dtype, int variant, int splits, int M, int N, int K, const void *A,
                                 const void *B, void *C, const mpgemm_epilogue *epi, void *workspace,
                                 size_t workspace_bytes, hipStream_t stream);

/* Host-side view of the INT4 -> FP6 conversion the FP6 kernels apply on the
 * device (same source): `in` is one run of 16 HOST bytes = 32 nibbles, word
 * d = bytes 4d..4d+3 (little-endian); `out` (6 words, HOST) receives a
 * 192-bit little-endian string of 32 six-bit E3M2 codes, field f at bits
 * [6f, 6f+6). Field 8d + 4h + i holds the code of the nibble in byte i of
 * word d, low nibble for h = 0, high nibble for h = 1 (i.e. k offset
 * 8d + 2i + h). For tests of the encoding; never touches the GPU. */
void mpgemm_s4_run_to_fp6(const uint8_t *in, uint32_t *out);

/* Host-side view of the conversion the INT4 kernel with the conversion
 * inside the GEMM applies on the device (same source): `in` is one run of 16
 * HOST bytes = 32 nibbles (word d = bytes 4d..4d+3, little-endian); `out` (6
 * words, HOST) receives 32 six-bit FP6 E2M3 codes, field f at bits
 * [6f, 6f+6) of the 192-bit little-endian string. The code of a nibble v is
 * v + 8 (the nibble with its top bit flipped), value (v + 8) / 8. Input
 * words (x, y) = (word 2p, word 2p + 1) fill fields 16p .. 16p + 15 with
 * their nibbles (nibble n of a word at bits 4n..4n+3) in the order
 * x0 y1 x3 y4 x6 y7 x1 y2 x4 y5 x7 y0 x2 y3 x5 y6. For tests of the
 * encoding; never touches the GPU. */
void mpgemm_s4_run_to_e2m3(const uint8_t *in, uint32_t *out);

#ifdef __cplusplus
}
#endif

#endif /* MPGEMM_H */
