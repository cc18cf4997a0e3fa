/*
 * oracle.c - CPU oracle for the dense product C = A * B in three precisions.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark load this file's library. The GPU library
 * neither links nor calls it, and it shares no code, header or table with the
 * GPU library.
 *
 * What it computes. The paper's primitive is a matrix multiply-accumulate
 * D = A*B + C (Background, "Tensor Cores, WMMA, and PTX mma.sync"); a GEMM
 * starts from C = 0, so every entry is the plain definition
 *
 *     C[i][j] = sum_{k=0}^{K-1} A(i,k) * B(k,j)
 *
 * with A row-major M x K (A(i,k) at i*K + k) and B column-major K x N
 * (B(k,j) at j*K + k), the ".row.col" operand order of the paper's INT4 MMA
 * (Listing "lst:int4-primitives", part (c)). C is M x N row-major.
 *
 *   FP16 -> FP32 (paper Table VI: FP16 inputs, f32 accumulators). Each binary16
 *   value is decoded exactly to binary64 by oracle_half_to_double; every product
 *   of two binary16 values is exact in binary64 (11 x 11 significand bits), and
 *   the products are summed in k order in binary64. The oracle also returns
 *   D[i][j] = sum_k |A(i,k)| * |B(k,j)|, the scale against which a GPU FP32
 *   result is judged.
 *
 *   INT8 -> INT32 (paper Run 2; signed operands). Exact int64 sums.
 *
 *   INT4 -> INT32 (paper Run 3; the ".s4.s4.s32" MMA: signed 4-bit operands,
 *   32-bit integer accumulation, no dequantisation or scaling - Scope and
 *   Generality). Two values per byte along K, low nibble = even k, two's
 *   complement; decoded by oracle_s4_value. Exact int64 sums.
 *
 * Integer results are returned as int64 so the caller can check they fit the
 * INT32 output of the GPU path.
 *
 * Work split: static slices of the output rows over nthreads POSIX threads. A
 * row subset (rows != NULL) computes only the listed rows, in list order.
 * Within an element the k order is always 0..K-1, so the result does not
 * depend on the thread count.
 *
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off (no FMA contraction, no
 * reassociation).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OK = 0, E_ARG = 1, E_NONFINITE = 2, E_NOMEM = 3, E_THREAD = 4 };

/* IEEE 754 binary16 -> binary64, from the format: 1 sign bit, 5 exponent bits
 * with bias 15, 10 fraction bits. Exponent 0: subnormal f * 2^-24 (or zero);
 * exponent 31: infinity (f == 0) or NaN; otherwise (1024 + f) * 2^(e - 25). */
double oracle_half_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1F;
    int f = h & 0x3FF;
    double mag;
    if (e == 0)
        mag = ldexp((double)f, -24);
    else if (e == 31)
        mag = f ? NAN : INFINITY;
    else
        mag = ldexp((double)(1024 + f), e - 25);
    return sign ? -mag : mag;
}

/* Signed 4-bit value number k of a packed row: byte k/2, low nibble for even
 * k, high nibble for odd k; a nibble n >= 8 stands for n - 16. */
int oracle_s4_value(const uint8_t *row, long k)
{
    unsigned byte = row[k / 2];
    unsigned nib = (k % 2 == 0) ? (byte & 0x0Fu) : (byte >> 4);
    return nib >= 8 ? (int)nib - 16 : (int)nib;
}

typedef struct {
    int dtype; /* 0 f16, 1 s8, 2 s4 */
    long M, N, K;
    const void *A, *B;
    const double *Bd; /* f16: B decoded to binary64, N x K */
    const int8_t *Bi; /* s4: B decoded to int8, N x K */
    void *C;          /* double (f16) or int64 (s8, s4) */
    double *D;        /* f16 only: sum of |a||b| */
    const int32_t *rows;
    long r0, r1;      /* this thread's slice of output rows */
    int status;
} job_t;

static void *run_job(void *p)
{
    job_t *jb = (job_t *)p;
    const long N = jb->N, K = jb->K;
    double *ad = NULL;
    int8_t *ai = NULL;
    if (jb->dtype == 0) {
        ad = (double *)malloc(sizeof(double) * (size_t)(K ? K : 1));
        if (!ad) { jb->status = E_NOMEM; return NULL; }
    } else if (jb->dtype == 2) {
        ai = (int8_t *)malloc((size_t)(K ? K : 1));
        if (!ai) { jb->status = E_NOMEM; return NULL; }
    }
    for (long r = jb->r0; r < jb->r1; ++r) {
        long i = jb->rows ? (long)jb->rows[r] : r;
        if (jb->dtype == 0) {
            const uint16_t *arow = (const uint16_t *)jb->A + i * K;
            for (long k = 0; k < K; ++k) {
                ad[k] = oracle_half_to_double(arow[k]);
                if (!isfinite(ad[k])) { jb->status = E_NONFINITE; goto done; }
            }
            double *crow = (double *)jb->C + r * N;
            double *drow = jb->D + r * N;
            for (long j = 0; j < N; ++j) {
                const double *bcol = jb->Bd + j * K;
                double acc = 0.0, den = 0.0;
                for (long k = 0; k < K; ++k) {
                    acc += ad[k] * bcol[k];
                    den += fabs(ad[k]) * fabs(bcol[k]);
                }
                crow[j] = acc;
                drow[j] = den;
            }
        } else if (jb->dtype == 1) {
            const int8_t *arow = (const int8_t *)jb->A + i * K;
            int64_t *crow = (int64_t *)jb->C + r * N;
            for (long j = 0; j < N; ++j) {
                const int8_t *bcol = (const int8_t *)jb->B + j * K;
                int64_t acc = 0;
                for (long k = 0; k < K; ++k)
                    acc += (int64_t)arow[k] * (int64_t)bcol[k];
                crow[j] = acc;
            }
        } else {
            const uint8_t *arow = (const uint8_t *)jb->A + i * (K / 2);
            for (long k = 0; k < K; ++k)
                ai[k] = (int8_t)oracle_s4_value(arow, k);
            int64_t *crow = (int64_t *)jb->C + r * N;
            for (long j = 0; j < N; ++j) {
                const int8_t *bcol = jb->Bi + j * K;
                int64_t acc = 0;
                for (long k = 0; k < K; ++k)
                    acc += (int64_t)ai[k] * (int64_t)bcol[k];
                crow[j] = acc;
            }
        }
    }
done:
    free(ad);
    free(ai);
    return NULL;
}

typedef struct {
    long lo, hi;
    const uint16_t *src;
    double *dst;
    const uint8_t *src4;
    int8_t *dst4;
    long K;
    int bad;
} decode_t;

static void *run_decode(void *p)
{
    decode_t *d = (decode_t *)p;
    if (d->src) {
        for (long x = d->lo; x < d->hi; ++x) {
            d->dst[x] = oracle_half_to_double(d->src[x]);
            if (!isfinite(d->dst[x])) d->bad = 1;
        }
    } else {
        for (long j = d->lo; j < d->hi; ++j)
            for (long k = 0; k < d->K; ++k)
                d->dst4[j * d->K + k] = (int8_t)oracle_s4_value(d->src4 + j * (d->K / 2), k);
    }
    return NULL;
}

/* Decode all of B once (binary16 -> binary64, or nibbles -> int8), in parallel. */
static int decode_b(int dtype, long N, long K, const void *B, double *Bd, int8_t *Bi, int nthreads)
{
    pthread_t th[256];
    decode_t dj[256];
    long total = (dtype == 0) ? N * K : N;
    int T = nthreads;
    if (T > total) T = (int)(total > 0 ? total : 1);
    for (int t = 0; t < T; ++t) {
        dj[t].lo = total * t / T;
        dj[t].hi = total * (t + 1) / T;
        dj[t].src = dtype == 0 ? (const uint16_t *)B : NULL;
        dj[t].dst = Bd;
        dj[t].src4 = dtype == 2 ? (const uint8_t *)B : NULL;
        dj[t].dst4 = Bi;
        dj[t].K = K;
        dj[t].bad = 0;
    }
    int started = 0, st = OK;
    for (int t = 0; t < T; ++t) {
        if (pthread_create(&th[t], NULL, run_decode, &dj[t]) != 0) { st = E_THREAD; break; }
        ++started;
    }
    for (int t = 0; t < started; ++t) pthread_join(th[t], NULL);
    for (int t = 0; t < started; ++t)
        if (dj[t].bad) st = E_NONFINITE;
    return st;
}

static int run(int dtype, long M, long N, long K, const void *A, const void *B, void *C, double *D,
               const int32_t *rows, long nrows, int nthreads)
{
    if (M < 0 || N < 0 || K < 0 || nthreads < 1 || nthreads > 256) return E_ARG;
    if (dtype == 2 && K % 2) return E_ARG;
    long R = rows ? nrows : M;
    if (R < 0) return E_ARG;
    if (rows)
        for (long r = 0; r < R; ++r)
            if (rows[r] < 0 || rows[r] >= M) return E_ARG;
    if (R == 0 || N == 0) return OK;
    if (!A || !B || !C || (dtype == 0 && !D)) return E_ARG;

    double *Bd = NULL;
    int8_t *Bi = NULL;
    int st = OK;
    if (dtype == 0) {
        Bd = (double *)malloc(sizeof(double) * (size_t)(N * K > 0 ? N * K : 1));
        if (!Bd) return E_NOMEM;
        st = decode_b(0, N, K, B, Bd, NULL, nthreads);
    } else if (dtype == 2) {
        Bi = (int8_t *)malloc((size_t)(N * K > 0 ? N * K : 1));
        if (!Bi) return E_NOMEM;
        st = decode_b(2, N, K, B, NULL, Bi, nthreads);
    }
    if (st != OK) { free(Bd); free(Bi); return st; }

    int T = nthreads;
    if (T > R) T = (int)R;
    pthread_t th[256];
    job_t jobs[256];
    for (int t = 0; t < T; ++t) {
        job_t *jb = &jobs[t];
        jb->dtype = dtype; jb->M = M; jb->N = N; jb->K = K;
        jb->A = A; jb->B = B; jb->Bd = Bd; jb->Bi = Bi; jb->C = C; jb->D = D;
        jb->rows = rows;
        jb->r0 = R * t / T;
        jb->r1 = R * (t + 1) / T;
        jb->status = OK;
    }
    int started = 0;
    for (int t = 0; t < T; ++t) {
        if (pthread_create(&th[t], NULL, run_job, &jobs[t]) != 0) { st = E_THREAD; break; }
        ++started;
    }
    for (int t = 0; t < started; ++t) pthread_join(th[t], NULL);
    for (int t = 0; t < started; ++t)
        if (jobs[t].status != OK) st = jobs[t].status;
    free(Bd);
    free(Bi);
    return st;
}

/* C (double, R x N) and D (double, R x N) for binary16 A (M x K) and B (K x N
 * column-major). R = nrows when rows != NULL, else M. Returns 0 on success,
 * 2 if an input is infinite or NaN. */
int oracle_gemm_f16(long M, long N, long K, const uint16_t *A, const uint16_t *B,
                    double *C, double *D, const int32_t *rows, long nrows, int nthreads)
{
    return run(0, M, N, K, A, B, C, D, rows, nrows, nthreads);
}

/* C (int64, R x N) for int8 A (M x K) and B (K x N column-major). */
int oracle_gemm_s8(long M, long N, long K, const int8_t *A, const int8_t *B,
                   int64_t *C, const int32_t *rows, long nrows, int nthreads)
{
    return run(1, M, N, K, A, B, C, NULL, rows, nrows, nthreads);
}

/* C (int64, R x N) for packed signed 4-bit A (M x K/2 bytes) and B (N x K/2
 * bytes); K must be even. */
int oracle_gemm_s4(long M, long N, long K, const uint8_t *A, const uint8_t *B,
                   int64_t *C, const int32_t *rows, long nrows, int nthreads)
{
    return run(2, M, N, K, A, B, C, NULL, rows, nrows, nthreads);
}
