/* Drives the CPU oracle under a sanitizer build (AddressSanitizer +
 * UndefinedBehaviorSanitizer, or ThreadSanitizer): every dtype, full and
 * row-subset runs, several thread counts, ragged and degenerate shapes.
 * Checks that the threaded results equal the single-threaded ones and, on
 * small shapes, a naive sum written here; any sanitizer report or mismatch
 * makes the process fail. Inputs come from a local linear congruential
 * generator (values only; nothing of the oracle's arithmetic is shared). */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_gemm_f16(long M, long N, long K, const uint16_t *A, const uint16_t *B, double *C, double *D,
                    const int32_t *rows, long nrows, int nthreads);
int oracle_gemm_s8(long M, long N, long K, const int8_t *A, const int8_t *B, int64_t *C, const int32_t *rows,
                   long nrows, int nthreads);
int oracle_gemm_s4(long M, long N, long K, const uint8_t *A, const uint8_t *B, int64_t *C, const int32_t *rows,
                   long nrows, int nthreads);

static uint64_t state = 12345;
static uint32_t next(void) {
    state = state * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)(state >> 33);
}

/* a finite binary16 pattern of small magnitude: exponent 10..17 */
static uint16_t half_bits(void) {
    uint32_t r = next();
    return (uint16_t)(((r & 1) << 15) | ((10 + (r >> 1) % 8) << 10) | ((r >> 4) & 0x3FF));
}

static int fail(const char *what, long M, long N, long K) {
    fprintf(stderr, "FAIL %s %ldx%ldx%ld\n", what, M, N, K);
    return 1;
}

static int check_shape(long M, long N, long K) {
    const long kb = (K + 1) / 2;
    uint16_t *Ah = malloc(sizeof(uint16_t) * (M * K + 1)), *Bh = malloc(sizeof(uint16_t) * (N * K + 1));
    int8_t *A8 = malloc(M * K + 1), *B8 = malloc(N * K + 1);
    uint8_t *A4 = malloc(M * kb + 1), *B4 = malloc(N * kb + 1);
    for (long i = 0; i < M * K; ++i) { Ah[i] = half_bits(); A8[i] = (int8_t)next(); }
    for (long i = 0; i < N * K; ++i) { Bh[i] = half_bits(); B8[i] = (int8_t)next(); }
    for (long i = 0; i < M * kb; ++i) A4[i] = (uint8_t)next();
    for (long i = 0; i < N * kb; ++i) B4[i] = (uint8_t)next();
    double *C1 = malloc(sizeof(double) * (M * N + 1)), *D1 = malloc(sizeof(double) * (M * N + 1));
    double *C2 = malloc(sizeof(double) * (M * N + 1)), *D2 = malloc(sizeof(double) * (M * N + 1));
    int64_t *I1 = malloc(sizeof(int64_t) * (M * N + 1)), *I2 = malloc(sizeof(int64_t) * (M * N + 1));
    int32_t *rows = malloc(sizeof(int32_t) * (M + 1));
    long nr = 0;
    for (long i = M - 1; i >= 0; i -= 2) rows[nr++] = (int32_t)i;  /* every other row, reversed */
    int bad = 0;
    if (oracle_gemm_f16(M, N, K, Ah, Bh, C1, D1, NULL, M, 1) || oracle_gemm_f16(M, N, K, Ah, Bh, C2, D2, NULL, M, 5))
        bad |= fail("f16 call", M, N, K);
    if (memcmp(C1, C2, sizeof(double) * M * N) || memcmp(D1, D2, sizeof(double) * M * N))
        bad |= fail("f16 threads", M, N, K);
    if (oracle_gemm_f16(M, N, K, Ah, Bh, C2, D2, rows, nr, 3)) bad |= fail("f16 rows call", M, N, K);
    for (long r = 0; r < nr; ++r)
        if (memcmp(C2 + r * N, C1 + (long)rows[r] * N, sizeof(double) * N)) bad |= fail("f16 rows", M, N, K);
    if (oracle_gemm_s8(M, N, K, A8, B8, I1, NULL, M, 1) || oracle_gemm_s8(M, N, K, A8, B8, I2, NULL, M, 7))
        bad |= fail("s8 call", M, N, K);
    if (memcmp(I1, I2, sizeof(int64_t) * M * N)) bad |= fail("s8 threads", M, N, K);
    if (M * N * K <= 4096)
        for (long i = 0; i < M; ++i)
            for (long j = 0; j < N; ++j) {
                int64_t s = 0;
                for (long k = 0; k < K; ++k) s += (int64_t)A8[i * K + k] * B8[j * K + k];
                if (s != I1[i * N + j]) bad |= fail("s8 naive", M, N, K);
            }
    if ((K & 1) == 0) {
        if (oracle_gemm_s4(M, N, K, A4, B4, I1, NULL, M, 1) || oracle_gemm_s4(M, N, K, A4, B4, I2, rows, nr, 4))
            bad |= fail("s4 call", M, N, K);
        for (long r = 0; r < nr; ++r)
            if (memcmp(I2 + r * N, I1 + (long)rows[r] * N, sizeof(int64_t) * N)) bad |= fail("s4 rows", M, N, K);
    }
    free(Ah); free(Bh); free(A8); free(B8); free(A4); free(B4);
    free(C1); free(D1); free(C2); free(D2); free(I1); free(I2); free(rows);
    return bad;
}

int main(void) {
    const long shapes[][3] = {{1, 1, 2}, {3, 5, 8}, {7, 3, 6}, {16, 16, 32}, {33, 17, 66}, {64, 9, 128},
                              {5, 70, 100}, {2, 2, 0}, {40, 31, 258}};
    int bad = 0;
    for (unsigned s = 0; s < sizeof(shapes) / sizeof(shapes[0]); ++s)
        bad |= check_shape(shapes[s][0], shapes[s][1], shapes[s][2]);
    /* argument errors must be reported, not crash */
    int64_t c[4];
    const int32_t badrow[1] = {9};
    int8_t a[8] = {0};
    if (oracle_gemm_s8(2, 2, 4, a, a, c, badrow, 1, 2) == 0) bad |= fail("bad row accepted", 2, 2, 4);
    if (oracle_gemm_s4(2, 2, 3, (uint8_t *)a, (uint8_t *)a, c, NULL, 2, 2) == 0) bad |= fail("odd K accepted", 2, 2, 3);
    printf(bad ? "oracle driver: FAILED\n" : "oracle driver: ok\n");
    return bad;
}
