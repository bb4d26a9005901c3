/*
 * oracle_gemm.c -- plain CPU oracle for dense GEMM, C = A . B.
 *
 * TEST INFRASTRUCTURE ONLY.  The test suite, the package smoke check and the
 * benchmark's CPU-baseline leg are the only code allowed to load this library.
 * The GPU library never links, includes or calls it, and this file includes
 * nothing from the GPU library: the two share no code.
 *
 * What is computed (paper, Sec. 4.1 "Multi-Level Tiling Method": the problem
 * is an M x K x N GEMM with A the M x K input, B the K x N input and C the
 * M x N output; Sec. 4.2.2 "Memory Tile Design": A and C are kept row-major
 * in memory, B row- or column-major -- here B is row-major):
 *
 *   C[i][j] = sum_{k=0}^{K-1} A[i][k] * B[k][j],   0 <= i < M, 0 <= j < N.
 *
 *   int8 -> int32 : every product and the running sum are exact in int64; the
 *                   sum is then checked against the int32 range.  Out-of-range
 *                   results are counted and stored wrapped modulo 2^32.
 *   bf16 -> fp64  : every bf16 operand is widened exactly (its 16 bits are the
 *                   top half of an IEEE binary32, which is exact in binary64);
 *                   a product of two bf16 values has at most 16 significand
 *                   bits, so it is exact in binary64; the products are summed
 *                   in binary64 with k ascending.
 *
 * Loop order is i-k-j: one row of accumulators per output row, then for each
 * k (ascending) the scaled row k of B is added into it.  Every C[i][j] is
 * therefore the same left-to-right sum over k as the textbook i-j-k loop, so
 * results are identical to it (build with -O2 and without -ffast-math so that
 * the floating-point additions are never reassociated).  Threads split the
 * output rows; a row is never shared between threads.
 *
 * Strides: lda, ldb, ldc are row strides in elements (row-major storage).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)
#define ORACLE_ENOMEM (-2)

/* ------------------------------------------------------------------------ */
/* bf16 widening: a bf16 value is the upper 16 bits of a binary32.          */
/* ------------------------------------------------------------------------ */
double oracle_bf16_to_double(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static int bad_args(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
                    const void *B, int64_t ldb, const void *C, int64_t ldc)
{
    if (M < 0 || N < 0 || K < 0) return 1;
    if (M > 0 && K > 0 && (A == NULL || lda < K)) return 1;
    if (K > 0 && N > 0 && (B == NULL || ldb < N)) return 1;
    if (M > 0 && N > 0 && (C == NULL || ldc < N)) return 1;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Row-block threading.                                                     */
/* ------------------------------------------------------------------------ */
enum { KIND_I8_I32, KIND_I8_I64, KIND_BF16_F64 };

typedef struct {
    int kind;
    int64_t row0, row1, N, K;
    const void *A; int64_t lda;
    const void *B; int64_t ldb;
    void *C; int64_t ldc;
    int64_t overflow;   /* int8 -> int32: results outside the int32 range */
    int status;
} job_t;

static void run_rows_int(job_t *j)
{
    const int8_t *A = (const int8_t *)j->A;
    const int8_t *B = (const int8_t *)j->B;
    int64_t *acc = (int64_t *)malloc((size_t)(j->N > 0 ? j->N : 1) * sizeof(int64_t));
    if (!acc) { j->status = ORACLE_ENOMEM; return; }
    for (int64_t i = j->row0; i < j->row1; ++i) {
        for (int64_t c = 0; c < j->N; ++c) acc[c] = 0;
        for (int64_t k = 0; k < j->K; ++k) {
            const int64_t a = (int64_t)A[i * j->lda + k];
            const int8_t *brow = B + k * j->ldb;
            for (int64_t c = 0; c < j->N; ++c) acc[c] += a * (int64_t)brow[c];
        }
        if (j->kind == KIND_I8_I64) {
            int64_t *crow = (int64_t *)j->C + i * j->ldc;
            for (int64_t c = 0; c < j->N; ++c) crow[c] = acc[c];
        } else {
            int32_t *crow = (int32_t *)j->C + i * j->ldc;
            for (int64_t c = 0; c < j->N; ++c) {
                if (acc[c] < INT32_MIN || acc[c] > INT32_MAX) j->overflow++;
                crow[c] = (int32_t)(uint32_t)(uint64_t)acc[c];   /* wrap mod 2^32 */
            }
        }
    }
    free(acc);
}

static void run_rows_bf16(job_t *j)
{
    const uint16_t *A = (const uint16_t *)j->A;
    const uint16_t *B = (const uint16_t *)j->B;
    double *acc = (double *)malloc((size_t)(j->N > 0 ? j->N : 1) * sizeof(double));
    double *brow_d = (double *)malloc((size_t)(j->N > 0 ? j->N : 1) * sizeof(double));
    if (!acc || !brow_d) { free(acc); free(brow_d); j->status = ORACLE_ENOMEM; return; }
    for (int64_t i = j->row0; i < j->row1; ++i) {
        for (int64_t c = 0; c < j->N; ++c) acc[c] = 0.0;
        for (int64_t k = 0; k < j->K; ++k) {
            const double a = oracle_bf16_to_double(A[i * j->lda + k]);
            const uint16_t *brow = B + k * j->ldb;
            for (int64_t c = 0; c < j->N; ++c) brow_d[c] = oracle_bf16_to_double(brow[c]);
            for (int64_t c = 0; c < j->N; ++c) acc[c] += a * brow_d[c];
        }
        double *crow = (double *)j->C + i * j->ldc;
        for (int64_t c = 0; c < j->N; ++c) crow[c] = acc[c];
    }
    free(acc);
    free(brow_d);
}

static void *job_main(void *p)
{
    job_t *j = (job_t *)p;
    if (j->kind == KIND_BF16_F64) run_rows_bf16(j);
    else run_rows_int(j);
    return NULL;
}

static int run_threaded(int kind, int64_t M, int64_t N, int64_t K,
                        const void *A, int64_t lda, const void *B, int64_t ldb,
                        void *C, int64_t ldc, int nthreads, int64_t *overflow)
{
    if (overflow) *overflow = 0;
    if (bad_args(M, N, K, A, lda, B, ldb, C, ldc)) return ORACLE_EINVAL;
    if (M == 0 || N == 0) return ORACLE_OK;
    if (nthreads < 1) nthreads = 1;
    if ((int64_t)nthreads > M) nthreads = (int)M;

    job_t *jobs = (job_t *)calloc((size_t)nthreads, sizeof(job_t));
    pthread_t *tids = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    if (!jobs || !tids) { free(jobs); free(tids); return ORACLE_ENOMEM; }
    for (int t = 0; t < nthreads; ++t) {
        job_t *j = &jobs[t];
        j->kind = kind;
        j->row0 = M * t / nthreads;
        j->row1 = M * (t + 1) / nthreads;
        j->N = N; j->K = K;
        j->A = A; j->lda = lda; j->B = B; j->ldb = ldb; j->C = C; j->ldc = ldc;
    }
    int started = 0;
    for (int t = 1; t < nthreads; ++t) {
        if (pthread_create(&tids[t], NULL, job_main, &jobs[t]) != 0) break;
        started = t;
    }
    job_main(&jobs[0]);
    for (int t = 1; t <= started; ++t) pthread_join(tids[t], NULL);
    /* rows of threads that could not be started are computed here */
    for (int t = started + 1; t < nthreads; ++t) job_main(&jobs[t]);

    int status = ORACLE_OK;
    int64_t ovf = 0;
    for (int t = 0; t < nthreads; ++t) {
        if (jobs[t].status != ORACLE_OK) status = jobs[t].status;
        ovf += jobs[t].overflow;
    }
    if (overflow) *overflow = ovf;
    free(jobs);
    free(tids);
    return status;
}

/* ------------------------------------------------------------------------ */
/* Public oracle entry points.                                              */
/* ------------------------------------------------------------------------ */

/* int8 x int8 -> int32.  *overflow (may be NULL) receives the number of
 * results outside [-2^31, 2^31-1]; those are stored wrapped modulo 2^32. */
int oracle_gemm_i8_i32(int64_t M, int64_t N, int64_t K,
                       const int8_t *A, int64_t lda, const int8_t *B, int64_t ldb,
                       int32_t *C, int64_t ldc, int nthreads, int64_t *overflow)
{
    return run_threaded(KIND_I8_I32, M, N, K, A, lda, B, ldb, C, ldc, nthreads, overflow);
}

/* int8 x int8 -> int64 (exact for any K below 2^49). */
int oracle_gemm_i8_i64(int64_t M, int64_t N, int64_t K,
                       const int8_t *A, int64_t lda, const int8_t *B, int64_t ldb,
                       int64_t *C, int64_t ldc, int nthreads)
{
    return run_threaded(KIND_I8_I64, M, N, K, A, lda, B, ldb, C, ldc, nthreads, NULL);
}

/* bf16 x bf16 -> binary64 (operands passed as raw bf16 bit patterns). */
int oracle_gemm_bf16_f64(int64_t M, int64_t N, int64_t K,
                         const uint16_t *A, int64_t lda, const uint16_t *B, int64_t ldb,
                         double *C, int64_t ldc, int nthreads)
{
    return run_threaded(KIND_BF16_F64, M, N, K, A, lda, B, ldb, C, ldc, nthreads, NULL);
}

/* ------------------------------------------------------------------------ */
/* Freivalds' check of a claimed int8 product (R. Freivalds, 1977).         */
/* ------------------------------------------------------------------------ */
/* SplitMix64 finaliser (G. Steele, D. Lea, C. Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014), used as a counter-based
 * generator: value n of stream `seed` is mix(seed + (n+1) * golden gamma). */
static uint64_t splitmix64_at(uint64_t seed, uint64_t n)
{
    uint64_t z = seed + (n + 1) * 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* For `trials` random vectors r with entries in [-2^16, 2^16), checks
 * A.(B.r) == C.r exactly (128-bit integer arithmetic, nothing wrapped), so a
 * product that does not fit in int32 never passes.  A wrong C passes one
 * trial with probability at most 1/2^17 per row.  Returns the number of
 * (trial, row) pairs that disagree (0 means every trial is consistent), or a
 * negative error code. */
int64_t oracle_freivalds_i8_i32(int64_t M, int64_t N, int64_t K,
                                const int8_t *A, int64_t lda, const int8_t *B, int64_t ldb,
                                const int32_t *C, int64_t ldc, int trials, uint64_t seed)
{
    if (bad_args(M, N, K, A, lda, B, ldb, C, ldc) || trials < 0) return ORACLE_EINVAL;
    if (M == 0 || N == 0) return 0;
    __int128 *r = (__int128 *)malloc((size_t)N * sizeof(__int128));
    __int128 *br = (__int128 *)malloc((size_t)(K > 0 ? K : 1) * sizeof(__int128));
    if (!r || !br) { free(r); free(br); return ORACLE_ENOMEM; }
    int64_t bad = 0;
    for (int t = 0; t < trials; ++t) {
        for (int64_t c = 0; c < N; ++c)
            r[c] = (__int128)((int64_t)(splitmix64_at(seed + (uint64_t)t, (uint64_t)c) >> 47) - 65536);
        for (int64_t k = 0; k < K; ++k) {
            __int128 s = 0;
            const int8_t *brow = B + k * ldb;
            for (int64_t c = 0; c < N; ++c) s += (__int128)brow[c] * r[c];
            br[k] = s;
        }
        for (int64_t i = 0; i < M; ++i) {
            __int128 lhs = 0, rhs = 0;
            const int8_t *arow = A + i * lda;
            for (int64_t k = 0; k < K; ++k) lhs += (__int128)arow[k] * br[k];
            const int32_t *crow = C + i * ldc;
            for (int64_t c = 0; c < N; ++c) rhs += (__int128)crow[c] * r[c];
            if (lhs != rhs) bad++;
        }
    }
    free(r);
    free(br);
    return bad;
}

/* ------------------------------------------------------------------------ */
/* Reduced-precision outputs.  The paper also reports int8 GEMMs with int16  */
/* and int8 outputs ("precision-reduced") and bf16 GEMMs with bf16 outputs  */
/* (Sec. 5.1, Sec. 5.2.3) but states no rounding or requantisation rule.    */
/* The reading implemented here, applied elementwise to the exact results   */
/* of the routines above:                                                   */
/*                                                                          */
/*   int32 -> int8 / int16 : q = v / 2^shift rounded to the nearest integer, */
/*                            ties to even, then clamped to the output range; */
/*   fp64  -> bf16         : the nearest bf16 value, ties to even (8          */
/*                            significant bits, subnormal spacing 2^-133,     */
/*                            values beyond the largest finite bf16 after      */
/*                            rounding become infinities).                     */
/* ------------------------------------------------------------------------ */

/* Nearest integer to v / 2^shift, ties to even, computed exactly in int64. */
static int64_t div_pow2_nearest_even(int64_t v, int shift)
{
    const int64_t d = (int64_t)1 << shift;
    int64_t q = v / d;                       /* truncates toward zero */
    if (v % d != 0 && v < 0) q -= 1;         /* floor */
    const int64_t r = v - q * d;             /* 0 <= r < d */
    if (shift > 0) {
        const int64_t half = d / 2;
        if (r > half || (r == half && q % 2 != 0)) q += 1;
    }
    return q;
}

int oracle_requant_i32(const int32_t *in, int64_t n, int shift, int bits, int32_t *out)
{
    if (n < 0 || (n > 0 && (in == NULL || out == NULL)) || shift < 0 || shift > 31 ||
        (bits != 8 && bits != 16))
        return ORACLE_EINVAL;
    const int64_t hi = ((int64_t)1 << (bits - 1)) - 1, lo = -hi - 1;
    for (int64_t i = 0; i < n; ++i) {
        int64_t q = div_pow2_nearest_even((int64_t)in[i], shift);
        if (q > hi) q = hi;
        if (q < lo) q = lo;
        out[i] = (int32_t)q;
    }
    return ORACLE_OK;
}

uint16_t oracle_bf16_from_double(double x)
{
    const uint16_t sign = signbit(x) ? 0x8000u : 0u;
    if (isnan(x)) return (uint16_t)(sign | 0x7FC0u);   /* NaN stays NaN (the quiet NaN) */
    const double ax = fabs(x);
    if (ax == 0.0) return sign;
    int e;
    (void)frexp(ax, &e);                     /* ax = m * 2^e, 0.5 <= m < 1 */
    int ulp_exp = e - 8;                     /* 8 significant bits */
    if (ulp_exp < -133) ulp_exp = -133;      /* subnormal bf16 spacing */
    const double r = nearbyint(ldexp(ax, -ulp_exp));   /* ties to even (default mode) */
    const double y = ldexp(r, ulp_exp);
    if (y > 0x1.fep127) return (uint16_t)(sign | 0x7F80u);   /* beyond the largest finite bf16 */
    const float f = (float)y;                /* exact: y has at most 8 significant bits */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return (uint16_t)(sign | (uint16_t)((u >> 16) & 0x7FFFu));
}

int oracle_round_bf16(const double *in, int64_t n, uint16_t *out)
{
    if (n < 0 || (n > 0 && (in == NULL || out == NULL))) return ORACLE_EINVAL;
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_bf16_from_double(in[i]);
    return ORACLE_OK;
}
