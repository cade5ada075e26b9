/*
 * Oracle: the plain definition of the matrix product that the adaptive GEMM
 * path computes (paper Section 4.1 and Section 5.1: every template, split and
 * schedule reaches the same C = A * B, only the order of fp32 additions
 * differs).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may link, load or call
 * this file; it exists so that tests, the smoke check and the CPU baseline of
 * the benchmark can compare the GPU path against an obviously correct result.
 * It shares no code, header or table with the GPU library.
 *
 *   C_ref[i][j] = sum_{k=0}^{K-1} A[i][k] * B[k][j]     (fp64, ascending k)
 *   D[i][j]     = sum_{k=0}^{K-1} |A[i][k] * B[k][j]|   (fp64)
 *
 * Inputs are 16-bit storage formats (bf16 or fp16), decoded here to their exact
 * values. A bf16 or fp16 value has at most 11 significant bits, so every
 * product of two of them is exact in fp64 and only the additions round.
 *
 * Layouts: A is row-major M x K with leading dimension lda (elements),
 * B is row-major K x N with leading dimension ldb, the outputs are row-major
 * with leading dimension ldc. Rows [row0, row1) are computed; the others are
 * untouched, so any subset of rows can be checked at any size.
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math [-fopenmp] -shared -fPIC.
 * The optional OpenMP loop runs over rows only, so the order of additions in
 * every entry is the same for any thread count.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

/* bf16: the upper 16 bits of an IEEE binary32. */
static double dec_bf16(uint16_t h) {
    uint32_t bits = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* fp16 (IEEE binary16): sign, 5-bit exponent (bias 15), 10-bit fraction. */
static double dec_fp16(uint16_t h) {
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int f = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);               /* zero or subnormal */
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(f | 0x400), e - 25);  /* 1.f * 2^(e-15) */
    return sign ? -v : v;
}

typedef double (*decode_fn)(uint16_t);

static decode_fn pick(int fmt) { return fmt == 1 ? dec_fp16 : dec_bf16; }

/* fmt: 0 = bf16, 1 = fp16. D may be NULL. */
int oracle_gemm(int fmt, int64_t M, int64_t N, int64_t K,
                const uint16_t *A, int64_t lda, const uint16_t *B, int64_t ldb,
                double *C, double *D, int64_t ldc, int64_t row0, int64_t row1) {
    if (M < 0 || N < 0 || K < 0 || row0 < 0 || row1 > M || row0 > row1) return -1;
    decode_fn dec = pick(fmt);
    int64_t i;
#pragma omp parallel for schedule(dynamic, 1)
    for (i = row0; i < row1; ++i) {
        double *c = C + (size_t)i * (size_t)ldc;
        double *d = D ? D + (size_t)i * (size_t)ldc : NULL;
        for (int64_t j = 0; j < N; ++j) {
            c[j] = 0.0;
            if (d) d[j] = 0.0;
        }
        for (int64_t k = 0; k < K; ++k) {
            double a = dec(A[(size_t)i * (size_t)lda + (size_t)k]);
            const uint16_t *brow = B + (size_t)k * (size_t)ldb;
            for (int64_t j = 0; j < N; ++j) {
                double p = a * dec(brow[j]);
                c[j] += p;
                if (d) d[j] += fabs(p);
            }
        }
    }
    return 0;
}

/* Single entries (I[t], J[t]) one by one, for checks at sizes where whole rows
 * are too costly. Ascending k, as above. */
int oracle_gemm_entries(int fmt, int64_t M, int64_t N, int64_t K,
                        const uint16_t *A, int64_t lda, const uint16_t *B, int64_t ldb,
                        const int64_t *I, const int64_t *J, int64_t n,
                        double *C, double *D) {
    decode_fn dec = pick(fmt);
    for (int64_t t = 0; t < n; ++t)
        if (I[t] < 0 || I[t] >= M || J[t] < 0 || J[t] >= N) return -1;
    int64_t t;
#pragma omp parallel for schedule(static)
    for (t = 0; t < n; ++t) {
        double c = 0.0, d = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            double p = dec(A[(size_t)I[t] * (size_t)lda + (size_t)k]) *
                       dec(B[(size_t)k * (size_t)ldb + (size_t)J[t]]);
            c += p;
            d += fabs(p);
        }
        C[t] = c;
        if (D) D[t] = d;
    }
    return 0;
}

/* Decode a buffer of 16-bit values (used to read back bf16 / fp16 outputs). */
void oracle_decode(int fmt, const uint16_t *src, double *dst, int64_t n) {
    decode_fn dec = pick(fmt);
    for (int64_t t = 0; t < n; ++t) dst[t] = dec(src[t]);
}

int oracle_threads(void) {
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
