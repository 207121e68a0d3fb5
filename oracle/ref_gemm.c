/*
 * Oracle: plain fp64 GEMM rows, C[i][j] = sum_k A[i][k] * B[j][k].
 *
 * TEST INFRASTRUCTURE ONLY. Built by oracle/build.py with gcc; loaded by the
 * tests, the smoke check and the CPU-baseline leg of the benchmark, never by the
 * product library.
 *
 * The fused operator keeps the plain GEMM's numerical meaning (Overview,
 * architecture and output paragraph); the local kernel computes
 * acc = a . b^T with B held as N x K, K contiguous (the paper's annotated local
 * kernel). This file is that definition written out: every output element is one
 * fp64 sum over k in ascending order of exact fp64 products of the inputs
 * (bf16 or fp32 values are exactly representable in fp64 and so are their
 * products). No blocking, no reassociation.
 *
 * dtype codes: 0 = bf16 (uint16 bit patterns), 1 = fp32.
 */
#include <stdint.h>
#include <string.h>

static double load_elem(const void* base, int dtype, int64_t idx) {
    if (dtype == 0) {
        uint32_t w = ((uint32_t)((const uint16_t*)base)[idx]) << 16;
        float f;
        memcpy(&f, &w, sizeof f);
        return (double)f;
    }
    return (double)((const float*)base)[idx];
}

/* Rows listed in `rows` (n_rows of them) of C = A . B^T.
 * A: row-major with K columns; B: N x K row-major; C: n_rows x N fp64 (row r of C
 * holds output row rows[r]). */
void oracle_gemm_rows(const void* A, int a_dtype, const void* B, int b_dtype,
                      int64_t N, int64_t K, const int64_t* rows, int64_t n_rows, double* C) {
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < n_rows; r++) {
        int64_t i = rows[r];
        for (int64_t j = 0; j < N; j++) {
            double acc = 0.0;
            for (int64_t k = 0; k < K; k++)
                acc += load_elem(A, a_dtype, i * K + k) * load_elem(B, b_dtype, j * K + k);
            C[r * N + j] = acc;
        }
    }
}

/* Single elements (i, j) of C = A . B^T. */
void oracle_gemm_elems(const void* A, int a_dtype, const void* B, int b_dtype, int64_t K,
                       const int64_t* ii, const int64_t* jj, int64_t n, double* out) {
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < n; r++) {
        double acc = 0.0;
        for (int64_t k = 0; k < K; k++)
            acc += load_elem(A, a_dtype, ii[r] * K + k) * load_elem(B, b_dtype, jj[r] * K + k);
        out[r] = acc;
    }
}

int oracle_num_threads(void) {
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
