/*
 * Oracle (TEST INFRASTRUCTURE ONLY): the plain definition of the sparse
 * product the paper's kernel computes (Section VI, Algorithm "High-Performance
 * UnionSparse Kernel": Y = W X for the decoded weight matrix). IE-BME is
 * lossless, so the result is the ordinary matrix product of the masked INT4
 * weights with the INT4 activations, accumulated here in int64.
 *
 *   W  : int8 [M][K]   row-major, values in [-8, 7] (0 = pruned)
 *   Xt : int8 [N][K]   row-major, row n is activation column n
 *   Y  : int64 [M][N]  row-major, Y[m][n] = sum_k W[m][k] * Xt[n][k]
 *
 * One OpenMP thread per block of output rows; no blocking, no vectorisation
 * hints. Only tests, the smoke check and the CPU-baseline leg of the
 * benchmark call it.
 */
#include <stdint.h>

void oracle_matmul_i64(const int8_t *W, const int8_t *Xt, int64_t M, int64_t K,
                       int64_t N, int64_t *Y)
{
    int64_t m;
#pragma omp parallel for schedule(static)
    for (m = 0; m < M; ++m) {
        for (int64_t n = 0; n < N; ++n) {
            int64_t acc = 0;
            for (int64_t k = 0; k < K; ++k)
                acc += (int64_t)W[m * K + k] * (int64_t)Xt[n * K + k];
            Y[m * N + n] = acc;
        }
    }
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads for later products (n >= 1); used to time the product on one core. */
void oracle_set_threads(int n)
{
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    omp_set_num_threads(n);
#else
    (void)n;
#endif
}
