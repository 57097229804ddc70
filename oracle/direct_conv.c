/*
 * CPU oracle helper -- TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).
 *
 * Direct causal convolution y[t] = sum_{j=0}^{t} h[t-j] u[j] (eq. "cnn",
 * Sec. 2 of the paper), float64, written exactly as the definition: one dot
 * product per output, no FFT, no blocking, no reordering of the sum.  Rows are
 * independent and are spread over OpenMP threads.
 */
#include <stdint.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* h, u, y: [nrows, L] row-major float64; row i of y is h[i] (*) u[i]. */
void oracle_causal_conv_rows(const double* h, const double* u, double* y,
                             int64_t nrows, int64_t L)
{
    int64_t i;
#pragma omp parallel for schedule(dynamic, 1)
    for (i = 0; i < nrows; ++i) {
        const double* hi = h + i * L;
        const double* ui = u + i * L;
        double* yi = y + i * L;
        for (int64_t t = 0; t < L; ++t) {
            double acc = 0.0;
            for (int64_t j = 0; j <= t; ++j)
                acc += hi[t - j] * ui[j];
            yi[t] = acc;
        }
    }
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
