/*
 * CPU oracle for merged multi-model CNN inference: the two contractions
 * (direct convolution and fully connected layer), written out from their
 * definitions.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product library links, loads or
 * calls this file; it is used by the tests, the smoke check and the CPU
 * baseline leg of the benchmark. It shares no code with the HIP path.
 *
 * Data are float32 in NCHW order; every sum is accumulated in double and
 * rounded to float once, at the end. OpenMP spreads independent outputs
 * over cores; it never splits a sum.
 *
 * Model merging (Section 4 of the paper) changes where a layer's weights
 * live, not what a model computes, so nothing here knows about merging: the
 * oracle evaluates each model on its own frames with its effective weights.
 */
#include <stdint.h>
#include <stdlib.h>

/*
 * Direct 2-D convolution (cross-correlation, as deep-learning frameworks
 * define it):
 *   y[n,o,p,q] = bias[o] + sum_{c,i,j} x[n,c, p*s-pad+i, q*s-pad+j] * w[o,c,i,j]
 * with reads outside the input taken as zero, and
 *   Ho = floor((H + 2*pad - kh) / s) + 1, Wo likewise.
 * x: [n][c][h][w], w: [o][c][kh][kw], bias: [o] or NULL, y: [n][o][Ho][Wo].
 *
 * For one output plane (n, o) the terms are added in the order c, i, j; a
 * double accumulator plane holds the partial sums of all (p, q) at once.
 */
void oracle_conv2d(const float *x, int64_t n, int64_t c, int64_t h, int64_t w,
                   const float *wt, int64_t o, int64_t kh, int64_t kw,
                   int64_t s, int64_t pad, const float *bias, float *y)
{
    const int64_t ho = (h + 2 * pad - kh) / s + 1;
    const int64_t wo = (w + 2 * pad - kw) / s + 1;
#pragma omp parallel
    {
        double *acc = (double *)malloc(sizeof(double) * (size_t)(ho * wo));
#pragma omp for collapse(2) schedule(dynamic, 1)
        for (int64_t nn = 0; nn < n; ++nn) {
            for (int64_t oo = 0; oo < o; ++oo) {
                const double b0 = bias ? (double)bias[oo] : 0.0;
                for (int64_t t = 0; t < ho * wo; ++t)
                    acc[t] = b0;
                for (int64_t cc = 0; cc < c; ++cc) {
                    const float *xp = x + (nn * c + cc) * h * w;
                    for (int64_t i = 0; i < kh; ++i) {
                        for (int64_t j = 0; j < kw; ++j) {
                            const double wv =
                                wt[((oo * c + cc) * kh + i) * kw + j];
                            for (int64_t p = 0; p < ho; ++p) {
                                const int64_t hi = p * s - pad + i;
                                if (hi < 0 || hi >= h)
                                    continue;
                                double *ap = acc + p * wo;
                                const float *xr = xp + hi * w;
                                for (int64_t q = 0; q < wo; ++q) {
                                    const int64_t wi = q * s - pad + j;
                                    if (wi >= 0 && wi < w)
                                        ap[q] += wv * (double)xr[wi];
                                }
                            }
                        }
                    }
                }
                float *yp = y + (nn * o + oo) * ho * wo;
                for (int64_t t = 0; t < ho * wo; ++t)
                    yp[t] = (float)acc[t];
            }
        }
        free(acc);
    }
}

/*
 * Fully connected layer on a flattened input:
 *   y[n,o] = bias[o] + sum_k x[n,k] * w[o,k]
 * x: [n][k] (an NCHW tensor flattened in its own order), w: [o][k].
 */
void oracle_fc(const float *x, int64_t n, int64_t k, const float *wt,
               int64_t o, const float *bias, float *y)
{
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t nn = 0; nn < n; ++nn) {
        for (int64_t oo = 0; oo < o; ++oo) {
            double acc = bias ? (double)bias[oo] : 0.0;
            const float *xr = x + nn * k;
            const float *wr = wt + oo * k;
            for (int64_t kk = 0; kk < k; ++kk)
                acc += (double)xr[kk] * (double)wr[kk];
            y[nn * o + oo] = (float)acc;
        }
    }
}

/* Threads the OpenMP runtime will use (reported next to the CPU timing). */
int oracle_threads(void)
{
    int t = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            t = omp_get_num_threads();
#endif
        }
    }
    return t;
}
