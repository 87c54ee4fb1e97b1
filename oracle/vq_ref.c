/*
 * NOVA-KV test oracle -- plain fp64 nearest-codeword search.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this library; the product path never
 * does.  It shares no code with the GPU library.
 *
 * A vector quantizer's encoder maps a subvector to the index of its nearest
 * codeword (paper, Sec. "Transform coding", quantization paragraph); in the
 * transform domain that codeword is the one at the smallest squared Euclidean
 * distance, found exhaustively (paper, Sec. "Calibration").  This file is that definition
 * written out: the squared distance sum_i (u_i - c_i)^2 accumulated over i in
 * order, in fp64, and the smallest index among equal minima.
 *
 * Build: gcc -O3 -mavx2 -fopenmp -ffp-contract=off -shared -fPIC (see oracle/build.py).
 * -ffp-contract=off keeps each square and each sum a separately rounded
 * operation, exactly as written.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

/*
 * u     [n][g]   points (fp64)
 * cb_t  [g][k]   codebook, transposed: cb_t[i*k + c] is coordinate i of codeword c
 * codes [n]      index of the nearest codeword (lowest index among ties)
 * best  [n]      its squared distance
 * second[n]      the second-smallest squared distance over the other indices
 *                (equals best when a duplicate codeword ties)
 */
void oracle_nearest_codeword(const double *u, int64_t n, int32_t g,
                             const double *cb_t, int32_t k,
                             int32_t *codes, double *best, double *second)
{
#pragma omp parallel
    {
        double *dist = (double *)malloc(sizeof(double) * (size_t)k);
#pragma omp for schedule(static)
        for (int64_t j = 0; j < n; ++j) {
            const double *x = u + j * g;
            for (int32_t c = 0; c < k; ++c)
                dist[c] = 0.0;
            for (int32_t i = 0; i < g; ++i) {
                const double xi = x[i];
                const double *row = cb_t + (int64_t)i * k;
                for (int32_t c = 0; c < k; ++c) {
                    const double e = xi - row[c];
                    dist[c] = dist[c] + e * e;
                }
            }
            double b1 = INFINITY, b2 = INFINITY;
            int32_t arg = 0;
            for (int32_t c = 0; c < k; ++c) {
                const double s = dist[c];
                if (s < b1) {
                    b2 = b1;
                    b1 = s;
                    arg = c;
                } else if (s < b2) {
                    b2 = s;
                }
            }
            codes[j] = arg;
            best[j] = b1;
            second[j] = b2;
        }
        free(dist);
    }
}
