/*
 * Test infrastructure: the oracle's group-wise steps 6-7 in plain C, for
 * checking whole full-size outputs (the numpy form materialises every
 * per-group accumulator and needs minutes per layer at those sizes).
 * Only the tests may load it.  It shares nothing with the HIP path.
 *
 * Group-wise W4A4 (the per-group variant of Sec. 3.1): for an output (m, n)
 * and each group g of G consecutive codes along K, the integer dot product
 * of the two code slices is exact; the fp32 partial is the accumulator
 * times the activation group scale, then times the weight group scale, each
 * product rounded to fp32; the output's fp32 sum adds the partials one
 * group after another, starting from +0.  This is the reading the numpy
 * oracle (w4a4_group.py) states, and the tests require the two to agree
 * bit for bit.
 *
 * Build: gcc -O3 -ffp-contract=off -fno-fast-math -shared -fPIC
 * (no contraction: every product and sum is its own fp32 rounding).
 */
#include <stdint.h>

/*
 * S[m * N + n] for m0 <= m < m1 and n0 <= n < n1.
 *   qx  int8 codes [M, K], row-major (one code per byte, -8..7)
 *   sx  fp32 activation group scales [M, K / G]
 *   qw  int8 codes [N, K], row-major
 *   sw  fp32 weight group scales [N, K / G]
 *   S   fp32 output [M, N]; only the rectangle is written
 * The caller checks K % G == 0, G <= 2^18 (so |accumulator| <= 2^24 and its
 * conversion to fp32 is exact) and the rectangle's bounds.
 */
void oracle_group_sum_rect(const int8_t *qx, const float *sx, const int8_t *qw, const float *sw,
                           int64_t N, int64_t K, int64_t G, int64_t m0, int64_t m1, int64_t n0, int64_t n1,
                           float *S)
{
    const int64_t ng = K / G;
    for (int64_t m = m0; m < m1; ++m) {
        for (int64_t n = n0; n < n1; ++n) {
            float s = 0.0f;
            for (int64_t g = 0; g < ng; ++g) {
                const int8_t *a = qx + m * K + g * G;
                const int8_t *b = qw + n * K + g * G;
                int32_t acc = 0;
                for (int64_t k = 0; k < G; ++k)
                    acc += (int32_t)a[k] * (int32_t)b[k];
                float t = (float)acc;
                t = t * sx[m * ng + g];
                t = t * sw[n * ng + g];
                s = s + t;
            }
            S[m * N + n] = s;
        }
    }
}
