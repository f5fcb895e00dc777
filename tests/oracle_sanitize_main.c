/* Drives every oracle entry point on small cases; built with
 * -fsanitize=address,undefined by tests/test_oracle_sanitize.py so that any
 * out-of-bounds access or undefined behaviour in the oracle fails the test. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_cayley(int k, const int* g, int* blade_out, double* sign);
int oracle_mv_mul(int k, const int* g, const double* x, const double* y, double* z);
int oracle_conv_nd(int k, const int* g, int64_t B, int64_t C_in, int64_t C_out,
                   int64_t d_image, int64_t d_filter, const double* input,
                   const double* filters, const double* bias, double* output, int nthreads);
int oracle_conv_points(int k, const int* g, int64_t B, int64_t C_in, int64_t C_out,
                       int64_t d_image, int64_t d_filter, const double* input,
                       const double* filters, const double* bias, int64_t n,
                       const int64_t* bs, const int64_t* cos, const int64_t* ps, double* out);
int oracle_act(int nb, int64_t B, int64_t C, int64_t P, int mode, int K, const int* idx,
               const double* weight, const double* bias, const double* input, double* output);
int oracle_linear(int k, const int* g, int64_t B, int64_t C_in, int64_t C_out,
                  const double* input, const double* weight, const double* bias,
                  double* output);

static double* filled(size_t n)
{
    double* p = (double*)malloc(n * sizeof(double));
    for (size_t i = 0; i < n; ++i) p[i] = (double)((i * 7919u) % 101) / 50.0 - 1.0;
    return p;
}

static int64_t ipow(int64_t a, int k)
{
    int64_t r = 1;
    for (int t = 0; t < k; ++t) r *= a;
    return r;
}

int main(void)
{
    const int gs[3][3] = {{-1, 0, 0}, {1, -1, 0}, {1, 0, -1}};
    for (int k = 1; k <= 3; ++k) {
        const int* g = gs[k - 1];
        const int nb = 1 << k;
        int blade[64];
        double sign[64];
        if (oracle_cayley(k, g, blade, sign) != nb) return 1;
        double x[8], y[8], z[8];
        for (int i = 0; i < nb; ++i) { x[i] = i + 1; y[i] = 2 - i; }
        if (oracle_mv_mul(k, g, x, y, z)) return 2;
        const int64_t B = 2, Ci = 3, Co = 2, D = 6, F = 3, Do = D - F + 1;
        double* in = filled((size_t)(B * Ci * ipow(D, k) * nb));
        double* f = filled((size_t)(Ci * Co * ipow(F, k) * nb));
        double* b = filled((size_t)(Co * nb));
        double* out = filled((size_t)(B * Co * ipow(Do, k) * nb));
        if (oracle_conv_nd(k, g, B, Ci, Co, D, F, in, f, b, out, 3)) return 3;
        int64_t bs[2] = {0, 1}, cs[2] = {1, 0}, ps[2] = {0, ipow(Do, k) - 1};
        double pts[16];
        if (oracle_conv_points(k, g, B, Ci, Co, D, F, in, f, NULL, 2, bs, cs, ps, pts)) return 4;
        int idx[2] = {0, nb - 1};
        double aw[4] = {0.5, -0.5, 1.0, 2.0}, ab[2] = {0.1, -0.1};
        double* ao = filled((size_t)(B * Co * ipow(Do, k) * nb));
        if (oracle_act(nb, B, Co, ipow(Do, k), 0, 2, idx, aw, ab, out, ao)) return 5;
        if (oracle_act(nb, B, Co, ipow(Do, k), 2, 2, idx, NULL, NULL, out, out)) return 6;
        double* lo = filled((size_t)(B * Co * nb));
        if (oracle_linear(k, g, B, Ci, Co, in, f, b, lo)) return 7;
        /* rejected arguments must not touch memory */
        if (oracle_conv_nd(k, g, B, Ci, Co, 2, 3, in, f, b, out, 1) == 0) return 8;
        int64_t bad_b = B;
        if (oracle_conv_points(k, g, B, Ci, Co, D, F, in, f, b, 1, &bad_b, cs, ps, pts) == 0)
            return 9;
        free(in); free(f); free(b); free(out); free(ao); free(lo);
    }
    puts("ok");
    return 0;
}
