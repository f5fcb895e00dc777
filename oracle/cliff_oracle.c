/*
 * Plain, slow fp64 reference ("oracle") for the Clifford convolution, the
 * Clifford linear layer and the multivector activation of "Fast Clifford
 * Neural Layers" (arXiv 2507.01040).
 *
 * TEST INFRASTRUCTURE ONLY.  This file exists to check the GPU library.  It
 * shares no code, header, table or constant with it, and the GPU library must
 * never call it: only the tests, the smoke check and the benchmark's CPU
 * baseline load it.
 *
 * Everything is computed in double precision from the caller's values, with
 * the summation order of the paper's algorithms.  No intrinsics, no
 * fast-math; build with -ffp-contract=off.
 *
 * Conventions (readings of the paper where it is silent):
 *  - Blade order inside a multivector: by grade, then lexicographically in the
 *    generator indices: k=2: (1, e1, e2, e12); k=3: (1, e1, e2, e3, e12, e13,
 *    e23, e123).  Blade indices are 0-based.
 *  - Product order in the convolution: filter on the left (Algorithm 1 writes
 *    filters[...] * input[...]).
 *  - Spatial indices are row-major, first axis slowest; the convolution is a
 *    cross-correlation (input[p + q], no flip).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define MAXK 3
#define MAXNB 8

/* ------------------------------------------------------------------------ */
/* Blade basis (Background, "Clifford Algebra": e_I is the product of the    */
/* generators of I in increasing index order, e_{} = 1).                      */
/* ------------------------------------------------------------------------ */

typedef struct {
    int len;
    int gen[MAXK]; /* generator indices 1..k in increasing order */
} blade_word;

/* Enumerate the subsets of {1..k} by grade, then lexicographically. */
static int make_basis(int k, blade_word* basis)
{
    int n = 0;
    for (int grade = 0; grade <= k; ++grade) {
        /* lexicographic enumeration of the grade-subsets via an index array */
        int idx[MAXK];
        for (int t = 0; t < grade; ++t) idx[t] = t + 1;
        for (;;) {
            basis[n].len = grade;
            for (int t = 0; t < grade; ++t) basis[n].gen[t] = idx[t];
            ++n;
            /* next combination */
            int t = grade - 1;
            while (t >= 0 && idx[t] == k - grade + t + 1) --t;
            if (t < 0) break;
            ++idx[t];
            for (int u = t + 1; u < grade; ++u) idx[u] = idx[u - 1] + 1;
        }
    }
    return n;
}

static int find_blade(const blade_word* basis, int nb, const int* gens, int len)
{
    for (int i = 0; i < nb; ++i) {
        if (basis[i].len != len) continue;
        int same = 1;
        for (int t = 0; t < len; ++t)
            if (basis[i].gen[t] != gens[t]) { same = 0; break; }
        if (same) return i;
    }
    return -1;
}

/*
 * Product of two basis blades by rewriting the word e_I e_J with the defining
 * relations e_i e_j = -e_j e_i (i != j) and e_i e_i = g_i (Background,
 * "Clifford Algebra"):
 *   1. concatenate the generator words of I and J;
 *   2. bubble-sort the word, flipping the sign at every exchange of two
 *      adjacent distinct generators;
 *   3. replace every adjacent equal pair e_i e_i by the scalar g_i.
 * Returns the blade index of the result and stores its coefficient (-1, 0 or
 * +1) in *coef.
 */
static int word_product(int k, const int* g, const blade_word* basis, int nb,
                        int a, int b, double* coef)
{
    int w[2 * MAXK];
    int n = 0;
    for (int t = 0; t < basis[a].len; ++t) w[n++] = basis[a].gen[t];
    for (int t = 0; t < basis[b].len; ++t) w[n++] = basis[b].gen[t];
    double c = 1.0;
    int swapped = 1;
    while (swapped) {
        swapped = 0;
        for (int t = 0; t + 1 < n; ++t) {
            if (w[t] > w[t + 1]) {
                int tmp = w[t]; w[t] = w[t + 1]; w[t + 1] = tmp;
                c = -c;
                swapped = 1;
            }
        }
    }
    int out[2 * MAXK];
    int m = 0;
    for (int t = 0; t < n; ++t) {
        if (t + 1 < n && w[t] == w[t + 1]) {
            c *= (double)g[w[t] - 1];
            ++t; /* both generators of the pair are consumed */
        } else {
            out[m++] = w[t];
        }
    }
    (void)k;
    *coef = c;
    return find_blade(basis, nb, out, m);
}

/* Public: the multiplication table, blade_out[a*nb+b] and sign[a*nb+b] such
 * that e_a e_b = sign * e_{blade_out}.  Returns N_B, or -1 on bad k. */
int oracle_cayley(int k, const int* g, int* blade_out, double* sign)
{
    if (k < 1 || k > MAXK) return -1;
    blade_word basis[MAXNB];
    int nb = make_basis(k, basis);
    for (int a = 0; a < nb; ++a)
        for (int b = 0; b < nb; ++b) {
            double c;
            blade_out[a * nb + b] = word_product(k, g, basis, nb, a, b, &c);
            sign[a * nb + b] = c;
        }
    return nb;
}

typedef struct {
    int nb;
    int blade[MAXNB * MAXNB];
    double sign[MAXNB * MAXNB];
} cayley;

static void make_cayley(int k, const int* g, cayley* t)
{
    t->nb = oracle_cayley(k, g, t->blade, t->sign);
}

/* Geometric product z += x * y of two multivectors (distribute, then
 * simplify each basis product with the table). */
static void mv_mul_acc(const cayley* t, const double* x, const double* y,
                       double* z)
{
    const int nb = t->nb;
    for (int a = 0; a < nb; ++a)
        for (int b = 0; b < nb; ++b)
            z[t->blade[a * nb + b]] += t->sign[a * nb + b] * x[a] * y[b];
}

/* Public: z = x * y for one pair of multivectors. */
int oracle_mv_mul(int k, const int* g, const double* x, const double* y,
                  double* z)
{
    if (k < 1 || k > MAXK) return -1;
    cayley t;
    make_cayley(k, g, &t);
    for (int i = 0; i < t.nb; ++i) z[i] = 0.0;
    mv_mul_acc(&t, x, y, z);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 1: k-D Clifford convolution (no padding, unit stride, no        */
/* dilation).                                                                */
/* ------------------------------------------------------------------------ */

typedef struct {
    int k, nb;
    int64_t B, C_in, C_out, d_image, d_filter, d_out;
    int64_t n_pos, n_tap, n_img;   /* d_out^k, d_filter^k, d_image^k */
    const double* input;   /* [B, C_in, d_image^k, N_B]   */
    const double* filters; /* [C_in, C_out, d_filter^k, N_B] */
    const double* bias;    /* [C_out, N_B] or NULL          */
    cayley tab;
} conv_problem;

/* Split a flat row-major index over an n^k grid into k coordinates. */
static void unflatten(int64_t flat, int k, int64_t n, int64_t* c)
{
    for (int t = k - 1; t >= 0; --t) {
        c[t] = flat % n;
        flat /= n;
    }
}

static int64_t flatten(const int64_t* c, int k, int64_t n)
{
    int64_t f = 0;
    for (int t = 0; t < k; ++t) f = f * n + c[t];
    return f;
}

/* One output multivector output[b, co, p] (Algorithm 1, body of the p loop). */
static void conv_one(const conv_problem* P, int64_t b, int64_t co, int64_t p,
                     double* o)
{
    const int nb = P->nb;
    int64_t pc[MAXK], qc[MAXK], ic[MAXK];
    unflatten(p, P->k, P->d_out, pc);
    for (int i = 0; i < nb; ++i) o[i] = 0.0;
    for (int64_t ci = 0; ci < P->C_in; ++ci) {
        for (int64_t q = 0; q < P->n_tap; ++q) {
            unflatten(q, P->k, P->d_filter, qc);
            for (int t = 0; t < P->k; ++t) ic[t] = pc[t] + qc[t];
            int64_t src = flatten(ic, P->k, P->d_image);
            const double* w =
                P->filters + ((ci * P->C_out + co) * P->n_tap + q) * nb;
            const double* x =
                P->input + ((b * P->C_in + ci) * P->n_img + src) * nb;
            mv_mul_acc(&P->tab, w, x, o); /* o = o + filters * input */
        }
    }
    if (P->bias)
        for (int i = 0; i < nb; ++i) o[i] += P->bias[co * nb + i];
}

typedef struct {
    const conv_problem* P;
    double* output;
    int64_t first, last; /* range of (b, co) pairs */
} conv_job;

static void* conv_worker(void* arg)
{
    conv_job* J = (conv_job*)arg;
    const conv_problem* P = J->P;
    for (int64_t bc = J->first; bc < J->last; ++bc) {
        int64_t b = bc / P->C_out, co = bc % P->C_out;
        for (int64_t p = 0; p < P->n_pos; ++p)
            conv_one(P, b, co, p,
                     J->output + ((b * P->C_out + co) * P->n_pos + p) * P->nb);
    }
    return NULL;
}

static int64_t ipow(int64_t a, int k)
{
    int64_t r = 1;
    for (int t = 0; t < k; ++t) r *= a;
    return r;
}

static int setup_problem(conv_problem* P, int k, const int* g, int64_t B,
                         int64_t C_in, int64_t C_out, int64_t d_image,
                         int64_t d_filter, const double* input,
                         const double* filters, const double* bias)
{
    if (k < 1 || k > MAXK || B < 0 || C_in < 1 || C_out < 1 || d_filter < 1 ||
        d_image < d_filter)
        return -1;
    P->k = k;
    make_cayley(k, g, &P->tab);
    P->nb = P->tab.nb;
    P->B = B; P->C_in = C_in; P->C_out = C_out;
    P->d_image = d_image; P->d_filter = d_filter;
    P->d_out = d_image - d_filter + 1;
    P->n_pos = ipow(P->d_out, k);
    P->n_tap = ipow(d_filter, k);
    P->n_img = ipow(d_image, k);
    P->input = input; P->filters = filters; P->bias = bias;
    return 0;
}

/* Public: the whole convolution, output [B, C_out, d_out^k, N_B], with the
 * (b, c_out) pairs split over nthreads POSIX threads. */
int oracle_conv_nd(int k, const int* g, int64_t B, int64_t C_in, int64_t C_out,
                   int64_t d_image, int64_t d_filter, const double* input,
                   const double* filters, const double* bias, double* output,
                   int nthreads)
{
    conv_problem P;
    if (setup_problem(&P, k, g, B, C_in, C_out, d_image, d_filter, input,
                      filters, bias))
        return -1;
    int64_t pairs = B * C_out;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > pairs) nthreads = (int)(pairs > 0 ? pairs : 1);
    pthread_t th[256];
    conv_job jobs[256];
    if (nthreads > 256) nthreads = 256;
    for (int t = 0; t < nthreads; ++t) {
        jobs[t].P = &P;
        jobs[t].output = output;
        jobs[t].first = pairs * t / nthreads;
        jobs[t].last = pairs * (t + 1) / nthreads;
    }
    for (int t = 1; t < nthreads; ++t)
        pthread_create(&th[t], NULL, conv_worker, &jobs[t]);
    conv_worker(&jobs[0]);
    for (int t = 1; t < nthreads; ++t) pthread_join(th[t], NULL);
    return 0;
}

/* Public: selected outputs only.  For sample s, out[s*N_B ..] =
 * output[b[s], co[s], p[s]] where p is the flat row-major output position. */
int oracle_conv_points(int k, const int* g, int64_t B, int64_t C_in,
                       int64_t C_out, int64_t d_image, int64_t d_filter,
                       const double* input, const double* filters,
                       const double* bias, int64_t n, const int64_t* bs,
                       const int64_t* cos, const int64_t* ps, double* out)
{
    conv_problem P;
    if (setup_problem(&P, k, g, B, C_in, C_out, d_image, d_filter, input,
                      filters, bias))
        return -1;
    for (int64_t s = 0; s < n; ++s) {
        if (bs[s] < 0 || bs[s] >= B || cos[s] < 0 || cos[s] >= C_out ||
            ps[s] < 0 || ps[s] >= P.n_pos)
            return -2;
        conv_one(&P, bs[s], cos[s], ps[s], out + s * P.nb);
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 3: multivector activation.  Spatial positions (if any) sit      */
/* between the channel and the blade axis and are treated like extra batch   */
/* entries that share the channel's weight and bias.                         */
/* ------------------------------------------------------------------------ */

/* Public.  input/output [B, C, P, N_B]; mode 0 = Linear, 1 = Sum, 2 = Mean;
 * idx: K 0-based blade indices; weight [C, K] and bias [C] (Linear only). */
int oracle_act(int nb, int64_t B, int64_t C, int64_t P, int mode, int K,
               const int* idx, const double* weight, const double* bias,
               const double* input, double* output)
{
    if (nb < 1 || nb > MAXNB || K < 1 || K > nb || mode < 0 || mode > 2)
        return -1;
    for (int t = 0; t < K; ++t)
        if (idx[t] < 0 || idx[t] >= nb) return -1;
    for (int64_t b = 0; b < B; ++b)
        for (int64_t c = 0; c < C; ++c)
            for (int64_t p = 0; p < P; ++p) {
                const double* x = input + ((b * C + c) * P + p) * nb;
                double* y = output + ((b * C + c) * P + p) * nb;
                double s = 0.0;
                if (mode == 0) {
                    for (int t = 0; t < K; ++t) s += x[idx[t]] * weight[c * K + t];
                    s = s + bias[c];
                } else {
                    for (int t = 0; t < K; ++t) s = s + x[idx[t]];
                    if (mode == 2) s = s / (double)K;
                }
                double sig = 1.0 / (1.0 + exp(-s));
                for (int j = 0; j < nb; ++j) y[j] = x[j] * sig;
            }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 2: Clifford linear layer.                                       */
/* ------------------------------------------------------------------------ */

/* Public.  input [B, C_in, N_B], weight [C_in, C_out, N_B], bias [C_out, N_B]
 * or NULL; output [B, C_out, N_B]:
 *   output[b, co] = sum_ci weight[ci, co] * input[b, ci] + bias[co]
 * (geometric product, weight on the left). */
int oracle_linear(int k, const int* g, int64_t B, int64_t C_in, int64_t C_out,
                  const double* input, const double* weight, const double* bias,
                  double* output)
{
    if (k < 1 || k > MAXK || B < 0 || C_in < 1 || C_out < 1) return -1;
    cayley t;
    make_cayley(k, g, &t);
    const int nb = t.nb;
    for (int64_t b = 0; b < B; ++b)
        for (int64_t co = 0; co < C_out; ++co) {
            double o[MAXNB];
            for (int i = 0; i < nb; ++i) o[i] = 0.0;
            for (int64_t ci = 0; ci < C_in; ++ci)
                mv_mul_acc(&t, weight + (ci * C_out + co) * nb, input + (b * C_in + ci) * nb, o);
            for (int i = 0; i < nb; ++i)
                output[(b * C_out + co) * nb + i] = o[i] + (bias ? bias[co * nb + i] : 0.0);
        }
    return 0;
}
