// C ABI of libcliffconv: argument checks, the signature-driven sign table and
// kernel dispatch.  No device memory is allocated here; every call only
// enqueues kernels on the caller's stream.
#include <atomic>
#include <stdint.h>
#include <stdlib.h>

#include <initializer_list>

#include "cliffconv.h"
#include "common.hpp"

namespace cliff {

bool debug_enabled()
{
    static const bool on = [] {
        const char* v = getenv("CLIFFCONV_DEBUG");
        return v && v[0] && !(v[0] == '0' && v[1] == 0);
    }();
    return on;
}

LaunchObserver* launch_observer = nullptr;

int device_cus()
{
    if (launch_observer) return launch_observer->cus;
    static std::atomic<int> cus[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    int c = cus[dev].load(std::memory_order_relaxed);
    if (c == 0) {
        if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return 0;
        cus[dev].store(c, std::memory_order_relaxed);
    }
    return c;
}

}  // namespace cliff

namespace {

using namespace cliff;

// Automatic choice of the fused small-block kernel, from the GPU time of both
// paths on 12 small blocks (2D: fused 1.2-2.2x faster up to 0.28 GFLOP, slower
// from 1.1; 3D: faster up to 0.03 GFLOP, even at 0.17, slower at 0.32).
constexpr int64_t CLIFF_BLOCK_FUSED_MAX_C = 16;
constexpr int64_t CLIFF_BLOCK_FUSED_MAX_FLOPS_2D = 300000000;
constexpr int64_t CLIFF_BLOCK_FUSED_MAX_FLOPS_3D = 100000000;

bool valid_k(int k) { return k >= 1 && k <= 3; }

bool valid_signature(int k, const int8_t* g)
{
    bool any = false;
    for (int t = 0; t < k; ++t) {
        if (g[t] < -1 || g[t] > 1) return false;
        any = any || g[t] != 0;
    }
    return any;  // a signature needs at least one non-zero entry
}

// Sign table of the geometric product (paper, Background, "Clifford
// Algebra"), closed form on generator bitmasks: for basis blades with masks
// a and b, e_a e_b = (-1)^{#pairs (p in a, q in b) with p > q}
//                    * prod_{t in a AND b} g_t * e_{a XOR b};
// the first factor counts the exchanges that sort the concatenated word, the
// second contracts the repeated generators with e_t e_t = g_t.
int blade_product_sign(int k, const int8_t* g, int a, int b)
{
    int swaps = 0;
    for (int q = 0; q < k; ++q)
        if ((b >> q) & 1) swaps += __builtin_popcount(a >> (q + 1));
    int s = (swaps & 1) ? -1 : 1;
    for (int t = 0; t < k; ++t)
        if (((a & b) >> t) & 1) s *= g[t];
    return s;
}

// Table in storage (grade-lex) order: (w * x)_i = sum_j sign[i][j] w_src[i][j] x_j.
void make_table(int k, const int8_t* g, int8_t* src, int8_t* sign)
{
    const int nb = 1 << k;
    for (int i = 0; i < nb; ++i)
        for (int j = 0; j < nb; ++j) {
            const int mi = blade_perm(nb, i), mj = blade_perm(nb, j);
            const int ma = mi ^ mj;
            src[i * nb + j] = (int8_t)blade_perm(nb, ma);
            sign[i * nb + j] = (int8_t)blade_product_sign(k, g, ma, mj);
        }
}

SignMasks pack_signs(int nb, const int8_t* sign)
{
    SignMasks m{0, 0};
    for (int e = 0; e < nb * nb; ++e) {
        if (sign[e] == 0) m.zero |= 1ull << e;
        if (sign[e] < 0) m.neg |= 1ull << e;
    }
    return m;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
bool aligned4(const void* p) { return ((uintptr_t)p & 3u) == 0; }

bool overlaps(const void* a, int64_t a_bytes, const void* b, int64_t b_bytes)
{
    if (!a || !b || a_bytes <= 0 || b_bytes <= 0) return false;
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + (uintptr_t)b_bytes && b0 < a0 + (uintptr_t)a_bytes;
}

// Product of non-negative factors, or -1 once it reaches 2^40.
int64_t checked_count(std::initializer_list<int64_t> f)
{
    int64_t n = 1;
    for (int64_t v : f) {
        if (v < 0) return -1;
        if (v != 0 && n > ((int64_t)1 << 40) / v) return -1;
        n *= v;
    }
    return n < ((int64_t)1 << 40) ? n : -1;
}

int64_t ipow(int64_t a, int k)
{
    int64_t r = 1;
    for (int t = 0; t < k; ++t) r *= a;
    return r;
}

cliff_status check_act(const cliff_act_desc* act, int nb, bool* linear)
{
    if (act->mode < CLIFF_AGG_LINEAR || act->mode > CLIFF_AGG_MEAN) return CLIFF_EINVAL;
    if (act->K < 1 || act->K > nb) return CLIFF_EINVAL;
    unsigned seen = 0;
    for (int t = 0; t < act->K; ++t) {
        const int b = act->blade_idx[t];
        if (b < 0 || b >= nb || ((seen >> b) & 1u)) return CLIFF_EINVAL;
        seen |= 1u << b;
    }
    *linear = act->mode == CLIFF_AGG_LINEAR;
    if (*linear && (!act->weight || !act->bias)) return CLIFF_EINVAL;
    if (*linear && (!aligned4(act->weight) || !aligned4(act->bias))) return CLIFF_EALIGN;
    return CLIFF_OK;
}

ActParams to_params(const cliff_act_desc* act)
{
    ActParams a;
    a.mode = -1;
    a.K = 0;
    for (int b = 0; b < 8; ++b) a.slot[b] = -1;
    a.weight = nullptr;
    a.bias = nullptr;
    if (act) {
        a.mode = act->mode;
        a.K = act->K;
        for (int t = 0; t < act->K; ++t) a.slot[act->blade_idx[t]] = t;
        if (act->mode == CLIFF_AGG_LINEAR) {
            a.weight = act->weight;
            a.bias = act->bias;
        }
    }
    return a;
}

// Linear layers: the streamed kernel from 16384 rows on (measured on MI355X
// over 7 widths: from there it beats every convolution tile; below, the
// tiny and medium tiles are 1-4 us faster).
bool linear_stream_pays(const ConvProblem& p)
{
    return p.B >= 16 * 1024;
}

}  // namespace

extern "C" {

cliff_status clifford_conv_nd_algo(int k, const int8_t* g, int64_t B, int64_t C_in,
                                   int64_t C_out, int64_t d_image, int64_t d_filter,
                                   const float* input, const float* filters, const float* bias,
                                   float* output, const cliff_act_desc* act, void* stream,
                                   int algo)
{
    if (!g || !input || !filters || !output) return CLIFF_EINVAL;
    if (!valid_k(k) || !valid_signature(k, g)) return CLIFF_EINVAL;
    if (algo < CLIFF_ALGO_AUTO || algo > CLIFF_ALGO_MFMA_STREAM) return CLIFF_EINVAL;
    const int nb = 1 << k;
    bool linear = false;
    if (act) {
        const cliff_status s = check_act(act, nb, &linear);
        if (s != CLIFF_OK) return s;
    }
    if (B < 0 || C_in < 1 || C_out < 1 || d_filter < 1 || d_image < d_filter)
        return CLIFF_ESHAPE;
    const int64_t d_out = d_image - d_filter + 1;
    const int64_t n_in = checked_count({B, C_in, ipow(d_image, k), nb});
    const int64_t n_f = checked_count({C_in, C_out, ipow(d_filter, k), nb});
    const int64_t n_out = checked_count({B, C_out, ipow(d_out, k), nb});
    if (d_image >= (1 << 20) || n_in < 0 || n_f < 0 || n_out < 0) return CLIFF_ESHAPE;
    if (!aligned16(input) || !aligned16(filters) || !aligned16(output) ||
        (bias && !aligned16(bias)))
        return CLIFF_EALIGN;
    const int64_t out_bytes = n_out * 4;
    if (overlaps(output, out_bytes, input, n_in * 4) ||
        overlaps(output, out_bytes, filters, n_f * 4) ||
        overlaps(output, out_bytes, bias, C_out * nb * 4) ||
        (linear && (overlaps(output, out_bytes, act->weight, C_out * act->K * 4) ||
                    overlaps(output, out_bytes, act->bias, C_out * 4))))
        return CLIFF_EOVERLAP;
    const bool mfma_forced = algo >= CLIFF_ALGO_MFMA;
    if (B == 0) return CLIFF_OK;

    int8_t src[64], sign[64];
    make_table(k, g, src, sign);
    ConvProblem p;
    p.k = k;
    p.nb = nb;
    p.B = B;
    p.C_in = C_in;
    p.C_out = C_out;
    p.d_image = d_image;
    p.d_filter = d_filter;
    p.d_out = d_out;
    p.x = input;
    p.w = filters;
    p.bias = bias;
    p.y = output;
    p.sign = pack_signs(nb, sign);
    p.act = to_params(act);
    p.mfma_shape = algo >= CLIFF_ALGO_MFMA_WIDE && algo <= CLIFF_ALGO_MFMA_TINY
                       ? algo - CLIFF_ALGO_MFMA_WIDE
                       : -1;
    hipStream_t st = (hipStream_t)stream;

    if (algo == CLIFF_ALGO_DIRECT) return launch_conv_direct(p, st);
    if (algo == CLIFF_ALGO_MFMA_STREAM) return launch_linear_mfma(p, st);
    if ((algo == CLIFF_ALGO_AUTO || algo == CLIFF_ALGO_MFMA) && d_image == 1 &&
        linear_stream_pays(p)) {
        const cliff_status s = launch_linear_mfma(p, st);
        if (s != CLIFF_EUNSUPPORTED) return s;
    }
    const cliff_status s = k == 1 ? launch_conv1d_mfma(p, st) : launch_conv_mfma(p, st);
    if (s != CLIFF_EUNSUPPORTED || mfma_forced) return s;
    return launch_conv_direct(p, st);
}

cliff_status clifford_conv_nd(int k, const int8_t* g, int64_t B, int64_t C_in, int64_t C_out,
                              int64_t d_image, int64_t d_filter, const float* input,
                              const float* filters, const float* bias, float* output,
                              const cliff_act_desc* act, void* stream)
{
    return clifford_conv_nd_algo(k, g, B, C_in, C_out, d_image, d_filter, input, filters, bias,
                                 output, act, stream, CLIFF_ALGO_AUTO);
}

cliff_status clifford_linear(int k, const int8_t* g, int64_t B, int64_t C_in, int64_t C_out,
                             const float* input, const float* weight, const float* bias,
                             float* output, const cliff_act_desc* act, void* stream)
{
    // Algorithm 2 is Algorithm 1 with a single position and a single tap
    return clifford_conv_nd_algo(k, g, B, C_in, C_out, 1, 1, input, weight, bias, output, act,
                                 stream, CLIFF_ALGO_AUTO);
}

cliff_status clifford_block2_nd_path(int k, const int8_t* g, int64_t B, int64_t C_in,
                                    int64_t C_mid, int64_t C_out, int64_t d_image,
                                    int64_t d_filter, const float* input, const float* filters1,
                                    const float* bias1, const cliff_act_desc* act1,
                                    const float* filters2, const float* bias2,
                                    const cliff_act_desc* act2, float* workspace, float* output,
                                    void* stream, int path)
{
    if (!g || !input || !filters1 || !filters2 || !workspace || !output) return CLIFF_EINVAL;
    if (!valid_k(k) || !valid_signature(k, g)) return CLIFF_EINVAL;
    if (path < CLIFF_BLOCK_AUTO || path > CLIFF_BLOCK_FUSED) return CLIFF_EINVAL;
    const int nb = 1 << k;
    bool lin1 = false, lin2 = false;
    if (act1) {
        const cliff_status s = check_act(act1, nb, &lin1);
        if (s != CLIFF_OK) return s;
    }
    if (act2) {
        const cliff_status s = check_act(act2, nb, &lin2);
        if (s != CLIFF_OK) return s;
    }
    if (B < 0 || C_in < 1 || C_mid < 1 || C_out < 1 || d_filter < 1 ||
        d_image < 2 * d_filter - 1)
        return CLIFF_ESHAPE;
    const int64_t d_mid = d_image - d_filter + 1, d_out = d_mid - d_filter + 1;
    const int64_t n_in = checked_count({B, C_in, ipow(d_image, k), nb});
    const int64_t n_f1 = checked_count({C_in, C_mid, ipow(d_filter, k), nb});
    const int64_t n_mid = checked_count({B, C_mid, ipow(d_mid, k), nb});
    const int64_t n_f2 = checked_count({C_mid, C_out, ipow(d_filter, k), nb});
    const int64_t n_out = checked_count({B, C_out, ipow(d_out, k), nb});
    if (d_image >= (1 << 20) || n_in < 0 || n_f1 < 0 || n_mid < 0 || n_f2 < 0 || n_out < 0)
        return CLIFF_ESHAPE;
    if (!aligned16(input) || !aligned16(filters1) || !aligned16(filters2) ||
        !aligned16(workspace) || !aligned16(output) || (bias1 && !aligned16(bias1)) ||
        (bias2 && !aligned16(bias2)))
        return CLIFF_EALIGN;
    // The workspace and the output are written; neither may overlap anything
    // else the block reads or writes.
    struct Buf {
        const void* p;
        int64_t bytes;
    };
    const Buf reads[] = {{input, n_in * 4},
                         {filters1, n_f1 * 4},
                         {bias1, C_mid * nb * 4},
                         {filters2, n_f2 * 4},
                         {bias2, C_out * nb * 4},
                         {lin1 ? act1->weight : nullptr, C_mid * (act1 ? act1->K : 0) * 4},
                         {lin1 ? act1->bias : nullptr, C_mid * 4},
                         {lin2 ? act2->weight : nullptr, C_out * (act2 ? act2->K : 0) * 4},
                         {lin2 ? act2->bias : nullptr, C_out * 4}};
    for (const Buf& r : reads)
        if (overlaps(workspace, n_mid * 4, r.p, r.bytes) || overlaps(output, n_out * 4, r.p, r.bytes))
            return CLIFF_EOVERLAP;
    if (overlaps(workspace, n_mid * 4, output, n_out * 4)) return CLIFF_EOVERLAP;
    if (B == 0) return CLIFF_OK;

    hipStream_t st = (hipStream_t)stream;
    bool fused = path == CLIFF_BLOCK_FUSED;
    if (path == CLIFF_BLOCK_AUTO) {
        // The fused kernel wins while the block is latency-bound: few
        // channels (its MFMA tiles are not staged for reuse) and a small
        // total amount of work.
        const int64_t flops = 2 * B * nb * nb * ipow(d_filter, k) *
                              (C_in * C_mid * ipow(d_mid, k) + C_mid * C_out * ipow(d_out, k));
        fused = k >= 2 && C_in <= CLIFF_BLOCK_FUSED_MAX_C && C_mid <= CLIFF_BLOCK_FUSED_MAX_C &&
                C_out <= CLIFF_BLOCK_FUSED_MAX_C &&
                flops <= (k == 2 ? CLIFF_BLOCK_FUSED_MAX_FLOPS_2D : CLIFF_BLOCK_FUSED_MAX_FLOPS_3D);
    }
    if (fused) {
        int8_t src[64], sign[64];
        make_table(k, g, src, sign);
        BlockProblem p;
        p.k = k;
        p.B = B;
        p.C_in = C_in;
        p.C_mid = C_mid;
        p.C_out = C_out;
        p.d_image = d_image;
        p.d_filter = d_filter;
        p.x = input;
        p.w1 = filters1;
        p.b1 = bias1;
        p.w2 = filters2;
        p.b2 = bias2;
        p.y = output;
        p.sign = pack_signs(nb, sign);
        p.act1 = to_params(act1);
        p.act2 = to_params(act2);
        const cliff_status s = launch_block_small(p, st);
        if (s != CLIFF_EUNSUPPORTED || path == CLIFF_BLOCK_FUSED) return s;
    }
    // two launches through the workspace
    cliff_status s = clifford_conv_nd(k, g, B, C_in, C_mid, d_image, d_filter, input, filters1,
                                      bias1, workspace, act1, stream);
    if (s != CLIFF_OK) return s;
    return clifford_conv_nd(k, g, B, C_mid, C_out, d_mid, d_filter, workspace, filters2, bias2,
                            output, act2, stream);
}

cliff_status clifford_block2_nd(int k, const int8_t* g, int64_t B, int64_t C_in, int64_t C_mid,
                                int64_t C_out, int64_t d_image, int64_t d_filter,
                                const float* input, const float* filters1, const float* bias1,
                                const cliff_act_desc* act1, const float* filters2,
                                const float* bias2, const cliff_act_desc* act2,
                                float* workspace, float* output, void* stream)
{
    return clifford_block2_nd_path(k, g, B, C_in, C_mid, C_out, d_image, d_filter, input,
                                   filters1, bias1, act1, filters2, bias2, act2, workspace,
                                   output, stream, CLIFF_BLOCK_AUTO);
}

cliff_status multivector_act(int nb, int64_t B, int64_t C, int64_t P,
                             const cliff_act_desc* act, const float* input, float* output,
                             void* stream)
{
    if (!act || !input || !output) return CLIFF_EINVAL;
    if (nb != 2 && nb != 4 && nb != 8) return CLIFF_EINVAL;
    bool linear = false;
    const cliff_status s = check_act(act, nb, &linear);
    if (s != CLIFF_OK) return s;
    if (B < 0 || C < 1 || P < 1) return CLIFF_ESHAPE;
    const int64_t n = checked_count({B, C, P, nb});
    if (n < 0) return CLIFF_ESHAPE;
    if (!aligned16(input) || !aligned16(output)) return CLIFF_EALIGN;
    const int64_t bytes = n * 4;
    if ((output != input && overlaps(output, bytes, input, bytes)) ||
        (linear && (overlaps(output, bytes, act->weight, C * act->K * 4) ||
                    overlaps(output, bytes, act->bias, C * 4))))
        return CLIFF_EOVERLAP;
    if (B == 0) return CLIFF_OK;
    return launch_act(nb, B, C, P, to_params(act), input, output, (hipStream_t)stream);
}

cliff_status cliffconv_cayley_table(int k, const int8_t* g, int8_t* src, int8_t* sign)
{
    if (!g || !src || !sign) return CLIFF_EINVAL;
    if (!valid_k(k)) return CLIFF_EINVAL;
    for (int t = 0; t < k; ++t)
        if (g[t] < -1 || g[t] > 1) return CLIFF_EINVAL;
    make_table(k, g, src, sign);
    return CLIFF_OK;
}

const char* cliffconv_status_string(cliff_status s)
{
    switch (s) {
    case CLIFF_OK: return "ok";
    case CLIFF_EINVAL: return "invalid argument (null pointer, k, signature or activation)";
    case CLIFF_ESHAPE: return "invalid shape";
    case CLIFF_EALIGN: return "pointer not aligned";
    case CLIFF_EOVERLAP: return "output overlaps an input";
    case CLIFF_EUNSUPPORTED: return "unsupported by the library";
    case CLIFF_EDEVICE: return "HIP device error";
    case CLIFF_ESCRATCH: return "intermediate exceeds the library's fixed scratch array";
    }
    return "unknown status";
}

}  // extern "C"
