// Per-output k-D Clifford convolution (paper, Algorithm 1): one thread per
// output multivector output[b, co, p], fp32 fused multiply-adds on the vector
// ALUs.  This is the general path: any k in {1, 2, 3} and any filter size,
// and the fallback for shapes whose slab does not fit the matrix-core tiling.
// Consecutive threads own consecutive positions of one (b, co), so the
// multivector loads of a wavefront are contiguous.
#include <stdio.h>

#include "common.hpp"
#include "direct_geom.hpp"
#include "epilogue.hpp"

namespace cliff {
namespace {

template <int KD, int NB>
__global__ __launch_bounds__(256) void conv_direct_kernel(DirectArgs a)
{
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= a.total) return;
    // (batch entry, output channel, position) and offsets: direct_geom.hpp
    const DirectThread d = direct_thread<KD>(a, t);
    const int co = d.co;

    float sg[NB][NB];
#pragma unroll
    for (int i = 0; i < NB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) sg[i][j] = sign_of(a.sign, i * NB + j);

    float o[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) o[i] = 0.f;

    for (int ci = 0; ci < a.C_in; ++ci) {
        const float* xb = a.x + direct_x(a, d, ci, NB);
        const float* wb = a.w + direct_w(a, d, ci, NB);
        for (int64_t q = 0; q < a.ntap; ++q) {
            const int64_t qoff = direct_qoff<KD>(a, q);
            float wv[NB], xv[NB];
#pragma unroll
            for (int i = 0; i < NB; ++i) {
                wv[i] = wb[q * NB + i];
                xv[i] = xb[qoff * NB + i];
            }
            // o += w * x, filter on the left
#pragma unroll
            for (int i = 0; i < NB; ++i)
#pragma unroll
                for (int j = 0; j < NB; ++j)
                    o[i] = fmaf(sg[i][j] * wv[src_blade(NB, i, j)], xv[j], o[i]);
        }
    }
    if (a.bias) {
#pragma unroll
        for (int i = 0; i < NB; ++i) o[i] += a.bias[co * NB + i];
    }
    if (a.act.mode >= 0) {
        float part = 0.f;
#pragma unroll
        for (int i = 0; i < NB; ++i) part += gate_coef(a.act, gate_slot(a.act, i), co) * o[i];
        const float g = gate_sigmoid(a.act, part, co);
#pragma unroll
        for (int i = 0; i < NB; ++i) o[i] *= g;
    }
    float* yp = a.y + t * NB;
#pragma unroll
    for (int i = 0; i < NB; ++i) yp[i] = o[i];
}

template <int KD, int NB>
cliff_status run(const ConvProblem& p, hipStream_t stream)
{
    DirectArgs a;
    a.x = p.x;
    a.w = p.w;
    a.bias = p.bias;
    a.y = p.y;
    a.C_in = (int)p.C_in;
    a.C_out = (int)p.C_out;
    a.D = (int)p.d_image;
    a.Do = (int)p.d_out;
    a.df = (int)p.d_filter;
    a.npos = a.nimg = a.ntap = 1;
    for (int d = 0; d < KD; ++d) {
        a.npos *= p.d_out;
        a.nimg *= p.d_image;
        a.ntap *= p.d_filter;
    }
    a.total = p.B * p.C_out * a.npos;
    a.sign = p.sign;
    a.act = p.act;
    const int64_t blocks = (a.total + 255) / 256;
    if (blocks >= (1ll << 31)) return CLIFF_EUNSUPPORTED;
    if (debug_enabled())
        fprintf(stderr, "cliffconv: conv_direct k=%d d_filter=%d, %lld workgroups of 256\n", KD,
                (int)p.d_filter, (long long)blocks);
    if (observe_launch(LAUNCH_CONV_DIRECT, {KD, NB}, blocks, 256, 0, &a)) return CLIFF_OK;
    clear_hip_error();
    hipLaunchKernelGGL((conv_direct_kernel<KD, NB>), dim3((unsigned)blocks), dim3(256), 0,
                       stream, a);
    return hipGetLastError() == hipSuccess ? CLIFF_OK : CLIFF_EDEVICE;
}

}  // namespace

cliff_status launch_conv_direct(const ConvProblem& p, hipStream_t stream)
{
    switch (p.k) {
    case 1: return run<1, 2>(p, stream);
    case 2: return run<2, 4>(p, stream);
    case 3: return run<3, 8>(p, stream);
    default: return CLIFF_EUNSUPPORTED;
    }
}

}  // namespace cliff
