// Standalone multivector activation (paper, Algorithm 3) on [B, C, P, N_B]:
// one thread per multivector, the gate computed once per multivector (not
// once per blade), blades loaded and stored as 16-byte vectors.  The kernel
// streams its input once and its output once, so HBM bandwidth bounds it.
#include "common.hpp"
#include "epilogue.hpp"

namespace cliff {
namespace {

struct ActKArgs {
    const float* x;
    float* y;
    int64_t n;  // B * C * P multivectors
    int64_t C, P;
    ActParams act;
};

template <int NB>
__global__ __launch_bounds__(256) void act_kernel(ActKArgs a)
{
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= a.n) return;
    const int c = (int)((t / a.P) % a.C);
    float v[NB];
    if (NB == 2) {
        const float2 u = reinterpret_cast<const float2*>(a.x)[t];
        v[0] = u.x;
        v[1] = u.y;
    } else {
#pragma unroll
        for (int h = 0; h < NB / 4; ++h) {
            const float4 u = reinterpret_cast<const float4*>(a.x)[t * (NB / 4) + h];
            v[4 * h + 0] = u.x;
            v[4 * h + 1] = u.y;
            v[4 * h + 2] = u.z;
            v[4 * h + 3] = u.w;
        }
    }
    float part = 0.f;
#pragma unroll
    for (int i = 0; i < NB; ++i) part += gate_coef(a.act, gate_slot(a.act, i), c) * v[i];
    const float g = gate_sigmoid(a.act, part, c);
    if (NB == 2) {
        reinterpret_cast<float2*>(a.y)[t] = make_float2(v[0] * g, v[1] * g);
    } else {
#pragma unroll
        for (int h = 0; h < NB / 4; ++h)
            reinterpret_cast<float4*>(a.y)[t * (NB / 4) + h] =
                make_float4(v[4 * h] * g, v[4 * h + 1] * g, v[4 * h + 2] * g, v[4 * h + 3] * g);
    }
}

}  // namespace

cliff_status launch_act(int nb, int64_t B, int64_t C, int64_t P, const ActParams& act,
                        const float* x, float* y, hipStream_t stream)
{
    ActKArgs a;
    a.x = x;
    a.y = y;
    a.n = B * C * P;
    a.C = C;
    a.P = P;
    a.act = act;
    const int64_t blocks = (a.n + 255) / 256;
    if (blocks >= (1ll << 31)) return CLIFF_EUNSUPPORTED;
    switch (nb) {
    case 2: hipLaunchKernelGGL(act_kernel<2>, dim3((unsigned)blocks), dim3(256), 0, stream, a); break;
    case 4: hipLaunchKernelGGL(act_kernel<4>, dim3((unsigned)blocks), dim3(256), 0, stream, a); break;
    case 8: hipLaunchKernelGGL(act_kernel<8>, dim3((unsigned)blocks), dim3(256), 0, stream, a); break;
    default: return CLIFF_EUNSUPPORTED;
    }
    return hipGetLastError() == hipSuccess ? CLIFF_OK : CLIFF_EDEVICE;
}

}  // namespace cliff
