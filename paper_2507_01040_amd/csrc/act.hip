// Standalone multivector activation (paper, Algorithm 3) on [B, C, P, N_B].
//
// The kernel streams its input once and its output once, so HBM bandwidth
// bounds it (8 N_B bytes per multivector).  Each workgroup owns a run of
// positions of one (b, c) pair, so the channel's gate weights and bias are
// uniform (scalar loads, computed once per workgroup), and each thread issues
// all loads of its VPT multivectors before any arithmetic.  The gate is
// computed once per multivector, not once per blade.  Data that is read or
// written once is accessed non-temporally.
#include <stdio.h>

#include "act_geom.hpp"
#include "common.hpp"
#include "epilogue.hpp"

namespace cliff {
namespace {

typedef float vf2 __attribute__((ext_vector_type(2)));
typedef float vf4 __attribute__((ext_vector_type(4)));



template <int NB>
struct MV {
    float v[NB];
};

template <int NB>
__device__ inline MV<NB> load_mv(const float* p)
{
    MV<NB> m;
    if constexpr (NB == 2) {
        const vf2 u = __builtin_nontemporal_load(reinterpret_cast<const vf2*>(p));
        m.v[0] = u.x;
        m.v[1] = u.y;
    } else {
#pragma unroll
        for (int h = 0; h < NB / 4; ++h) {
            const vf4 u = __builtin_nontemporal_load(reinterpret_cast<const vf4*>(p) + h);
            m.v[4 * h + 0] = u.x;
            m.v[4 * h + 1] = u.y;
            m.v[4 * h + 2] = u.z;
            m.v[4 * h + 3] = u.w;
        }
    }
    return m;
}

template <int NB>
__device__ inline void store_mv(float* p, const MV<NB>& m)
{
    if constexpr (NB == 2) {
        __builtin_nontemporal_store(vf2{m.v[0], m.v[1]}, reinterpret_cast<vf2*>(p));
    } else {
#pragma unroll
        for (int h = 0; h < NB / 4; ++h)
            __builtin_nontemporal_store(
                vf4{m.v[4 * h], m.v[4 * h + 1], m.v[4 * h + 2], m.v[4 * h + 3]},
                reinterpret_cast<vf4*>(p) + h);
    }
}

template <int NB>
__global__ __launch_bounds__(ACT_THREADS) void act_kernel(ActKArgs a)
{
    // (b, c) of this workgroup and its positions: act_geom.hpp
    const int64_t bc = act_bc(a, blockIdx.x);
    const int c = (int)(bc % a.C);
    float coef[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) coef[i] = gate_coef(a.act, gate_slot(a.act, i), c);

    const float* xb = a.x + act_base(a, bc, NB);
    float* yb = a.y + act_base(a, bc, NB);
    MV<NB> m[ACT_VPT];
#pragma unroll
    for (int v = 0; v < ACT_VPT; ++v) {
        const int64_t p = act_pos(a, blockIdx.x, bc, threadIdx.x, v);
        if (p < a.P) m[v] = load_mv<NB>(xb + p * NB);
    }
#pragma unroll
    for (int v = 0; v < ACT_VPT; ++v) {
        const int64_t p = act_pos(a, blockIdx.x, bc, threadIdx.x, v);
        if (p < a.P) {
            float part = 0.f;
#pragma unroll
            for (int i = 0; i < NB; ++i) part += coef[i] * m[v].v[i];
            const float g = gate_sigmoid(a.act, part, c);
#pragma unroll
            for (int i = 0; i < NB; ++i) m[v].v[i] *= g;
            store_mv<NB>(yb + p * NB, m[v]);
        }
    }
}

}  // namespace

cliff_status launch_act(int nb, int64_t B, int64_t C, int64_t P, const ActParams& act,
                        const float* x, float* y, hipStream_t stream)
{
    ActKArgs a;
    a.x = x;
    a.y = y;
    a.P = P;
    a.n_pblk = (P + ACT_THREADS * ACT_VPT - 1) / (ACT_THREADS * ACT_VPT);
    a.C = (int)C;
    a.act = act;
    const int64_t blocks = a.n_pblk * B * C;
    if (blocks >= (1ll << 31) || C >= (1ll << 31)) return CLIFF_EUNSUPPORTED;
    if (debug_enabled())
        fprintf(stderr, "cliffconv: multivector_act N_B=%d, %lld workgroups of %d\n", nb,
                (long long)blocks, ACT_THREADS);
    if (observe_launch(LAUNCH_ACT, {nb}, blocks, ACT_THREADS, 0, &a)) return CLIFF_OK;
    clear_hip_error();
    switch (nb) {
    case 2: hipLaunchKernelGGL(act_kernel<2>, dim3((unsigned)blocks), dim3(ACT_THREADS), 0, stream, a); break;
    case 4: hipLaunchKernelGGL(act_kernel<4>, dim3((unsigned)blocks), dim3(ACT_THREADS), 0, stream, a); break;
    case 8: hipLaunchKernelGGL(act_kernel<8>, dim3((unsigned)blocks), dim3(ACT_THREADS), 0, stream, a); break;
    default: return CLIFF_EUNSUPPORTED;
    }
    return hipGetLastError() == hipSuccess ? CLIFF_OK : CLIFF_EDEVICE;
}

}  // namespace cliff
