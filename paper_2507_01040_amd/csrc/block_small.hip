// Fused two-layer Clifford block for small problems: convolution (paper,
// Algorithm 1) + bias + multivector activation (Algorithm 3), twice, in one
// launch, with the intermediate multivectors kept in LDS.
//
// Small blocks (the paper's small-parameter regime: a few channels, images of
// tens of pixels) are bound by launch and memory latency, not by the matrix
// cores: two launches of the convolution kernel each pay a launch, an HBM
// round trip for their inputs and one for their outputs.  Here a workgroup
// owns one batch entry and a band of R final-output slices (rows for k = 2,
// planes for k = 3).  It stages the input slices the band needs (R + 2
// (d_filter - 1)) and both layers' raw filters in LDS, computes the
// intermediate slices (R + d_filter - 1, the halo recomputed by neighbouring
// bands) into LDS with the first layer's epilogue, then the band's outputs
// with the second layer's epilogue straight to HBM.
//
// MFMA mapping as in the large kernel (v_mfma_f32_16x16x4_f32): A = 16 rows
// (output channel, blade) x 4 input blades, the raw filter blade src(i, j)
// read from LDS and multiplied by the table's sign; B = 4 input blades x 16
// output positions.  Each wave owns whole 16 x 16 output tiles; a tile's K
// steps rotate over BS_ACC accumulators, so consecutive MFMAs are independent
// (a single dependent chain issues at a fraction of the pipe's rate), and the
// fragment reads of a slice's taps are all issued before its MFMAs.
#include <stdio.h>

#include <algorithm>

#include "block_small_geom.hpp"
#include "common.hpp"
#include "epilogue.hpp"

namespace cliff {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int BS_THREADS = 256;
constexpr int BS_ACC = 4;  // independent accumulator chains per wave

template <int KD, int NB, int DF>
__global__ __launch_bounds__(BS_THREADS) void block_small_kernel(BlockArgs a)
{
    constexpr int NH = NB / 4;    // K-groups of 4 input blades
    // taps of one input slice handled together: all of them when d_filter is
    // a compile-time constant, else BS_ACC at a time
    constexpr int UB = DF > 0 ? (KD == 3 ? DF * DF : DF) : BS_ACC;
    const int df = DF > 0 ? DF : a.df;
    const int taps = a.taps;
    extern __shared__ f4 smem4[];
    float* smem = reinterpret_cast<float*>(smem4);

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    constexpr int NWAVE = BS_THREADS / 64;
    // band, layer, lane and tile geometry: block_small_geom.hpp
    const BsBand g = bs_band(a, KD, df, blockIdx.x);

    // 1. Stage the input band ([C0][R0][S0][NB], slices s0.. of each channel
    //    are contiguous in HBM) and both layers' raw filters, by direct
    //    global->LDS loads: float4 e of each array goes to LDS float4 e of its
    //    area, so a wave's 64 loads fill 1 KB from the wave's first float4 on.
    //    All of them are issued before the one wait (a load-to-register loop
    //    waits for each load before the next).
    {
        const int wave_u = __builtin_amdgcn_readfirstlane(wave);
        auto dma = [&](const float* src, int lds_f4) {
            __builtin_amdgcn_global_load_lds(
                src, (__attribute__((address_space(3))) void*)(smem + 4 * lds_f4), 16, 0, 0);
        };
        const int nx = a.C0 * bs_band_f4(g, NB);
        for (int e0 = wave_u * 64; e0 < nx; e0 += BS_THREADS)
            if (e0 + lane < nx) dma(a.x + bs_band_src(a, g, NB, e0 + lane), e0);
        const int n1 = a.C0 * a.C1 * taps * NB / 4, n2 = a.C1 * a.C2 * taps * NB / 4;
        for (int e0 = wave_u * 64; e0 < n1; e0 += BS_THREADS)
            if (e0 + lane < n1) dma(a.w1 + 4 * (e0 + lane), a.lds_w1 / 4 + e0);
        for (int e0 = wave_u * 64; e0 < n2; e0 += BS_THREADS)
            if (e0 + lane < n2) dma(a.w2 + 4 * (e0 + lane), a.lds_w2 / 4 + e0);
        __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    __syncthreads();

    const BsLane ln = bs_lane(NB, lane);
    const int i0 = ln.i0;
    float sg[NH];
    int srcb[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
        sg[h] = sign_of(a.sign, ln.i_a * NB + 4 * h + ln.kk);
        srcb[h] = src_blade(NB, ln.i_a, 4 * h + ln.kk);
    }

    // One layer (BsLayer: input [Cin][Rin][Sin][NB] in LDS at `in`, filters
    // at `w`, Rout x Sout output positions of Cout channels); `store(co, m,
    // v)` writes one lane's 4 blades.
    auto layer = [&](const float* in, const float* w, const BsLayer& L, const float* bias,
                     const ActParams& act, auto store) {
        const int Cin = L.Cin, Cout = L.Cout;
        const int npos = L.Rout * L.Sout;
        const int T = bs_tiles(L, NB);
        const bool has_act = act.mode >= 0;
        int gslot[4] = {-1, -1, -1, -1};
        if (has_act) {
#pragma unroll
            for (int r = 0; r < 4; ++r) gslot[r] = gate_slot(act, i0 + r);
        }
        for (int t = wave; t < T; t += NWAVE) {  // wave-uniform tile loop
            const BsTile tl = bs_tile(L, KD, NB, taps, ln, t);
            // The epilogue's parameters, loaded before the MFMAs so that the
            // loads run during them.  The loads are unconditional (an absent
            // parameter reads the input's first floats instead, and the value
            // is not used): loads under a condition would be moved into the
            // epilogue, behind the last MFMA.
            const int co = tl.co;
            const bool cvalid = co < Cout;
            const int co_c = min(co, Cout - 1);
            const bool lin = act.mode == CLIFF_AGG_LINEAR;
            const f4 bias_v = *reinterpret_cast<const f4*>(bias ? bias + co_c * NB + i0 : a.x);
            float gw[4];
#pragma unroll
            for (int r2 = 0; r2 < 4; ++r2)
                gw[r2] = *(lin ? act.weight + (int64_t)co_c * act.K + max(gslot[r2], 0) : a.x);
            const float gb = *(lin ? act.bias + co_c : a.x);
            // BS_ACC partial sums over the K steps (independent MFMA chains),
            // added at the end
            f4 acc[BS_ACC];
#pragma unroll
            for (int q = 0; q < BS_ACC; ++q) acc[q] = f4{0.f, 0.f, 0.f, 0.f};
            const int nrt = KD == 3 ? df * df : df;  // taps per input slice
            for (int ci = 0; ci < Cin; ++ci) {
                const float* wc = w + bs_a_ci(L, tl, NB, taps, ci);
                const float* xc = in + bs_b_ci(L, tl, NB, ci);
#pragma unroll
                for (int qs = 0; qs < (DF > 0 ? DF : 1); ++qs) {
                    for (int qsr = 0; qsr < (DF > 0 ? 1 : df); ++qsr) {
                        const int qs_ = DF > 0 ? qs : qsr;
                        // UB taps of the slice at a time: all their fragment
                        // reads first, then their MFMAs
                        for (int u0 = 0; u0 < nrt; u0 += UB) {
                            float av[UB * NH], bv[UB * NH];
#pragma unroll
                            for (int q = 0; q < UB; ++q) {
                                const int u = u0 + q;
                                if (DF == 0 && u >= nrt) break;
                                const int qy = KD == 3 ? u / df : 0;
                                const int qx = KD == 3 ? u - qy * df : u;
                                const int tap = qs_ * nrt + u;
#pragma unroll
                                for (int h = 0; h < NH; ++h) {
                                    // (2D: whole offsets per read, measured 4-9 %
                                    // faster; 3D: the channel bases, 1-2 %)
                                    if constexpr (KD == 2) {
                                        av[q * NH + h] =
                                            w[bs_a_ofs(L, tl, NB, taps, ci, tap, srcb[h])] * sg[h];
                                        bv[q * NH + h] = in[bs_b_ofs(L, tl, NB, ci, qs_, qy, qx, h)];
                                    } else {
                                        av[q * NH + h] = wc[bs_a_tap(NB, tap, srcb[h])] * sg[h];
                                        bv[q * NH + h] = xc[bs_b_tap(L, NB, qs_, qy, qx, h)];
                                    }
                                }
                            }
#pragma unroll
                            for (int q = 0; q < UB * NH; ++q) {
                                if (DF == 0 && u0 + q / NH >= nrt) break;
                                acc[q % BS_ACC] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                    av[q], bv[q], acc[q % BS_ACC], 0, 0, 0);
                            }
                        }
                    }
                }
            }
            f4 v = acc[0];
#pragma unroll
            for (int q = 1; q < BS_ACC; ++q) v += acc[q];
            // epilogue: bias, activation (gate over the channel's N_B blades;
            // gate_coef's weights: the Linear gate's, 1 for Sum and Mean, 0
            // outside the subset)
            const int m = tl.m;
            if (cvalid && bias) v += bias_v;
            if (has_act) {
                float part = 0.f;
                if (cvalid) {
#pragma unroll
                    for (int r2 = 0; r2 < 4; ++r2)
                        part += (gslot[r2] < 0 ? 0.f : lin ? gw[r2] : 1.f) * v[r2];
                }
                if (NB == 8) part += __shfl_xor(part, 16);
                const float gate = cvalid ? gate_from_sum(act, part, gb) : 0.f;
                v *= gate;
            }
            if (cvalid && m < npos) store(co, m, v);
        }
    };

    // 2. First layer: input band -> intermediate band [C1][R1][S1][NB] in LDS.
    float* y1 = smem + a.lds_y1;
    layer(smem, smem + a.lds_w1, bs_layer1(a, g), a.b1, a.act1, [&](int co, int m, f4 v) {
        *reinterpret_cast<f4*>(y1 + bs_y1_ofs(g, NB, co, m, i0)) = v;
    });
    __syncthreads();
    // 3. Second layer: intermediate band -> output slices s0..s0+R2 in HBM.
    layer(y1, smem + a.lds_w2, bs_layer2(a, g), a.b2, a.act2, [&](int co, int m, f4 v) {
        *reinterpret_cast<f4*>(a.y + bs_y_ofs(a, g, NB, co, m, i0)) = v;
    });
}

}  // namespace

// LDS bytes the fused block needs with R final slices per workgroup.
int64_t block_small_lds_bytes(int k, int64_t C0, int64_t C1, int64_t C2, int64_t d_image,
                              int64_t d_filter, int64_t R)
{
    const int64_t nb = 1 << k;
    const int64_t D0 = d_image, D1 = D0 - d_filter + 1;
    int64_t S0 = 1, S1 = 1, taps = 1;
    for (int t = 0; t < k - 1; ++t) {
        S0 *= D0;
        S1 *= D1;
    }
    for (int t = 0; t < k; ++t) taps *= d_filter;
    const int64_t R1 = R + d_filter - 1, R0 = R1 + d_filter - 1;
    return 4 * nb * (C0 * R0 * S0 + C1 * R1 * S1 + (C0 * C1 + C1 * C2) * taps);
}

cliff_status launch_block_small(const BlockProblem& p, hipStream_t stream)
{
    if (p.k < 2 || p.k > 3) return CLIFF_EUNSUPPORTED;
    const int64_t nb = 1 << p.k;
    const int64_t D0 = p.d_image, df = p.d_filter, D1 = D0 - df + 1, D2 = D1 - df + 1;
    if (D2 < 1) return CLIFF_EUNSUPPORTED;
    // Band height: one slice while that leaves fewer than 1024 workgroups
    // (small problems need the parallelism more than they mind recomputing
    // the halo), else d_filter - 1 slices (the halo recomputation at most
    // doubles the first layer's work); lowered while the LDS does not fit.
    constexpr int64_t LDS_MAX = 160 * 1024;  // all of a CU's LDS: latency-bound problems
    int64_t R = p.B * D2 < 1024 ? 1 : std::max<int64_t>(1, std::min<int64_t>(df - 1, D2));
    while (R > 1 && block_small_lds_bytes(p.k, p.C_in, p.C_mid, p.C_out, D0, df, R) > LDS_MAX)
        --R;
    const int64_t lds = block_small_lds_bytes(p.k, p.C_in, p.C_mid, p.C_out, D0, df, R);
    const int64_t n_band = (D2 + R - 1) / R;
    const int64_t n_blk = p.B * n_band;
    if (lds > LDS_MAX || n_blk >= (1ll << 31) || p.C_in > 256 || p.C_mid > 256 ||
        p.C_out > 256)
        return CLIFF_EUNSUPPORTED;
    int64_t S0 = 1, S1 = 1, taps = 1;
    for (int t = 0; t < p.k - 1; ++t) {
        S0 *= D0;
        S1 *= D1;
    }
    for (int t = 0; t < p.k; ++t) taps *= df;
    BlockArgs a;
    a.x = p.x;
    a.w1 = p.w1;
    a.b1 = p.b1;
    a.w2 = p.w2;
    a.b2 = p.b2;
    a.y = p.y;
    a.C0 = (int)p.C_in;
    a.C1 = (int)p.C_mid;
    a.C2 = (int)p.C_out;
    a.D0 = (int)D0;
    a.D1 = (int)D1;
    a.D2 = (int)D2;
    a.df = (int)df;
    a.taps = (int)taps;
    a.R = (int)R;
    a.n_band = (int)n_band;
    const int64_t R1 = R + df - 1, R0 = R1 + df - 1;
    a.lds_y1 = (int)(p.C_in * R0 * S0 * nb);
    a.lds_w1 = (int)(a.lds_y1 + p.C_mid * R1 * S1 * nb);
    a.lds_w2 = (int)(a.lds_w1 + p.C_in * p.C_mid * taps * nb);
    a.sign = p.sign;
    a.act1 = p.act1;
    a.act2 = p.act2;
    if (debug_enabled())
        fprintf(stderr,
                "cliffconv: block_small k=%d bands of %lld slices, %lld workgroups of %d, "
                "%lld LDS bytes\n",
                p.k, (long long)R, (long long)n_blk, BS_THREADS, (long long)lds);
    if (observe_launch(LAUNCH_BLOCK_SMALL, {p.k, p.k == 2 ? 4 : 8, (int)df}, n_blk, BS_THREADS,
                       lds, &a))
        return CLIFF_OK;
    auto go = [&](auto kernel) {
        clear_hip_error();
        hipLaunchKernelGGL(kernel, dim3((unsigned)n_blk), dim3(BS_THREADS), (size_t)lds, stream,
                           a);
    };
    // the paper's block filters (3) and pointwise blocks get unrolled taps
    if (p.k == 2) {
        if (df == 3) go(block_small_kernel<2, 4, 3>);
        else if (df == 1) go(block_small_kernel<2, 4, 1>);
        else go(block_small_kernel<2, 4, 0>);
    } else {
        if (df == 3) go(block_small_kernel<3, 8, 3>);
        else if (df == 1) go(block_small_kernel<3, 8, 1>);
        else go(block_small_kernel<3, 8, 0>);
    }
    return hipGetLastError() == hipSuccess ? CLIFF_OK : CLIFF_EDEVICE;
}

}  // namespace cliff
