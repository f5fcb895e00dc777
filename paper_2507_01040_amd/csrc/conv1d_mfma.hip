// 1-D Clifford convolution (paper, Algorithm 1 with k = 1, N_B = 2) as an
// implicit GEMM on the fp32 matrix cores (v_mfma_f32_16x16x4_f32).
//
// With two blades per multivector, one MFMA K-group of 4 covers two input
// channels x two blades:
//   A (16x4): rows = 8 output channels x 2 blades (co, i); column k = (c, j)
//             with c = k / 2 the channel of the current pair and j = k % 2 the
//             input blade.  Lane (row, k) reads the raw filter blade src(i, j)
//             and applies the table's sign: the expanded Clifford kernel is
//             never stored.
//   B (4x16): the same (c, j) by 16 output positions.
//   D (16x16): a lane ends with the two blades of two consecutive output
//             channels at one position -> 8-byte stores, blade-last layout.
// Output positions are flattened over (batch entry, x), so short signals (the
// paper's 1-D layers have d_image = 60) still fill whole tiles.  A workgroup
// owns P consecutive flattened positions and CO_WG output channels.  Its input
// window is the contiguous run of (entry, x) positions from its first output
// position to its last one plus d_filter - 1, crossing entry boundaries; the
// positions of an entry past d_out are staged too (they are the last taps of
// that entry).  Per stage (a group of input channels, double-buffered in LDS)
// it stages each channel's window and raw filters with direct global->LDS
// loads: 16-byte ones where the layout allows (even C_out for the filters;
// even d_image as well for the windows, which then start at an even
// position), 4-byte ones otherwise, which need no alignment.
#include <stdio.h>

#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "conv1d_geom.hpp"
#include "epilogue.hpp"

#ifndef CLIFF_SGB_IL  // MFMAs between two of the next step's LDS reads; 0: reads clumped
#define CLIFF_SGB_IL 2
#endif
#ifndef CLIFF_LDS1  // LDS bytes per workgroup at most (two stage buffers)
#define CLIFF_LDS1 (64 * 1024)
#endif
#ifndef CLIFF_W1  // wide tile: WCO, WPOS, MW, NW, input slots
#define CLIFF_W1 2, 2, 4, 4, 8
#endif
#ifndef CLIFF_SHAPE_MODEL1  // quantisation model for the tile choice of large layers
#define CLIFF_SHAPE_MODEL1 1
#endif
#ifndef CLIFF_X16  // 16-byte input staging when d_image and C_out are even
#define CLIFF_X16 1
#endif
#ifndef CLIFF_W1_WAVES  // wide tile: waves per SIMD the registers are sized for
#define CLIFF_W1_WAVES 2   // (d_filter 17: 3, measured +2 %; d_filter 3: 2, 3 is -2 %)
#endif
#ifndef CLIFF_W1_WAVES17
#define CLIFF_W1_WAVES17 3
#endif

namespace cliff {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));


template <int DF, int WCO, int WPOS, int MW, int NW, int SIN, int SW, int WAVES, int FW, int FX,
          int WK>
__global__ __launch_bounds__(64 * WCO * WPOS * WK, WAVES) void conv1d_mfma_kernel(C1Args a)
{
    // WK > 1: WK waves share every output tile, each taking every WK-th
    // channel pair of a stage; their partial sums meet in LDS before the
    // epilogue
    constexpr int NB = 2;
    constexpr int NT = 64 * WCO * WPOS * WK;
    constexpr int CPT = 8;  // output channels per 16-row tile
    constexpr int CO_WG = WCO * MW * CPT;
    constexpr int P = WPOS * NW * 16;

    extern __shared__ f4 smem4[];
    float* smem = reinterpret_cast<float*>(smem4);
    constexpr C1Tile TL{DF, WCO, WPOS, MW, NW, SIN, SW, FW, FX, WK};

    // Block geometry, staging and fragment offsets: the shared address
    // arithmetic of conv1d_geom.hpp.
    const C1Block g = c1_block(TL, a, blockIdx.x);
    const int df = g.df;
    const int tid = threadIdx.x;
    const int m0 = g.m0, m_end = g.m_end, co0 = g.co0;
    const int span2 = a.span2;
    const int wch = g.wch;  // floats per channel of filters
    // 32-bit byte offsets of each slot's source from the stage's bases
    // (slots past a full stage's floats, a uniform test, load nothing)
    const int x_floats = a.cc * span2, w_floats = a.cc * wch;
    uint32_t xoffb[SIN], woffb[SW];
#pragma unroll
    for (int t = 0; t < SIN; ++t) {
        xoffb[t] = 0;
        if (t * NT * FX < x_floats) xoffb[t] = c1_xoffb(TL, a, g, (t * NT + tid) * FX);
    }
#pragma unroll
    for (int t = 0; t < SW; ++t) {
        woffb[t] = 0;
        if (t * NT * FW < w_floats) woffb[t] = c1_woffb(TL, a, g, (t * NT + tid) * FW);
    }
    const char* xbase = reinterpret_cast<const char*>(a.x + c1_x_base(a, g));
    const char* wbase = reinterpret_cast<const char*>(a.w + c1_w_base(g));
    const int wave_u = __builtin_amdgcn_readfirstlane(tid >> 6);
    auto stage_channels = [&](int s) { return c1_stage_channels(a, s); };
    auto load_stage = [&](int s, int buf) {
        const int nv = stage_channels(s);
        const char* xs = xbase + c1_stage_x(a, s) * 4;
        const char* ws = wbase + c1_stage_w(a, g, s) * 4;
#pragma unroll
        for (int t = 0; t < SIN; ++t) {
            if (t * NT * FX < x_floats && c1_x_loads(a, (t * NT + tid) * FX, nv)) {
                auto* dst = (__attribute__((address_space(3))) void*)(
                    smem + c1_lds_x(TL, a, buf, t, wave_u));
                const float* src = reinterpret_cast<const float*>(xs + xoffb[t]);
                if constexpr (FX == 4)
                    __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
                else
                    __builtin_amdgcn_global_load_lds(src, dst, 4, 0, 0);
            }
        }
#pragma unroll
        for (int t = 0; t < SW; ++t) {
            if (t * NT * FW < w_floats && c1_w_loads(TL, g, (t * NT + tid) * FW, woffb[t], nv)) {
                auto* dst = (__attribute__((address_space(3))) void*)(
                    smem + c1_lds_w(TL, a, g, buf, t, wave_u));
                // a float source pointer and literal sizes: with a char
                // pointer the host pass silently drops the 16-byte form's
                // kernel stub (undefined symbol at load time)
                const float* src = reinterpret_cast<const float*>(ws + woffb[t]);
                if constexpr (FW == 4)
                    __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
                else
                    __builtin_amdgcn_global_load_lds(src, dst, 4, 0, 0);
            }
        }
    };

    const C1Lane L = c1_lane(TL, tid);
    const int lane = L.lane, wk = L.wk, wrest = L.wrest, wco = L.wco, kk = L.kk;
    const int c_sub = L.c_sub;
    const float sg = c1_a_sign(a, L);
    const int wofs = c1_a_ofs(TL, g, L);
    int xoff[NW];
#pragma unroll
    for (int nw = 0; nw < NW; ++nw) xoff[nw] = c1_b_ofs(TL, a, g, L, nw);

    f4 acc[MW][NW];
#pragma unroll
    for (int mw = 0; mw < MW; ++mw)
#pragma unroll
        for (int nw = 0; nw < NW; ++nw) acc[mw][nw] = f4{0.f, 0.f, 0.f, 0.f};

    // One channel pair: all taps.  MASKED: the pair's second channel does not
    // exist (odd channel count in the stage); its LDS slot holds stale data,
    // which is selected away (never multiplied, so stale NaN/Inf cannot leak).
    auto pair = [&](const float* S0, int c_l, auto masked) {
        constexpr bool MASKED = decltype(masked)::value;
        const bool on = !MASKED || c_sub == 0;
        const float* S = S0 + c1_b_pair(a, c_l);
        const float* Sw = S0 + c1_a_pair(g, c_l);
        float ar[MW], br[NW];  // raw fragments of the next tap
        auto read = [&](int tap) {
#pragma unroll
            for (int mw = 0; mw < MW; ++mw) ar[mw] = Sw[c1_a_step(g, wofs, mw, tap)];
#pragma unroll
            for (int nw = 0; nw < NW; ++nw) br[nw] = S[xoff[nw] + tap * NB];
        };
        auto step = [&](int tap, bool prefetch) {
            float av[MW], bv[NW];
#pragma unroll
            for (int mw = 0; mw < MW; ++mw) av[mw] = ar[mw];
#pragma unroll
            for (int nw = 0; nw < NW; ++nw) bv[nw] = br[nw];
            if constexpr (DF > 0) {
                // software pipelining: the reads of tap + 1 are issued before
                // this tap's MFMAs (measured faster with the taps unrolled,
                // slower with a runtime tap loop)
                if (prefetch) read(tap + 1);
#if !CLIFF_SGB_IL
                __builtin_amdgcn_sched_barrier(0);
#endif
            }
#pragma unroll
            for (int mw = 0; mw < MW; ++mw) av[mw] = MASKED && !on ? 0.f : av[mw] * sg;
            if constexpr (MASKED) {
#pragma unroll
                for (int nw = 0; nw < NW; ++nw) bv[nw] = on ? bv[nw] : 0.f;
            }
#pragma unroll
            for (int mw = 0; mw < MW; ++mw)
#pragma unroll
                for (int nw = 0; nw < NW; ++nw)
                    acc[mw][nw] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mw], bv[nw],
                                                                        acc[mw][nw], 0, 0, 0);
            if constexpr (DF > 0) {
#if CLIFF_SGB_IL
                __builtin_amdgcn_sched_group_barrier(0x002, MW, 0);
#pragma unroll
                for (int r = 0; r < MW + NW; ++r) {
                    __builtin_amdgcn_sched_group_barrier(0x008, CLIFF_SGB_IL, 0);
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, MW * NW, 0);
#endif
                __builtin_amdgcn_sched_barrier(0);
            } else if (prefetch) {
                read(tap + 1);
            }
        };
        read(0);
        if constexpr (DF > 0) {
#pragma unroll
            for (int tap = 0; tap < DF; ++tap) step(tap, tap + 1 < DF);
        } else {
            for (int tap = 0; tap < df; ++tap) step(tap, tap + 1 < df);
        }
    };
    auto compute = [&](int buf, int nv) {
        const float* S0 = smem + buf * a.stage_floats;
        const int nfull = nv & ~1;
        for (int c_l = 2 * wk; c_l < nfull; c_l += 2 * WK) pair(S0, c_l, std::false_type{});
        if ((nv & 1) && (nfull / 2) % WK == wk) pair(S0, nfull, std::true_type{});
    };

    load_stage(0, 0);
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    for (int s = 0; s < a.n_stage; ++s) {
        // buffer (s+1)&1 was last read in iteration s-1, before its barrier
        if (s + 1 < a.n_stage) load_stage(s + 1, (s + 1) & 1);
        compute(s & 1, stage_channels(s));
        __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    }

    if constexpr (WK > 1) {
        // The stage loop ended with a barrier, so LDS is free: K slices
        // 1..WK-1 leave their partial sums there, slice 0 adds them and stores.
        if (wk > 0) {
#pragma unroll
            for (int mw = 0; mw < MW; ++mw)
#pragma unroll
                for (int nw = 0; nw < NW; ++nw)
                    smem4[c1_red_f4(TL, wk, wrest, mw, nw, lane)] = acc[mw][nw];
        }
        __syncthreads();
        if (wk > 0) return;  // wave-uniform: no barrier follows
#pragma unroll
        for (int k = 1; k < WK; ++k)
#pragma unroll
            for (int mw = 0; mw < MW; ++mw)
#pragma unroll
                for (int nw = 0; nw < NW; ++nw)
                    acc[mw][nw] += smem4[c1_red_f4(TL, k, wrest, mw, nw, lane)];
    }

    // Epilogue: lane row 4 kk + r is channel 2 kk + r / 2, blade r % 2.
    const bool has_act = a.act.mode >= 0;
    int gslot0 = -1, gslot1 = -1;
    if (has_act) {
        gslot0 = gate_slot(a.act, 0);
        gslot1 = gate_slot(a.act, 1);
    }
    int64_t ybase[NW];
    bool mvalid[NW];
#pragma unroll
    for (int nw = 0; nw < NW; ++nw) {
        const int m = c1_out_pos(TL, g, L, nw);
        mvalid[nw] = m < m_end;
        ybase[nw] = c1_out_base(a, m);
    }
#pragma unroll
    for (int mw = 0; mw < MW; ++mw) {
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int co = c1_out_channel(TL, g, L, mw, half);
            const bool cvalid = co < a.C_out;
            float bias0 = 0.f, bias1 = 0.f, cf0 = 0.f, cf1 = 0.f;
            if (cvalid && a.bias) {
                bias0 = a.bias[co * NB];
                bias1 = a.bias[co * NB + 1];
            }
            if (has_act && cvalid) {
                cf0 = gate_coef(a.act, gslot0, co);
                cf1 = gate_coef(a.act, gslot1, co);
            }
#pragma unroll
            for (int nw = 0; nw < NW; ++nw) {
                float v0 = acc[mw][nw][2 * half] + bias0;
                float v1 = acc[mw][nw][2 * half + 1] + bias1;
                if (has_act && cvalid) {
                    const float g = gate_sigmoid(a.act, cf0 * v0 + cf1 * v1, co);
                    v0 *= g;
                    v1 *= g;
                }
                if (cvalid && mvalid[nw]) {
                    float* yp = a.y + ybase[nw] + c1_out_chan(a, co);
                    *reinterpret_cast<float2*>(yp) = make_float2(v0, v1);
                }
            }
        }
    }
}

template <int DF, int WCO, int WPOS, int MW, int NW, int SIN, int SW, int WAVES, int FW, int FX,
          int WK>
cliff_status run1d(const ConvProblem& p, hipStream_t stream)
{
    constexpr int NB = 2;
    constexpr int NT = 64 * WCO * WPOS * WK;
    constexpr int CO_WG = WCO * MW * 8;
    constexpr int P = WPOS * NW * 16;
    const int64_t D = p.d_image, Do = p.d_out, df = p.d_filter;
    const int64_t M = p.B * Do;
    const int64_t n_pblk = (M + P - 1) / P;
    const int64_t n_co_blk = (p.C_out + CO_WG - 1) / CO_WG;
    const int64_t n_blk = n_pblk * n_co_blk;
    // P consecutive flattened positions touch at most rows_max batch entries
    const int64_t rows_max = std::min<int64_t>(p.B, (P + Do - 2) / Do + 1);
    // (FX = 4: one more position, the window starting at an even one, and a
    // whole number of 16-byte pieces per channel)
    if (FX == 4 && D % 2 != 0) return CLIFF_EUNSUPPORTED;
    const int64_t span_max = P + rows_max * (df - 1) + (FX == 4 ? 1 : 0);
    const int64_t span2 = FX == 4 ? (span_max * NB + 3) / 4 * 4 : span_max * NB;
    const int64_t ch_floats = span2 + CO_WG * df * NB;
    // LDS: two stage buffers per workgroup, WAVES waves per SIMD resident
    const int64_t wg_per_cu = std::max<int64_t>(1, 4 * WAVES / (WCO * WPOS * WK));
    const int64_t lds_budget = std::min<int64_t>(CLIFF_LDS1, 160 * 1024 / wg_per_cu);
    const int64_t mfma_per_pair = df * MW * NW;
    int64_t ccp = 2 * std::max<int64_t>(1, (512 + mfma_per_pair - 1) / mfma_per_pair);
    ccp = std::min<int64_t>(ccp, (lds_budget / (2 * ch_floats * 4)) & ~int64_t(1));
    ccp = std::min<int64_t>(ccp, ((int64_t)SIN * NT * FX / span2) & ~int64_t(1));
    ccp = std::min<int64_t>(ccp, ((int64_t)SW * NT * FW / (CO_WG * df * NB)) & ~int64_t(1));
    ccp = std::min<int64_t>(ccp, (p.C_in + 1) & ~int64_t(1));
    if (WK > 1 && ccp > 2 * WK) ccp -= ccp % (2 * WK);  // equal pair shares for the K slices
    if (ccp < 2 || M >= (1ll << 31) || n_blk >= (1ll << 31) ||
        rows_max * p.C_in * D * NB >= (1ll << 30) || ccp * p.C_out * df * NB >= (1ll << 30))
        return CLIFF_EUNSUPPORTED;
    const int64_t cc = std::min<int64_t>(ccp, p.C_in);
    const int64_t stage_floats = ccp * ch_floats;
    // the K split's partial sums reuse the stage buffers after the loop
    const int64_t red_bytes = (int64_t)(WK - 1) * WCO * WPOS * MW * NW * 64 * 16;
    const int64_t lds_bytes = std::max<int64_t>(2 * stage_floats * 4, red_bytes);

    C1Args a;
    a.x = p.x;
    a.w = p.w;
    a.bias = p.bias;
    a.y = p.y;
    a.C_in = (int)p.C_in;
    a.C_out = (int)p.C_out;
    a.D = (int)D;
    a.Do = (int)Do;
    a.df = (int)df;
    a.M = (int)M;
    a.n_co_blk = (int)n_co_blk;
    a.n_blk = (int)n_blk;
    a.cc = (int)cc;
    a.ccp = (int)ccp;
    a.n_stage = (int)((p.C_in + cc - 1) / cc);
    a.span2 = (int)span2;
    a.stage_floats = (int)stage_floats;
    a.sign = p.sign;
    a.act = p.act;
    if (debug_enabled())
        fprintf(stderr,
                "cliffconv: conv1d_mfma d_filter=%d tile %dx%d waves of %dx%d MFMA tiles "
                "(%d channels x %d positions), %lld workgroups, %d channels/stage, "
                "%lld LDS bytes, %d-byte input and %d-byte filter loads\n",
                (int)df, WCO, WPOS, MW, NW, CO_WG, P, (long long)n_blk, (int)cc,
                (long long)lds_bytes, 4 * FX, 4 * FW);
    if (observe_launch(LAUNCH_CONV1D_MFMA, {DF, WCO, WPOS, MW, NW, SIN, SW, WAVES, FW, FX, WK}, n_blk,
                       NT, lds_bytes, &a))
        return CLIFF_OK;
    clear_hip_error();
    hipLaunchKernelGGL((conv1d_mfma_kernel<DF, WCO, WPOS, MW, NW, SIN, SW, WAVES, FW, FX, WK>),
                       dim3((unsigned)n_blk), dim3(NT), (size_t)lds_bytes, stream, a);
    return hipGetLastError() == hipSuccess ? CLIFF_OK : CLIFF_EDEVICE;
}

// 16-byte filter loads (fewer slots) when C_out is even, and then also
// 16-byte input loads when d_image is even; 4-byte loads otherwise.
// (FW1: the shape has a 4-byte filter form at all)
template <int DF, int WCO, int WPOS, int MW, int NW, int SIN, int SW1, int SW4, int WAVES,
          int WK = 1, bool FW1 = true>
cliff_status run1d_fw(const ConvProblem& p, hipStream_t stream)
{
    constexpr int SIN4 = (SIN + 3) / 4 + 1;  // 16-byte input slots (one more position)
    if (p.C_out % 2 == 0 && p.d_image % 2 == 0 && CLIFF_X16)
        return run1d<DF, WCO, WPOS, MW, NW, SIN4, SW4, WAVES, 4, 4, WK>(p, stream);
    if (p.C_out % 2 == 0)
        return run1d<DF, WCO, WPOS, MW, NW, SIN, SW4, WAVES, 4, 1, WK>(p, stream);
    // (the 4-byte filter slots need more registers: at most 2 waves per SIMD)
    if constexpr (FW1)
        return run1d<DF, WCO, WPOS, MW, NW, SIN, SW1, (WAVES < 2 ? WAVES : 2), 1, 1, WK>(p,
                                                                                       stream);
    return CLIFF_EUNSUPPORTED;
}

// Tile shapes (waves along channels x waves along positions, MFMA tiles per
// wave along channels x along positions):
//   wide   2x2 waves of 4x4 tiles: 64 channels x 128 positions (d_filter 17:
//          also 4x1 waves of 2x11 tiles, 64 channels x 176 positions, where
//          its blocks fill the last round of CUs better)
//   medium 2x1 waves of 4x2 tiles: 64 channels x  32 positions
//   narrow 1x4 waves of 1x4 tiles:  8 channels x 256 positions
//   tiny   1x2 tiles:                8 channels x  32 positions (long K loops
//          split over 4 waves)
template <int DF>
cliff_status run1d_shape(const ConvProblem& p, hipStream_t stream)
{
    // <DF, WCO, WPOS, MW, NW, input slots, filter slots with 4-byte and with
    // 16-byte loads, waves per SIMD>
    auto wide = [&] {
        return run1d_fw<DF, CLIFF_W1, 18, 6, DF == 17 ? CLIFF_W1_WAVES17 : CLIFF_W1_WAVES>(p, stream);
    };
    // the 176-position form: 4x1 waves of 2x11 tiles, 2 waves per SIMD (at
    // 3 it spills registers, and so do its 4-byte filter slots: even C_out
    // only)
    auto wide176 = [&] {
        if constexpr (DF == 17) return run1d_fw<DF, 4, 1, 2, 11, 8, 18, 6, 2, 1, false>(p, stream);
        return CLIFF_EUNSUPPORTED;
    };
    auto medium = [&] { return run1d_fw<DF, 2, 1, 4, 2, 8, 18, 9, 2>(p, stream); };
    auto narrow = [&] { return run1d_fw<DF, 1, 4, 1, 4, 16, 4, 2, 2>(p, stream); };
    // the tiny tile splits its K loop over 4 waves when that loop is long and
    // the workgroups are few (measured 1.5-1.8x faster there; with 2816
    // workgroups, or only 12 K steps, one wave per tile is 7-20 % faster)
    auto tiny = [&] {
        const int64_t tiles = ((p.B * p.d_out + 31) / 32) * ((p.C_out + 7) / 8);
        const int64_t ksteps = (p.C_in + 1) / 2 * p.d_filter;
        if (tiles < 1024 && ksteps >= 32)
            return run1d_fw<DF, 1, 1, 1, 2, 12, 12, 4, 4, 4>(p, stream);
        return run1d_fw<DF, 1, 1, 1, 2, 12, 12, 4, 4, 1>(p, stream);
    };
    const int64_t M = p.B * p.d_out;
    auto blocks = [&](int64_t co_wg, int64_t pos) {
        return ((M + pos - 1) / pos) * ((p.C_out + co_wg - 1) / co_wg);
    };
    // Layers of >= 1 GFLOP: the quantisation model of the 2D/3D kernel (a
    // shape's N blocks take ceil(N / CUs) rounds of whole blocks; rate
    // b * N / (rounds * CUs) * channel utilisation), fitted to forced-shape
    // timings of 10 1-D layers on MI355X: b = 0.90 (wide), 0.80 (narrow),
    // 0.68 (tiny).  Smaller layers keep the latency rule below.
    const double useful = 2.0 * M * p.C_out * 2 * p.C_in * 2 * p.d_filter;
    const int cus = device_cus();
    const bool model = CLIFF_SHAPE_MODEL1 && useful >= 1e9 && cus > 0;
    auto est = [&](int64_t co_wg, int64_t pos, double b) {
        const int64_t n = blocks(co_wg, pos);
        const int64_t rounds = (n + cus - 1) / cus;
        const double u = (double)p.C_out / (double)(((p.C_out + co_wg - 1) / co_wg) * co_wg);
        return b * (double)n / (double)(rounds * cus) * u;
    };
    // the wide tile's width: 176 positions where the model rates it higher
    // (b = 0.89 against 0.90, fitted like the others)
    auto wide_best = [&] {
        cliff_status s = CLIFF_EUNSUPPORTED;
        if (model && DF == 17 && est(64, 176, 0.89) > est(64, 128, 0.90)) s = wide176();
        if (s == CLIFF_EUNSUPPORTED) s = wide();
        return s;
    };
    switch (p.mfma_shape) {
    case 0: return wide_best();
    case 1: return medium();
    case 2: return narrow();
    case 3: return tiny();
    default: break;
    }
    if (model) {
        const double ew =
            p.C_out > 32 ? std::max(est(64, 128, 0.90), DF == 17 ? est(64, 176, 0.89) : 0.0)
                         : 0.0;
        const double en = est(8, 256, 0.80), et = est(8, 32, 0.68);
        cliff_status s = CLIFF_EUNSUPPORTED;
        if (ew >= en && ew >= et) s = wide_best();
        if (s == CLIFF_EUNSUPPORTED && en >= et) s = narrow();
        if (s == CLIFF_EUNSUPPORTED) s = tiny();
        if (s == CLIFF_EUNSUPPORTED) s = narrow();
        return s;
    }
    cliff_status s = CLIFF_EUNSUPPORTED;
    if (p.C_out > 32 && blocks(64, 128) >= 256) s = wide();
    if (s == CLIFF_EUNSUPPORTED) s = tiny();
    if (s == CLIFF_EUNSUPPORTED) s = narrow();
    return s;
}

}  // namespace

cliff_status launch_conv1d_mfma(const ConvProblem& p, hipStream_t stream)
{
    if (p.k != 1) return CLIFF_EUNSUPPORTED;
    // the filter lengths of the paper's layers get unrolled tap loops
    if (p.d_filter == 3) return run1d_shape<3>(p, stream);
    if (p.d_filter == 17) return run1d_shape<17>(p, stream);
    return run1d_shape<0>(p, stream);
}

}  // namespace cliff
