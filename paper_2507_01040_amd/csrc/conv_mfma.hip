// k-D Clifford convolution (paper, Algorithm 1) as an implicit GEMM on the
// CDNA4 fp32 matrix cores (v_mfma_f32_16x16x4_f32), k = 2 and 3.
//
// GEMM view.  With the blades folded into the channels the layer is a dense
// contraction
//     Y[(co, i), m] = sum_{q, ci, j} E[(co, i), (q, ci, j)] * X[(q, ci, j), m]
// with m an output position (b, p), X[(q, ci, j), m] = input[b, ci, p + q, j]
// and E the Clifford kernel expansion E[(co,i),(q,ci,j)] =
// s[i][j] * filters[ci, co, q, src(i, j)] (the paper's "Baseline" builds E in
// memory, with N_B-fold duplication; here it is never materialised: every
// lane of an MFMA A-fragment owns one fixed (i, j) pair, so it reads the raw
// filter blade src(i, j) from LDS and applies its sign in a register).
//
// MFMA roles.  A (16x4) = E rows (4 output channels x 4 blades for N_B = 4,
// 2 x 8 for N_B = 8) by 4 input blades j; B (4x16) = 4 input blades by 16
// consecutive output positions; D (16x16) leaves every lane with 4
// consecutive output blades of one (channel, position), so results go to HBM
// as 16-byte stores in the blade-last layout and the activation gate needs
// at most one cross-lane exchange.
//
// Work decomposition.  The flattened output positions m in [0, B d_out^k)
// are cut into blocks of P consecutive positions (they may span rows, planes
// and batch entries); a workgroup computes P positions x CO_WG output
// channels.  2D images may instead use row-aligned blocks (at most P
// positions of one output row, staging only the d_filter input rows and the
// columns they read): where whole-row slabs do not fit, and on the wide
// tiles where a row's blocks leave at most 2 % of their positions idle.  The K loop runs over "stages": cc input channels (2D) or cc
// input channels of one filter plane qz (3D); the host picks cc so a stage
// holds enough MFMAs per barrier.  For each stage and channel the workgroup
// stages in LDS (double-buffered, direct global->LDS loads):
//   * the slab: every input row the block's outputs touch for this stage,
//     rows of d_image multivectors, kept blade-packed ([row][x][4] for N_B = 4,
//     [row][half][x][4] for N_B = 8 so that a fragment read is 64 consecutive
//     words);
//   * the raw filters [co][tap][blade] of this stage (no expansion).
// The smallest tile splits its K loop over several waves of the workgroup
// (WK), whose partial sums meet in LDS before the epilogue.
#include <stdio.h>

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "common.hpp"
#include "conv_mfma_geom.hpp"
#include "epilogue.hpp"

#ifndef CLIFF_SGB_IL  // MFMAs between two of the next step's LDS reads; 0: reads clumped
#define CLIFF_SGB_IL 2
#endif

#ifndef CLIFF_PRO_SB  // scheduling barrier after a channel's prologue reads
#define CLIFF_PRO_SB 1
#endif

#ifndef CLIFF_W2_WIDTH_MODEL  // 2D 64-channel tile: 128 or 96 positions by the quantisation model
#define CLIFF_W2_WIDTH_MODEL 1
#endif

#ifndef CLIFF_ROWBLK  // 2D row-aligned blocks: 1 when no shape fits whole-row slabs, 2 always
#define CLIFF_ROWBLK 1
#endif
#ifndef CLIFF_SHAPE_MODEL  // quantisation model for the tile choice of large problems
#define CLIFF_SHAPE_MODEL 1
#endif
#ifndef CLIFF_CONV_NEG  // negated filter copy in LDS instead of sign multiplies (wide 3x3(x3) tiles)
#define CLIFF_CONV_NEG 1
#endif
#ifndef CLIFF_CONV_NEG2D  // ... also for the 2D tiles
#define CLIFF_CONV_NEG2D 0
#endif
namespace cliff {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));


template <int KD, int NB, int DF, int CCT, int WCO, int WPOS, int MW, int NW, int SLOTS,
          int WAVES_PER_SIMD, int WK, bool NEG>
__global__ __launch_bounds__(64 * WCO * WPOS * WK, WAVES_PER_SIMD) void conv_mfma_kernel(
    MfmaArgs a)
{
    // WK > 1: WK waves share every output tile, each taking every WK-th input
    // channel of a stage; their partial sums meet in LDS before the epilogue
    static_assert(WK == 1 || CCT != 1, "a K split needs several channels per stage");
    // NEG: negated filter copy in LDS instead of sign multiplies; one channel
    // per stage, unrolled taps
    static_assert(!NEG || (CCT == 1 && DF > 0 && WK == 1), "the negated copy needs CCT = 1");
    constexpr int NT = 64 * WCO * WPOS * WK;
    constexpr int CPT = 16 / NB;  // output channels per 16-row tile
    constexpr int CO_WG = WCO * MW * CPT;
    constexpr int P = WPOS * NW * 16;
    constexpr int NH = NB / 4;  // groups of 4 input blades (MFMA K = 4)

    extern __shared__ f4 smem4[];
    float* smem = reinterpret_cast<float*>(smem4);
    constexpr MfmaTile TL{KD, NB, DF, CCT, WCO, WPOS, MW, NW, SLOTS, WK, NEG};
    constexpr int FS = TL.fslots();  // NEG: filter float4 per lane and stage

    // Block geometry, staging offsets and fragment offsets: the shared
    // address arithmetic of conv_mfma_geom.hpp.
    const MfmaBlock g = mfma_block(TL, a, blockIdx.x);
    const int tid = threadIdx.x;
    const int df = g.df;
    const int D = g.D;
    const int cc = g.cc;
    const int slab_f4 = g.slab_f4;
    const int wch_f4 = g.wch_f4;
    const int lrow_floats = g.lrow_floats;
    const int m0 = g.m0, m_end = g.m_end;
    int goff[SLOTS];
#pragma unroll
    for (int t = 0; t < SLOTS; ++t) {
        // slots past the block's staged float4 (a uniform test) load nothing
        goff[t] = 0;
        if (t * NT < g.total_f4) goff[t] = mfma_slot_goff(TL, a, g, t * NT + tid);
    }

    const float* xbase = a.x + mfma_x_base(TL, a, g);
    const float* wbase = a.w + mfma_w_base(TL, g);
    const int wave_u = __builtin_amdgcn_readfirstlane(tid >> 6);
    auto stage_channels = [&](int s, int& ci0, int& qz) {
        return mfma_stage_channels(TL, a, g, s, ci0, qz);
    };
    auto load_stage = [&](int s, int buf) {
        int ci0, qz;
        const int nv = stage_channels(s, ci0, qz);
        const float* xs = xbase + mfma_stage_x(g, ci0, qz);
        const float* ws = wbase + mfma_stage_w(TL, g, ci0, qz);
        float* lbase = smem + mfma_lds_wave(a, buf, wave_u);
#pragma unroll
        for (int t = 0; t < SLOTS; ++t) {
            if (t * NT < g.total_f4 && mfma_slot_loads(TL, g, t * NT + tid, goff[t], nv)) {
                const float* src = goff[t] >= 0 ? xs + goff[t] : ws + (-1 - goff[t]);
                __builtin_amdgcn_global_load_lds(
                    src, (__attribute__((address_space(3))) void*)(lbase + mfma_lds_slot(TL, t)),
                    16, 0, 0);
            }
        }
    };

    // NEG: the stage's filters also go through registers (global loads
    // issued with the stage's direct loads, before its predecessor is
    // multiplied), then to LDS negated, after the wait that ends the
    // predecessor (the buffer was last read before the previous barrier).
    f4 wreg[FS > 0 ? FS : 1];
    int wsrc[FS > 0 ? FS : 1];
#pragma unroll
    for (int u = 0; u < FS; ++u) {
        const int e = u * NT + tid;
        wsrc[u] = e < cc * wch_f4 ? mfma_filter_src(TL, a, g, e) : 0;
    }
    auto load_filters = [&](int s) {
        int ci0, qz;
        stage_channels(s, ci0, qz);
        const float* ws = wbase + mfma_stage_w(TL, g, ci0, qz);
#pragma unroll
        for (int u = 0; u < FS; ++u)
            if (u * NT + tid < cc * wch_f4) wreg[u] = *reinterpret_cast<const f4*>(ws + wsrc[u]);
    };
    auto store_filters = [&](int buf) {
        float* lw = smem + buf * a.stage_floats;
#pragma unroll
        for (int u = 0; u < FS; ++u) {
            const int e = u * NT + tid;
            if (e < cc * wch_f4) *reinterpret_cast<f4*>(lw + mfma_wreg_lds(g, e, 1)) = -wreg[u];
        }
    };

    // Per-lane constants of the MFMA fragments.
    const MfmaLane L = mfma_lane(TL, tid);
    const int lane = L.lane, wk = L.wk, wrest = L.wrest, wco = L.wco, mrow = L.mrow;
    int wofs[NH];
    float sg[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
        sg[h] = mfma_a_sign(TL, a, L, h);
        wofs[h] = mfma_a_ofs(TL, a, g, L, h);
    }
    int xoff[NW];
#pragma unroll
    for (int nw = 0; nw < NW; ++nw) xoff[nw] = mfma_b_ofs(TL, g, L, nw);

    f4 acc[MW][NW];
#pragma unroll
    for (int mw = 0; mw < MW; ++mw)
#pragma unroll
        for (int nw = 0; nw < NW; ++nw) acc[mw][nw] = f4{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](int buf, int nv) {
      if constexpr (DF > 0) {
        // Software-pipelined over the whole stage: the raw fragments of the
        // next step (tap, blade group; after a channel's last step, the next
        // channel's first) are read from LDS while this step's MFMAs issue,
        // one read after every CLIFF_SGB_IL MFMAs (scheduling-group
        // barriers), so the matrix pipe never waits behind a clump of reads
        // and no read sits next to its consumer (measured +1.3-1.9 % for
        // reads issued ahead of the MFMAs, a further +1-2 % for spreading
        // them).  With d_filter = 1 (a step or two per channel) the pipeline
        // also crosses channels, which then go in pairs so that the fragment
        // buffer of every step is known at compile time; with 3x3(x3) filters
        // it restarts per channel (crossing measured no faster there, and it
        // costs registers).
        constexpr int T = DF * DF * NH;
        constexpr bool XCH = DF == 1;
        // Prefetch distance in steps: the tiny tile has only 2 MFMAs (64
        // cycles) per step, less than the LDS latency, so it reads 3 steps
        // ahead; the others 1.
        constexpr int PF = !XCH && MW * NW <= 2 ? 3 : 1;
        constexpr int RB = PF + 1;  // fragment buffers in the ring
        const int ncl = CCT > 0 ? CCT : nv;
        const float* S0 = smem + buf * a.stage_floats;
        float fa[RB][MW], fb[RB][NW];
        // (the step offsets take the block's strides as plain values: read
        // through the block struct inside this lambda, LLVM kept extra
        // address registers live in the loop, measured 1-3.6 % slower)
        auto ld = [&](int c, int u, float(&A)[MW], float(&Bv)[NW]) {
            const float* S = S0 + mfma_b_chan(slab_f4, c);
            const float* Sw = S0 + mfma_a_chan(wch_f4, c);
            const int h = u % NH, tap = u / NH, qy = tap / DF, qx = tap % DF;
#pragma unroll
            for (int mw = 0; mw < MW; ++mw) A[mw] = Sw[mfma_a_tap(TL, DF * DF, wofs[h], mw, tap)];
#pragma unroll
            for (int nw = 0; nw < NW; ++nw)
                Bv[nw] = S[mfma_b_tap(lrow_floats, D, xoff[nw], h, qy, qx)];
        };
        auto chan = [&](int c, auto base_c) {
            constexpr int BASE = decltype(base_c)::value;  // buffer of step 0
#pragma unroll
            for (int u = 0; u < T; ++u) {
                const int cur = (BASE + u) % RB;
                const int nxt = (BASE + u + PF) % RB;
                if (u + PF < T)
                    ld(c, u + PF, fa[nxt], fb[nxt]);
                else if (XCH && c + WK < ncl)
                    ld(c + WK, 0, fa[nxt], fb[nxt]);
#if !CLIFF_SGB_IL
                // keep the next step's reads ahead of this step's MFMAs
                __builtin_amdgcn_sched_barrier(0);
#endif
                float as[MW];
#pragma unroll
                for (int mw = 0; mw < MW; ++mw) as[mw] = NEG ? fa[cur][mw] : fa[cur][mw] * sg[u % NH];
#pragma unroll
                for (int mw = 0; mw < MW; ++mw)
#pragma unroll
                    for (int nw = 0; nw < NW; ++nw)
                        acc[mw][nw] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                            as[mw], fb[cur][nw], acc[mw][nw], 0, 0, 0);
#if CLIFF_SGB_IL
                // the sign multiplies first, then the next step's LDS reads
                // spread between this step's MFMAs
                if (!NEG) __builtin_amdgcn_sched_group_barrier(0x002, MW, 0);
#pragma unroll
                for (int r = 0; r < MW + NW; ++r) {
                    __builtin_amdgcn_sched_group_barrier(0x008, CLIFF_SGB_IL, 0);
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, MW * NW, 0);
#endif
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        auto prologue = [&](int c) {  // the first PF steps of channel c
#pragma unroll
            for (int u = 0; u < PF; ++u)
                if (u < T) ld(c, u, fa[u], fb[u]);
#if CLIFF_PRO_SB
            // issue the prologue's reads together, ahead of the first step
            // (else they are spread between the first step's own MFMAs, each
            // of which then waits for its read)
            __builtin_amdgcn_sched_barrier(0);
#endif
        };
        if constexpr (CCT == 1) {
            prologue(0);
            chan(0, std::integral_constant<int, 0>{});
        } else if constexpr (XCH) {
            // this wave's channels wk, wk + WK, ...
            if (wk < ncl) prologue(wk);
            for (int c = wk; c < ncl; c += 2 * WK) {
                chan(c, std::integral_constant<int, 0>{});
                if (c + WK < ncl) chan(c + WK, std::integral_constant<int, T & 1>{});
            }
        } else {
            for (int c = wk; c < ncl; c += WK) {
                prologue(c);
                chan(c, std::integral_constant<int, 0>{});
            }
        }
      } else {
      for (int c_l = wk; c_l < (CCT > 0 ? CCT : nv); c_l += WK) {
        const float* S = smem + buf * a.stage_floats + mfma_b_chan(slab_f4, c_l);
        const float* Sw = smem + buf * a.stage_floats + mfma_a_chan(wch_f4, c_l);
#pragma unroll
        for (int qy = 0; qy < (DF > 0 ? DF : 1); ++qy) {
            for (int qyr = 0; qyr < (DF > 0 ? 1 : df); ++qyr) {
                const int qy_ = DF > 0 ? qy : qyr;
#pragma unroll
                for (int qx = 0; qx < (DF > 0 ? DF : 1); ++qx) {
                    for (int qxr = 0; qxr < (DF > 0 ? 1 : df); ++qxr) {
                        const int qx_ = DF > 0 ? qx : qxr;
                        const int tap = qy_ * df + qx_;
#pragma unroll
                        for (int h = 0; h < NH; ++h) {
                            float av[MW], bv[NW];
#pragma unroll
                            for (int mw = 0; mw < MW; ++mw)
                                av[mw] = Sw[mfma_a_tap(TL, df * df, wofs[h], mw, tap)] * sg[h];
#pragma unroll
                            for (int nw = 0; nw < NW; ++nw)
                                bv[nw] = S[mfma_b_tap(lrow_floats, D, xoff[nw], h, qy_, qx_)];
#pragma unroll
                            for (int mw = 0; mw < MW; ++mw)
#pragma unroll
                                for (int nw = 0; nw < NW; ++nw)
                                    acc[mw][nw] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                        av[mw], bv[nw], acc[mw][nw], 0, 0, 0);
                        }
                    }
                }
            }
        }
      }
      }
    };

    // D fragment: lane holds output channel co and blades i0..i0+3 of one
    // position; gslot[r] is blade i0 + r's place in the gate's blade list.
    const int i0 = mfma_out_blade0(TL, L);
    const bool has_act = a.act.mode >= 0;
    const bool lin = a.act.mode == CLIFF_AGG_LINEAR;
    // Tiles with a split K loop (the smallest problems, bound by latency)
    // load the epilogue's parameters before the main loop, unconditionally
    // (an absent parameter reads the input's first floats, unused), so that
    // the loads run under the MFMAs: issued after the loop, each round trip
    // would follow the last MFMA, and under a condition the compiler moves
    // them there.  The other tiles load them in the epilogue, where their
    // registers are free.
    constexpr bool EARLY = WK > 1;
    constexpr int ME = EARLY ? MW : 1;
    int gslot[4] = {-1, -1, -1, -1};
    f4 ebb[ME];
    float ecf[ME][4], egb[ME];
    if constexpr (EARLY) {
        if (has_act) {
#pragma unroll
            for (int r = 0; r < 4; ++r) gslot[r] = gate_slot(a.act, i0 + r);
        }
#pragma unroll
        for (int mw = 0; mw < MW; ++mw) {
            const int co_c = min(mfma_out_channel(TL, g, L, mw), a.C_out - 1);
            ebb[mw] = *reinterpret_cast<const f4*>(a.bias ? a.bias + co_c * NB + i0 : a.x);
#pragma unroll
            for (int r = 0; r < 4; ++r)
                ecf[mw][r] = *(lin ? a.act.weight + (int64_t)co_c * a.act.K + max(gslot[r], 0)
                                   : a.x);
            egb[mw] = *(lin ? a.act.bias + co_c : a.x);
        }
    }

    // Main loop: one barrier per stage; the next stage's global loads are in
    // flight while the current one is multiplied.
    load_stage(0, 0);
    if constexpr (NEG) load_filters(0);
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    if constexpr (NEG) store_filters(0);
    __syncthreads();
    for (int s = 0; s < a.n_stage; ++s) {
        // buffer (s+1)&1 was last read in iteration s-1, before the barrier
        if (s + 1 < a.n_stage) {
            load_stage(s + 1, (s + 1) & 1);
            if constexpr (NEG) load_filters(s + 1);
        }
        int ci0, qz;
        compute(s & 1, stage_channels(s, ci0, qz));
        __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
        if constexpr (NEG)
            if (s + 1 < a.n_stage) store_filters((s + 1) & 1);
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
                    smem4[mfma_red_f4(TL, wk, wrest, mw, nw, lane)] = acc[mw][nw];
        }
        __syncthreads();
        if (wk > 0) return;  // wave-uniform: no barrier follows
#pragma unroll
        for (int k = 1; k < WK; ++k)
#pragma unroll
            for (int mw = 0; mw < MW; ++mw)
#pragma unroll
                for (int nw = 0; nw < NW; ++nw)
                    acc[mw][nw] += smem4[mfma_red_f4(TL, k, wrest, mw, nw, lane)];
    }

    // Epilogue: bias, optional multivector activation, 16-byte stores.
    if constexpr (!EARLY) {
        if (has_act) {
#pragma unroll
            for (int r = 0; r < 4; ++r) gslot[r] = gate_slot(a.act, i0 + r);
        }
    }
#pragma unroll
    for (int mw = 0; mw < MW; ++mw) {
        const int co = mfma_out_channel(TL, g, L, mw);
        const bool cvalid = co < a.C_out;
        f4 bb = f4{0.f, 0.f, 0.f, 0.f};
        float cf[4] = {0.f, 0.f, 0.f, 0.f};
        if constexpr (EARLY) {
            // gate_coef's weights from the loaded values
            if (cvalid && a.bias) bb = ebb[mw];
            if (has_act && cvalid) {
#pragma unroll
                for (int r = 0; r < 4; ++r) cf[r] = gslot[r] < 0 ? 0.f : lin ? ecf[mw][r] : 1.f;
            }
        } else {
            if (cvalid && a.bias) bb = *reinterpret_cast<const f4*>(a.bias + co * NB + i0);
            if (has_act && cvalid) {
#pragma unroll
                for (int r = 0; r < 4; ++r) cf[r] = gate_coef(a.act, gslot[r], co);
            }
        }
#pragma unroll
        for (int nw = 0; nw < NW; ++nw) {
            const int m = mfma_out_pos(TL, g, L, nw);
            f4 v = acc[mw][nw] + bb;
            if (has_act) {
                float part = cf[0] * v[0] + cf[1] * v[1] + cf[2] * v[2] + cf[3] * v[3];
                if (NB == 8) part += __shfl_xor(part, 16);
                float gate = 0.f;
                if (cvalid)
                    gate = EARLY ? gate_from_sum(a.act, part, egb[mw]) : gate_sigmoid(a.act, part, co);
                v *= gate;
            }
            if (cvalid && m < m_end)
                *reinterpret_cast<f4*>(a.y + mfma_out_ofs(TL, a, m, co, i0)) = v;
        }
    }
}

struct TileCfg {
    int wco, wpos, mw, nw;
};

template <int KD, int NB, int DF, int CCT, int WCO, int WPOS, int MW, int NW, int SLOTS,
          int WAVES, int WK, int LDSKB, bool NEG>
cliff_status run(const ConvProblem& p, hipStream_t stream)
{
    constexpr int NT = 64 * WCO * WPOS * WK;
    constexpr int CPT = 16 / NB;
    constexpr int CO_WG = WCO * MW * CPT;
    constexpr int P = WPOS * NW * 16;
    const int64_t D = p.d_image, Do = p.d_out, df = p.d_filter;
    int64_t npos = 1;
    for (int t = 0; t < KD; ++t) npos *= Do;
    const int64_t M = p.B * npos;
    int64_t n_pos_blk = (M + P - 1) / P;
    const int64_t n_co_blk = (p.C_out + CO_WG - 1) / CO_WG;
    // 32-bit position indices; one d_image^2 plane of floats in 32 bits
    if (M >= (1ll << 31) || D * D * NB >= (1ll << 31)) return CLIFF_EUNSUPPORTED;
    // Upper bound of the slab rows of any block.
    const int64_t total_rows = M / Do;
    const int64_t R = std::min<int64_t>((P - 1) / Do + 2, total_rows);
    const int64_t planes = std::min<int64_t>(R, (R - 1) / Do + 2);
    const int64_t rows_max = R + planes * (df - 1);
    // per channel: LDS floats (slab, filters, NEG: negated filters) and the
    // floats staged by direct loads (slab, filters)
    const int64_t wch = CO_WG * df * df * NB;
    int64_t ch_floats = rows_max * D * NB + (NEG ? 2 : 1) * wch;
    int64_t ch_dma = rows_max * D * NB + wch;
    // Channels per stage: enough MFMAs per wave between barriers, within the
    // LDS budget (two buffers) and the staging slots.
    constexpr int64_t LDS_BUDGET = LDSKB * 1024;
    constexpr int64_t MFMA_PER_STAGE = 512;
    const int64_t mfma_per_ch = df * df * (NB / 4) * MW * NW;
    auto channels = [&](int64_t chf, int64_t chd) {
        int64_t c = std::min<int64_t>(p.C_in, (MFMA_PER_STAGE + mfma_per_ch - 1) / mfma_per_ch);
        c = std::min<int64_t>(c, LDS_BUDGET / (2 * chf * 4));
        c = std::min<int64_t>(c, (int64_t)SLOTS * NT / (chd / 4));
        if (CCT > 0) c = c >= CCT ? CCT : 0;
        if (WK > 1 && c > WK) c -= c % WK;  // equal channel shares for the K slices
        return c;
    };
    int64_t cc = channels(ch_floats, ch_dma);
    // Row-aligned blocks with column-window slabs (d_filter rows of
    // min(P, d_out) + d_filter - 1 positions): for 2D images whose whole-row
    // slabs do not fit, and on the wide tiles wherever a row's blocks leave
    // at most 2 % of their positions idle (d_out just under a multiple of
    // P): their slabs are 3 rows instead of up to 7, measured +0.1-0.9 % on
    // such images (d_out = 126, 254, 256, 382, 638) and far slower elsewhere.
    const int64_t nseg_r = (Do + P - 1) / P;
    const bool snug = MW * NW >= 32 && Do * 50 >= nseg_r * P * 49;
    int rowblk = 0;
    int64_t nseg = 1, sw = 0;
    if (KD == 2 && (CLIFF_ROWBLK == 2 || (p.rowblk == 2 && snug) ||
                    (cc < 1 && CLIFF_ROWBLK == 1 && p.rowblk == 1))) {
        sw = std::min<int64_t>(P, Do) + df - 1;
        const int64_t chf = df * sw * NB + (NEG ? 2 : 1) * wch;
        const int64_t chd = df * sw * NB + wch;
        const int64_t c = channels(chf, chd);
        if (c >= 1) {
            ch_floats = chf;
            ch_dma = chd;
            cc = c;
            nseg = (Do + P - 1) / P;
            n_pos_blk = p.B * Do * nseg;
            rowblk = 1;
        }
    }
    if (cc < 1 || (NEG && cc != 1)) return CLIFF_EUNSUPPORTED;
    (void)ch_dma;
    const int64_t n_blk = n_pos_blk * n_co_blk;
    if (n_blk >= (1ll << 31)) return CLIFF_EUNSUPPORTED;
    const int64_t stage_floats = cc * ch_floats;
    // the K split's partial sums reuse the stage buffers after the loop
    const int64_t red_bytes = (int64_t)(WK - 1) * WCO * WPOS * MW * NW * 64 * 16;
    const int64_t lds_bytes = std::max<int64_t>(2 * stage_floats * 4, red_bytes);
    if (lds_bytes > 160 * 1024) return CLIFF_EUNSUPPORTED;
    // staging offsets are 32-bit, relative to the block's first plane
    int64_t img = NB;
    for (int t = 0; t < KD; ++t) img *= D;
    // flattened blocks: planes of several batch entries, offsets relative to
    // the first (and images below 2^24 floats per plane); row-aligned
    // blocks: rows of one plane, cc channels from the block's first
    if ((!rowblk && (D * D * NB >= (1 << 24) ||
                     (cc + (planes + 2) * p.C_in) * img >= (1ll << 31))) ||
        (rowblk && (cc + 1) * img >= (1ll << 31)) ||
        cc * p.C_out * df * df * (KD == 3 ? df : 1) * NB >= (1ll << 31))
        return CLIFF_EUNSUPPORTED;
    if (p.blocks_out) {
        *p.blocks_out = n_blk;
        return CLIFF_OK;
    }

    MfmaArgs a;
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
    a.npos = (int)npos;
    a.cc = (int)cc;
    const int64_t n_cgrp = (p.C_in + cc - 1) / cc;
    a.n_stage = (int)(KD == 2 ? n_cgrp : n_cgrp * df);
    a.n_co_blk = (int)n_co_blk;
    a.n_blk = (int)n_blk;
    a.rowblk = rowblk;
    a.nseg = (int)nseg;
    a.sw = (int)sw;
    a.stage_floats = (int)stage_floats;
    a.sign = p.sign;
    a.act = p.act;
    if (debug_enabled())
        fprintf(stderr,
                "cliffconv: conv_mfma k=%d d_filter=%d tile %dx%d waves of %dx%d MFMA tiles "
                "(%d channels x %d positions), K split over %d waves, %lld workgroups, "
                "%d channels/stage, %lld LDS bytes%s%s\n",
                KD, (int)df, WCO, WPOS, MW, NW, CO_WG, P, WK, (long long)n_blk, (int)cc,
                (long long)lds_bytes, rowblk ? ", row-aligned blocks" : "",
                NEG ? ", negated filter copy" : "");
    if (observe_launch(LAUNCH_CONV_MFMA,
                       {KD, NB, DF, CCT, WCO, WPOS, MW, NW, SLOTS, WAVES, WK, NEG}, n_blk, NT,
                       lds_bytes, &a))
        return CLIFF_OK;
    clear_hip_error();
    hipLaunchKernelGGL((conv_mfma_kernel<KD, NB, DF, CCT, WCO, WPOS, MW, NW, SLOTS, WAVES, WK, NEG>),
                       dim3((unsigned)n_blk), dim3(NT), (size_t)lds_bytes, stream, a);
    return hipGetLastError() == hipSuccess ? CLIFF_OK : CLIFF_EDEVICE;
}

// Tile shapes: workgroup = WCO x WPOS waves, each wave MW x NW MFMA tiles
// (16 x 16 each): WCO * MW * (16 / N_B) output channels by WPOS * NW * 16
// positions.
//  wide    the large workloads; chosen by measurement on MI355X: k = 2 takes
//          all 64 channels in one workgroup (4 x 1 waves of 4 x 8 tiles,
//          2 waves/SIMD), k = 3 does best with 4 x 4 tiles at 3 waves/SIMD
//  medium  many channels, few positions: 32 positions per workgroup
//  narrow  few channels, many positions
//  tiny    4 (k = 2) or 2 (k = 3) channels by 32 positions, the K loop split
//          over 4 waves: small problems, spread over as many CUs as possible
#ifndef CLIFF_W2
#define CLIFF_W2 4, 1, 4, 8, 6, 2, 1, 80  // WCO, WPOS, MW, NW, SLOTS, waves/SIMD, K split,
                                         // LDS budget (KB, two stage buffers) (k = 2)
#endif
#ifndef CLIFF_W3
#define CLIFF_W3 2, 2, 4, 4, 6, 3  // same for k = 3
#endif
#define CLIFF_W2_32 2, 2, 4, 8, 10, 2, 1, 80 // k = 2 wide variant for C_out <= 32
// ... and for C_out <= 16 (8) 16 (8) channels by 512, 384 or 256 positions:
// one wave of channels, four of positions, 8, 6 or 4 MFMA tiles per wave
#define CLIFF_W2_16 1, 4, 4, 8, 10, 2, 1, 80
#define CLIFF_W2_16_384 1, 4, 4, 6, 10, 2, 1, 80
#define CLIFF_W2_16_256 1, 4, 4, 4, 10, 2, 1, 80
#define CLIFF_W2_8 1, 4, 2, 8, 10, 2, 1, 80
#define CLIFF_W2_8_384 1, 4, 2, 6, 10, 2, 1, 80
#define CLIFF_W2_8_256 1, 4, 2, 4, 10, 2, 1, 80
#ifndef CLIFF_W2_16ON
#define CLIFF_W2_16ON 1
#endif
#ifndef CLIFF_W2_8ON
#define CLIFF_W2_8ON 1
#endif
#ifndef CLIFF_W2_SMALL_MODEL
#define CLIFF_W2_SMALL_MODEL 1
#endif
// the 64-channel tile with 10 staging slots, for stages that need them
// (large images or filters; 6 slots measured 0.4 % faster where they suffice)
#define CLIFF_W2_S10 4, 1, 4, 8, 10, 2, 1, 80
// the 64-channel tile 96 and 112 positions wide (4x6, 4x7 tiles per wave)
#define CLIFF_W2_96 4, 1, 4, 6, 6, 2, 1, 80
#define CLIFF_W2_112 4, 1, 4, 7, 6, 2, 1, 80
#ifndef CLIFF_W2_112ON
#define CLIFF_W2_112ON 1
#endif
// ... and 64 positions wide (4x4 tiles per wave), for layers too small to
// fill the CUs with the wider blocks
#define CLIFF_W2_64 4, 1, 4, 4, 6, 2, 1, 80
#ifndef CLIFF_W2_64ON
#define CLIFF_W2_64ON 1
#endif
// the d_filter = 1 (linear) wide kernels keep 6 slots: with 9 they spill
#define CLIFF_W2_LIN 4, 1, 4, 8, 6, 2, 1, 80
#define CLIFF_W2_32_LIN 2, 2, 4, 8, 6, 2, 1, 80
#define CLIFF_W3_32 4, 1, 4, 8, 6, 2  // k = 3, 3x3x3 wide variant for 16 < C_out <= 32
#define CLIFF_W3_32_96 4, 1, 4, 6, 6, 2  // the same with 96 positions (6 tiles per wave)
#define CLIFF_W3_32_112 4, 1, 4, 7, 6, 2  // ... and 112 (7 tiles per wave)
#ifndef CLIFF_W3_112
#define CLIFF_W3_112 1
#endif
// k = 3, 3x3x3, C_out <= 8: one wave of channels, four of positions
// 2D 5x5 and 7x7 filters: unrolled instantiations like the 3x3 one
// (measured against the runtime tap loop: 5x5, C = 64, d 128 78.2 -> 87.0 %
// of the peak, d 260 82.8 -> 92.0 %; 7x7, C = 64, d 70 74.2 -> 87.9 %)
#ifndef CLIFF_DF5
#define CLIFF_DF5 1
#endif
#ifndef CLIFF_NARROW10
#define CLIFF_NARROW10 1
#endif
#ifndef CLIFF_DF7
#define CLIFF_DF7 1
#endif
#ifndef CLIFF_W3_8
#define CLIFF_W3_8 1, 4, 4, 4, 6, 3
#endif
#ifndef CLIFF_W3_8ON
#define CLIFF_W3_8ON 1
#endif
#define CLIFF_MEDIUM2 4, 1, 4, 2, 8, 4
#define CLIFF_MEDIUM3 4, 1, 4, 2, 8, 3
#define CLIFF_NARROW 1, 4, 2, 4, 8, 2
// tiny: one 4 (2D) / 2 (3D) channel x 32 position tile per workgroup, its K
// loop split over 4 waves (measured 1.1-2.2x faster than one wave on small
// problems, whose critical path is the K loop, not the tile)
#ifndef CLIFF_TINY_WK
#define CLIFF_TINY_WK 4
#endif
#define CLIFF_TINY2 1, 1, 1, 2, 12, 4, CLIFF_TINY_WK
#define CLIFF_TINY3 1, 1, 1, 2, 12, 3, CLIFF_TINY_WK

template <int NB, int WCO, int WPOS, int MW, int NW, int SLOTS, int WAVES, int WK = 1,
          int LDSKB = 64>
struct Shape {
    static constexpr int co_wg = WCO * MW * (16 / NB);
    static constexpr int pos = WPOS * NW * 16;
    static int64_t blocks(const ConvProblem& p, int64_t M)
    {
        return (M + pos - 1) / pos * ((p.C_out + co_wg - 1) / co_wg);
    }
};

template <int KD, int NB, int DF, int CCT, int WCO, int WPOS, int MW, int NW, int SLOTS, int WAVES,
          int WK, int LDSKB>
cliff_status run_shape_cfg(const ConvProblem& p, hipStream_t stream,
                           Shape<NB, WCO, WPOS, MW, NW, SLOTS, WAVES, WK, LDSKB>)
{
    // 3D, one channel per stage and no zero sign in the table: the negated
    // filter copy replaces the sign multiplies.  Measured (interleaved, same
    // box): 3D block layers +1.2-1.3 %, 3D C = 32 +0.1 %; the 2D tiles lose
    // 1.3-4 % (twice the filter bytes per stage, 2 workgroups per CU: the
    // copy's LDS writes before the stage barrier cost more than the
    // multiplies), so they keep the multiplies.
    if constexpr ((KD == 3 || CLIFF_CONV_NEG2D) && CCT == 1 && DF > 0 && WK == 1 && CLIFF_CONV_NEG)
        if (p.sign.zero == 0)
            return run<KD, NB, DF, CCT, WCO, WPOS, MW, NW, SLOTS, WAVES, WK, LDSKB, true>(p,
                                                                                         stream);
    return run<KD, NB, DF, CCT, WCO, WPOS, MW, NW, SLOTS, WAVES, WK, LDSKB, false>(p, stream);
}

template <int KD, int NB, int DF, class Wide, class... WideAlt>
cliff_status run_shapes(const ConvProblem& p, hipStream_t stream);

// 2D, few output channels: one of three widths of the same tile (512, 384
// or 256 positions).  On problems of >= 1 GFLOP the width whose workgroups
// occupy the fewest position slots per CU is taken: rounds of whole blocks
// on the CUs times the width, with the block count the kernel itself would
// launch (row-aligned blocks with their partly idle last segment of a row
// counted as whole blocks); ties go to the wider tile.  Otherwise, and when
// the tile is forced, 512.
template <int KD, int NB, int DF, class W512, class W384, class W256>
cliff_status run_small_channels(const ConvProblem& p, hipStream_t stream)
{
    using Fallback = Shape<NB, CLIFF_W2_32>;
    const int64_t M = p.B * p.d_out * p.d_out;
    const double useful = 2.0 * M * p.C_out * NB * p.C_in * NB * (double)(p.d_filter * p.d_filter);
    const int cus = device_cus();
    if (CLIFF_W2_SMALL_MODEL && p.mfma_shape < 0 && useful >= 1e9 && cus > 0) {
        constexpr int WCC = DF == 3 ? 1 : 0;
        auto slots = [&](auto shape) -> int64_t {
            int64_t n = 0;
            ConvProblem q = p;
            q.blocks_out = &n;
            q.rowblk = 2;  // as the first attempt below: row-aligned where snug
            if (run_shape_cfg<KD, NB, DF, WCC>(q, stream, shape) != CLIFF_OK) {
                q.rowblk = 1;  // whole-row slabs do not fit
                if (run_shape_cfg<KD, NB, DF, WCC>(q, stream, shape) != CLIFF_OK)
                    return INT64_MAX;
            }
            return (n + cus - 1) / cus * decltype(shape)::pos;
        };
        const int64_t s512 = slots(W512{}), s384 = slots(W384{}), s256 = slots(W256{});
        if (s384 < s512 && s384 <= s256) return run_shapes<KD, NB, DF, W384, Fallback>(p, stream);
        if (s256 < s512 && s256 < s384) return run_shapes<KD, NB, DF, W256, Fallback>(p, stream);
    }
    return run_shapes<KD, NB, DF, W512, Fallback>(p, stream);
}

template <int KD, int NB, int DF>
cliff_status run_shape(const ConvProblem& p, hipStream_t stream)
{
    // k = 2 has four wide tiles: 64 channels x 128 positions, for C_out <=
    // 32 a 32 x 256 one, and for C_out <= 16 and <= 8 16 and 8 channels by
    // 512 (384, 256) positions, so the channels are not half wasted
    if constexpr (KD == 2 && DF == 1) {
        if (p.C_out <= 32) return run_shapes<KD, NB, DF, Shape<NB, CLIFF_W2_32_LIN>>(p, stream);
        return run_shapes<KD, NB, DF, Shape<NB, CLIFF_W2_LIN>>(p, stream);
    } else if constexpr (KD == 2) {
        if (CLIFF_W2_8ON && p.C_out <= 8)
            return run_small_channels<KD, NB, DF, Shape<NB, CLIFF_W2_8>, Shape<NB, CLIFF_W2_8_384>,
                                      Shape<NB, CLIFF_W2_8_256>>(p, stream);
        if (CLIFF_W2_16ON && p.C_out <= 16)
            return run_small_channels<KD, NB, DF, Shape<NB, CLIFF_W2_16>,
                                      Shape<NB, CLIFF_W2_16_384>, Shape<NB, CLIFF_W2_16_256>>(
                p, stream);
        if (p.C_out <= 32) return run_shapes<KD, NB, DF, Shape<NB, CLIFF_W2_32>>(p, stream);
        // 64 channels; when their stage needs more slots (large filters or
        // images), the same tile with 10 slots, then the 32-channel tile,
        // before the narrower shapes
        // On problems of >= 1 GFLOP, 128 or 96 positions per block: the
        // width whose blocks fill the last round of CUs better (the 128 tile's
        // row-aligned blocks counted where they are snug, as the kernel takes
        // them; the 96 tile, with 24 MFMA tiles per wave, never takes them)
        using W128 = Shape<NB, CLIFF_W2>;
        using W112 = Shape<NB, CLIFF_W2_112>;
        using W96 = Shape<NB, CLIFF_W2_96>;
        const int64_t Do = p.d_out, M = p.B * Do * Do;
        const double useful = 2.0 * M * p.C_out * NB * p.C_in * NB * (double)(p.d_filter * p.d_filter);
        const int cus = device_cus();
        auto nblk = [&](int64_t P, bool snug_ok) {
            const int64_t nseg = (Do + P - 1) / P;
            return snug_ok && Do * 50 >= nseg * P * 49 ? p.B * Do * nseg : (M + P - 1) / P;
        };
        auto fill = [&](int64_t n) {
            return (double)n / (double)(((n + cus - 1) / cus) * cus);
        };
        if (CLIFF_W2_WIDTH_MODEL && p.mfma_shape < 0 && useful >= 1e9 && cus > 0) {
            const double f128 = fill(nblk(W128::pos, true));
            const double f112 = CLIFF_W2_112ON ? fill(nblk(W112::pos, false)) : 0.0;
            const double f96 = fill(nblk(W96::pos, false));
            // the 64-position form (with half the MFMAs per stage it runs at
            // about 0.85 of the wider tiles' rate when the CUs are full:
            // measured 75.5 against 88 %) only where it still comes out
            // ahead, and only where its 6-slot stage fits (a planning call of
            // the kernel's own host code, no launch): else its fallbacks
            // would be the 32-channel tile at half the blocks
            using W64 = Shape<NB, CLIFF_W2_64>;
            const double f64 = CLIFF_W2_64ON ? fill(nblk(W64::pos, false)) : 0.0;
            auto fits = [&](auto shape) {
                int64_t n = 0;
                ConvProblem q = p;
                q.blocks_out = &n;
                q.rowblk = 2;
                return run_shape_cfg<KD, NB, DF, DF == 3 ? 1 : 0>(q, stream, shape) == CLIFF_OK;
            };
            if (0.85 * f64 > std::max({f128, f112, f96}) && fits(W64{}))
                return run_shapes<KD, NB, DF, W64, Shape<NB, CLIFF_W2_S10>,
                                  Shape<NB, CLIFF_W2_32>>(p, stream);
            if (f112 > f128 && f112 >= f96)
                return run_shapes<KD, NB, DF, W112, Shape<NB, CLIFF_W2_S10>,
                                  Shape<NB, CLIFF_W2_32>>(p, stream);
            if (f96 > f128)
                return run_shapes<KD, NB, DF, W96, Shape<NB, CLIFF_W2_S10>,
                                  Shape<NB, CLIFF_W2_32>>(p, stream);
        }
        return run_shapes<KD, NB, DF, W128, Shape<NB, CLIFF_W2_S10>,
                          Shape<NB, CLIFF_W2_32>>(p, stream);
    } else {
        // k = 3 with 3x3x3 filters and 17..32 output channels: all of them
        // in one 32 x 128 tile (measured +0.9 % at C = 32 against two 16 x
        // 128 blocks; with 64 channels the 16 x 128 tile stays 2 % faster)
        // and with C_out <= 8 all of them in one 8 x 256 tile (measured 76 ->
        // 88-90 % of the peak against two 4-channel narrow blocks)
        if constexpr (DF == 3)
            if (CLIFF_W3_8ON && p.C_out <= 8)
                return run_shapes<KD, NB, DF, Shape<NB, CLIFF_W3_8>>(p, stream);
        if constexpr (DF == 3)
            if (p.C_out <= 32 && p.C_out > 16) {
                // Two widths, 128 and 96 positions: on problems of >= 1 GFLOP
                // the quantisation model (below) takes the one whose blocks
                // fill the last round of CUs better.  Measured (interleaved):
                // B = 8, d 32 -> 30 +2.8 % with 96, d 42 -> 40 +2.4 %; d 34
                // -> 32 (2048 blocks of 128) -4 % with 96; d 24 -> 22, where
                // only 96 makes the wide tile worth taking, +13 %.
                using W128 = Shape<NB, CLIFF_W3_32>;
                using W112 = Shape<NB, CLIFF_W3_32_112>;
                using W96 = Shape<NB, CLIFF_W3_32_96>;
                int64_t M = p.B;
                for (int t = 0; t < KD; ++t) M *= p.d_out;
                const double useful = 2.0 * M * p.C_out * NB * p.C_in * NB * 27.0;
                const int cus = device_cus();
                auto fill = [&](int64_t n) {
                    return (double)n / (double)(((n + cus - 1) / cus) * cus);
                };
                if (p.mfma_shape < 0 && useful >= 1e9 && cus > 0) {
                    const double f128 = fill(W128::blocks(p, M));
                    const double f112 = CLIFF_W3_112 ? fill(W112::blocks(p, M)) : 0.0;
                    const double f96 = fill(W96::blocks(p, M));
                    if (f112 > f128 && f112 >= f96) return run_shapes<KD, NB, DF, W112>(p, stream);
                    if (f96 > f128) return run_shapes<KD, NB, DF, W96>(p, stream);
                }
                return run_shapes<KD, NB, DF, W128>(p, stream);
            }
        return run_shapes<KD, NB, DF, Shape<NB, CLIFF_W3>>(p, stream);
    }
}

template <int KD, int NB, int DF, class Wide, class... WideAlt>
cliff_status run_shapes(const ConvProblem& p, hipStream_t stream)
{
    using Medium = std::conditional_t<KD == 2, Shape<NB, CLIFF_MEDIUM2>, Shape<NB, CLIFF_MEDIUM3>>;
    using Narrow = Shape<NB, CLIFF_NARROW>;
    using Tiny = std::conditional_t<KD == 2, Shape<NB, CLIFF_TINY2>, Shape<NB, CLIFF_TINY3>>;
    int64_t M = p.B;
    for (int t = 0; t < KD; ++t) M *= p.d_out;
    // Shape choice, from timing every shape on 2D/3D convolutions and linear
    // layers (d_image = d_filter = 1) of 7 to 9,000 GFLOP on MI355X (256 CUs):
    // wide once it fills every CU; medium for linear layers with >= 128
    // workgroups; narrow from 128 workgroups; tiny (the smallest tile, the
    // most workgroups) for the smallest problems.  A shape whose LDS or
    // staging needs do not fit returns CLIFF_EUNSUPPORTED and the next one in
    // the order is tried.
    const bool wide_ok = p.C_out * 2 > Wide::co_wg;
    const bool medium_ok = p.C_out * 2 > Medium::co_wg;
    const int64_t bw = wide_ok ? Wide::blocks(p, M) : 0;
    const int64_t bm = medium_ok ? Medium::blocks(p, M) : 0;
    const int64_t bn = Narrow::blocks(p, M);
    int first;
    if (bw >= 256)
        first = 0;
    else if (bm >= 128 && p.d_filter == 1)
        first = 1;
    else if (bn >= 128)
        first = 2;
    else if (bm >= 128)
        first = 1;
    else
        first = 3;
    // Convolutions of >= 1 GFLOP: a quantisation model instead, fitted to
    // timing every shape forced on 24 2D/3D problems (MI355X).  One block of
    // any shape keeps its CU's matrix cores busy, so a shape's N blocks take
    // ceil(N / CUs) rounds of whole blocks, and its rate is roughly
    //     b * N / (ceil(N / CUs) * CUs) * C_out / (its channel blocks * CO_WG)
    // with b its rate on large problems (fraction of the peak): wide 0.87
    // (2D) / 0.90 (3D), medium 0.74 / 0.81, narrow 0.74, tiny 0.25.  The largest
    // estimate goes first.  Smaller problems are latency-bound (the tiny
    // tile's split K loop wins there) and keep the rule above; linear layers
    // (d_filter = 1) too.
    const double useful = 2.0 * M * p.C_out * NB * p.C_in * NB *
                          std::pow((double)p.d_filter, KD);
    const int cus = device_cus();
    if (CLIFF_SHAPE_MODEL && p.d_filter > 1 && useful >= 1e9 && cus > 0) {
        auto est = [&](bool ok, int64_t n, int co_wg, double b) {
            if (!ok || n < 1) return 0.0;
            const int64_t rounds = (n + cus - 1) / cus;
            const double u =
                (double)p.C_out / (double)(((p.C_out + co_wg - 1) / co_wg) * co_wg);
            return b * (double)n / (double)(rounds * cus) * u;
        };
        const double e[4] = {est(wide_ok, bw, Wide::co_wg, KD == 2 ? 0.87 : 0.90),
                             est(medium_ok, bm, Medium::co_wg, KD == 2 ? 0.74 : 0.81),
                             est(true, bn, Narrow::co_wg, 0.74),
                             est(true, Tiny::blocks(p, M), Tiny::co_wg, 0.25)};
        first = 0;
        for (int i = 1; i < 4; ++i)
            if (e[i] > e[first]) first = i;
    }
    int order[4] = {first, 0, 2, 1};
    int n_order = 4;
    if (p.mfma_shape >= 0) {
        order[0] = p.mfma_shape;  // forced by the caller
        n_order = 1;
    }
    // the 3x3(x3) wide kernels stage one input channel at a time (a stage
    // already holds 288 MFMAs per wave, and the fixed count keeps their
    // register use down); the other shapes choose the channels per stage at
    // run time
    constexpr int WCC = DF == 3 ? 1 : 0;
    auto attempt = [&](const ConvProblem& q) {
        for (int i = 0; i < n_order; ++i) {
            const int o = order[i];
            if (i > 0 && o == order[0]) continue;
            const bool forced = q.mfma_shape >= 0;
            cliff_status s = CLIFF_EUNSUPPORTED;
            if (o == 0 && (wide_ok || forced))
                s = run_shape_cfg<KD, NB, DF, WCC>(q, stream, Wide{});
            if (o == 0)
                ((s = s == CLIFF_EUNSUPPORTED && (q.C_out * 2 > WideAlt::co_wg || forced)
                          ? run_shape_cfg<KD, NB, DF, WCC>(q, stream, WideAlt{})
                          : s),
                 ...);
            if (o == 1 && (medium_ok || forced))
                s = run_shape_cfg<KD, NB, DF, 0>(q, stream, Medium{});
            if (o == 2) s = run_shape_cfg<KD, NB, DF, 0>(q, stream, Narrow{});
            // 2D: the narrow tile with 10 staging slots, for stages that
            // need them (large filters)
            if constexpr (KD == 2 && CLIFF_NARROW10)
                if (o == 2 && s == CLIFF_EUNSUPPORTED)
                    s = run_shape_cfg<KD, NB, DF, 0>(q, stream, Shape<NB, CLIFF_W2_8_256>{});
            if (o == 3) s = run_shape_cfg<KD, NB, DF, 0>(q, stream, Tiny{});
            if (s != CLIFF_EUNSUPPORTED) return s;
        }
        if (q.mfma_shape < 0 && first != 3)
            return run_shape_cfg<KD, NB, DF, 0>(q, stream, Tiny{});
        return CLIFF_EUNSUPPORTED;
    };
    // whole-row slabs first (flattened blocks waste no positions) except on
    // the wide tiles where row-aligned blocks leave almost none idle (rowblk
    // 2); 2D images too wide for whole-row slabs in every shape then take
    // row-aligned blocks
    ConvProblem p0 = p;
    if (KD == 2 && CLIFF_ROWBLK == 1 && p0.rowblk == 0) p0.rowblk = 2;
    cliff_status s = attempt(p0);
    if (s == CLIFF_EUNSUPPORTED && KD == 2 && CLIFF_ROWBLK == 1) {
        ConvProblem q = p;
        q.rowblk = 1;
        s = attempt(q);
    }
    return s;
}

}  // namespace

cliff_status launch_conv_mfma(const ConvProblem& p, hipStream_t stream)
{
    // 3x3(x3) filters and the linear layer (d_filter = 1) get unrolled,
    // software-pipelined loops; other sizes a runtime tap loop
    if (p.k == 2) {
        if (p.d_filter == 3) return run_shape<2, 4, 3>(p, stream);
        if (p.d_filter == 1) return run_shape<2, 4, 1>(p, stream);
        if (CLIFF_DF5 && p.d_filter == 5) return run_shape<2, 4, 5>(p, stream);
        if (CLIFF_DF7 && p.d_filter == 7) return run_shape<2, 4, 7>(p, stream);
        return run_shape<2, 4, 0>(p, stream);
    }
    if (p.k == 3) {
        if (p.d_filter == 3) return run_shape<3, 8, 3>(p, stream);
        if (p.d_filter == 1) return run_shape<3, 8, 1>(p, stream);
        return run_shape<3, 8, 0>(p, stream);
    }
    return CLIFF_EUNSUPPORTED;
}

}  // namespace cliff
