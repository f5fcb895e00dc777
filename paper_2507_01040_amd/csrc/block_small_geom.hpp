// Address arithmetic of block_small_kernel (the fused two-layer block): where
// a workgroup's direct global->LDS loads read and land, which LDS words each
// MFMA fragment reads, and where each layer's outputs go.  The kernel and the
// host-side bounds checker (a CPU build of the library used by the tests)
// both call these functions, so the checker verifies the kernel's own
// arithmetic.
#pragma once

#include <stdint.h>

#include "common.hpp"

namespace cliff {

struct BlockArgs {
    const float* x;
    const float* w1;
    const float* b1;
    const float* w2;
    const float* b2;
    float* y;
    int C0, C1, C2;   // input, intermediate and output channels
    int D0, D1, D2;   // their spatial sizes
    int df, taps;     // d_filter and d_filter^k
    int R;            // final-output slices per workgroup
    int n_band;       // bands per batch entry
    int lds_y1, lds_w1, lds_w2;  // float offsets in LDS (the input band is at 0)
    SignMasks sign;
    ActParams act1, act2;
};

// Quotient of non-negative ints as an unsigned division (a shorter sequence
// than the signed one); every index divided here is non-negative.
__host__ __device__ inline int bs_udiv(int a, int b) { return (int)((unsigned)a / (unsigned)b); }

__host__ __device__ inline int bs_ipow(int a, int k)
{
    int r = 1;
    for (int t = 0; t < k; ++t) r *= a;
    return r;
}

// Workgroup bid's band: batch entry b, final-output slices s0 .. s0 + R2 - 1
// (rows for k = 2, planes for k = 3); the layers read R1 intermediate and R0
// input slices from s0 on.  S* = positions per slice.
struct BsBand {
    int b, s0, R2, R1, R0, S0, S1, S2;
};

__host__ __device__ inline BsBand bs_band(const BlockArgs& a, int KD, int df, int bid)
{
    BsBand g;
    g.b = bs_udiv(bid, a.n_band);
    g.s0 = (bid - g.b * a.n_band) * a.R;
    g.R2 = a.R < a.D2 - g.s0 ? a.R : a.D2 - g.s0;
    g.R1 = g.R2 + df - 1;
    g.R0 = g.R1 + df - 1;
    g.S0 = bs_ipow(a.D0, KD - 1);
    g.S1 = bs_ipow(a.D1, KD - 1);
    g.S2 = bs_ipow(a.D2, KD - 1);
    return g;
}

// Staging: float4 e of the input band ([C0][R0][S0][NB] in LDS from float 0)
// comes from input float bs_band_src; float4 e of a filter tensor lands at
// its area's float 4 e (a straight copy).
__host__ __device__ inline int bs_band_f4(const BsBand& g, int NB) { return g.R0 * g.S0 * NB / 4; }
__host__ __device__ inline int64_t bs_band_src(const BlockArgs& a, const BsBand& g, int NB, int e)
{
    const int ch4 = bs_band_f4(g, NB);
    const int ci = bs_udiv(e, ch4);
    const int r = e - ci * ch4;
    return (((int64_t)g.b * a.C0 + ci) * a.D0 + g.s0) * g.S0 * NB + 4 * r;
}

// One layer: input [Cin][Rin][Sin][NB] in LDS (slices of din^(k-1)
// positions, rows of din), output Rout x Sout positions of Cout channels.
struct BsLayer {
    int Cin, Rin, din, Sin, Cout, Rout, dout, Sout;
};

__host__ __device__ inline BsLayer bs_layer1(const BlockArgs& a, const BsBand& g)
{
    return BsLayer{a.C0, g.R0, a.D0, g.S0, a.C1, g.R1, a.D1, g.S1};
}
__host__ __device__ inline BsLayer bs_layer2(const BlockArgs& a, const BsBand& g)
{
    return BsLayer{a.C1, g.R1, a.D1, g.S1, a.C2, g.R2, a.D2, g.S2};
}

// Lane roles: A row mrow = (channel co_a, blade i_a) of a 16-row tile, MFMA K
// slot kk; D fragment rows 4 kk .. 4 kk + 3 = channel co_o, blades i0 .. i0+3.
struct BsLane {
    int mrow, kk, co_a, i_a, co_o, i0;
};

__host__ __device__ inline BsLane bs_lane(int NB, int lane)
{
    BsLane l;
    l.mrow = lane & 15;
    l.kk = lane >> 4;
    l.co_a = l.mrow / NB;
    l.i_a = l.mrow % NB;
    l.co_o = NB == 4 ? l.kk : (l.kk >> 1);
    l.i0 = NB == 4 ? 0 : 4 * (l.kk & 1);
    return l;
}

// Tile t of a layer (row tile rt = t mod RT over 16 / NB channels, column
// tile pt over 16 positions): the lane's A channel and B position, clamped
// into range (their products only reach outputs that are not stored), the
// float offsets of its fragment bases from the layer's filter and input
// areas, and its D fragment's output channel and position.
struct BsTile {
    int co_r, m_r, so, yy, xx;  // A row channel; B column position (slice, row, column)
    int a_base, b_base;         // float offsets in the filter and input areas
    int co, m;                  // D fragment channel and position (store if co < Cout, m < npos)
};

__host__ __device__ inline int bs_tiles(const BsLayer& L, int NB)
{
    const int npos = L.Rout * L.Sout;
    return ((npos + 15) / 16) * ((L.Cout + 16 / NB - 1) / (16 / NB));
}

__host__ __device__ inline BsTile bs_tile(const BsLayer& L, int KD, int NB, int taps,
                                          const BsLane& l, int t)
{
    const int CPT = 16 / NB;
    const int npos = L.Rout * L.Sout;
    const int RT = (L.Cout + CPT - 1) / CPT;
    const int pt = bs_udiv(t, RT), rt = t - pt * RT;
    BsTile T;
    T.co_r = rt * CPT + l.co_a < L.Cout - 1 ? rt * CPT + l.co_a : L.Cout - 1;
    T.m_r = pt * 16 + l.mrow < npos - 1 ? pt * 16 + l.mrow : npos - 1;
    T.so = bs_udiv(T.m_r, L.Sout);
    const int r = T.m_r - T.so * L.Sout;
    T.yy = KD == 3 ? bs_udiv(r, L.dout) : 0;
    T.xx = KD == 3 ? r - T.yy * L.dout : r;
    T.a_base = T.co_r * taps * NB;
    T.b_base = (T.so * L.Sin + T.yy * L.din + T.xx) * NB + l.kk;
    T.co = rt * CPT + l.co_o;
    T.m = pt * 16 + l.mrow;
    return T;
}

// Fragment reads of input channel ci, tap (qs, qy, qx) (qs: slice offset;
// 2D: qy = 0) and blade group h: A at the filter area's float bs_a_ofs (the
// raw blade srcb = src(i_a, 4 h + kk)), B at the input area's float
// bs_b_ofs; each is a per-channel base plus a per-tap offset, so that the
// kernel forms the bases once per channel.
__host__ __device__ inline int bs_a_ci(const BsLayer& L, const BsTile& T, int NB, int taps, int ci)
{
    return T.a_base + ci * L.Cout * taps * NB;
}
__host__ __device__ inline int bs_a_tap(int NB, int tap, int srcb) { return tap * NB + srcb; }
__host__ __device__ inline int bs_b_ci(const BsLayer& L, const BsTile& T, int NB, int ci)
{
    return T.b_base + ci * L.Rin * L.Sin * NB;
}
__host__ __device__ inline int bs_b_tap(const BsLayer& L, int NB, int qs, int qy, int qx, int h)
{
    return (qs * L.Sin + qy * L.din + qx) * NB + 4 * h;
}
__host__ __device__ inline int bs_a_ofs(const BsLayer& L, const BsTile& T, int NB, int taps,
                                        int ci, int tap, int srcb)
{
    return bs_a_ci(L, T, NB, taps, ci) + bs_a_tap(NB, tap, srcb);
}
__host__ __device__ inline int bs_b_ofs(const BsLayer& L, const BsTile& T, int NB, int ci, int qs,
                                        int qy, int qx, int h)
{
    return bs_b_ci(L, T, NB, ci) + bs_b_tap(L, NB, qs, qy, qx, h);
}

// Stores of one lane's 4 blades at (co, m): layer 1 into the intermediate
// area ([C1][R1][S1][NB]), layer 2 into the output tensor.
__host__ __device__ inline int bs_y1_ofs(const BsBand& g, int NB, int co, int m, int i0)
{
    return (co * g.R1 * g.S1 + m) * NB + i0;
}
__host__ __device__ inline int64_t bs_y_ofs(const BlockArgs& a, const BsBand& g, int NB, int co,
                                            int m, int i0)
{
    return ((((int64_t)g.b * a.C2 + co) * a.D2 + g.s0) * g.S2 + m) * NB + i0;
}

}  // namespace cliff
