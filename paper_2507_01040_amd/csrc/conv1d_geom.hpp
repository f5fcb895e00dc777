// Address arithmetic of conv1d_mfma_kernel (k = 1, N_B = 2): the block of
// flattened output positions a workgroup owns, its input window, where each
// lane's direct global->LDS loads read and land, which LDS words each MFMA
// fragment reads and where each output goes.  The kernel and the host-side
// bounds checker (a CPU build of the library used by the tests) both call
// these functions, so the checker verifies the kernel's own arithmetic.
#pragma once

#include <stdint.h>

#include "common.hpp"

namespace cliff {

// Quotient of non-negative ints as an unsigned division (a shorter sequence
// than the signed one); every index divided here is non-negative.
__host__ __device__ inline int c1_udiv(int a, int b) { return (int)((unsigned)a / (unsigned)b); }

struct C1Args {
    const float* x;
    const float* w;
    const float* bias;
    float* y;
    int C_in, C_out, D, Do, df;
    int M;          // B * d_out flattened output positions
    int n_co_blk;
    int n_blk;
    int cc;         // input channels per stage
    int ccp;        // channel slots per stage buffer: cc rounded up to even
    int n_stage;
    int span2;      // floats per channel window: 2 * (P + rows_max * (d_filter - 1))
    int stage_floats;
    SignMasks sign;
    ActParams act;
};

// One instantiation's compile-time shape as plain ints: DF filter length (0:
// run time), WCO x WPOS waves of MW x NW MFMA tiles, SIN input and SW filter
// staging slots per lane, FW / FX floats per filter / input direct load (4:
// 16 bytes, 1: 4 bytes), the K loop split over WK waves.
struct C1Tile {
    int DF, WCO, WPOS, MW, NW, SIN, SW, FW, FX, WK;
    __host__ __device__ constexpr int nt() const { return 64 * WCO * WPOS * WK; }
    __host__ __device__ constexpr int co_wg() const { return WCO * MW * 8; }
    __host__ __device__ constexpr int pos() const { return WPOS * NW * 16; }
};

constexpr uint32_t C1_NOLOAD = 0xffffffffu;

// The block: P consecutive flattened positions [m0, m_end) from batch entry
// b0 to b1, CO_WG channels from co0; its input window starts at position
// x_first of entry b0 (FX = 4: the even one at or before the first output)
// and spans `span` positions, crossing entry boundaries.
struct C1Block {
    int co0, m0, m_end, b0, b1, x_first, span, df, wch, w_lds;
};

__host__ __device__ inline C1Block c1_block(const C1Tile& T, const C1Args& a, int bid)
{
    C1Block g;
    g.df = T.DF > 0 ? T.DF : a.df;
    const int Do = a.Do, D = a.D, P = T.pos();
    // XCD-aware renumbering: consecutive tiles (which share input) go to the
    // same XCD and its L2.
    const int per = a.n_blk >> 3, rem = a.n_blk & 7;
    const int xcd = bid & 7, slot = bid >> 3;
    const int tile = xcd < rem ? xcd * (per + 1) + slot
                               : rem * (per + 1) + (xcd - rem) * per + slot;
    const int pos_blk = c1_udiv(tile, a.n_co_blk);
    const int co_blk = tile - pos_blk * a.n_co_blk;
    g.m0 = pos_blk * P;
    g.m_end = g.m0 + P < a.M ? g.m0 + P : a.M;
    g.co0 = co_blk * T.co_wg();
    g.b0 = c1_udiv(g.m0, Do);
    g.x_first = T.FX == 4 ? (g.m0 - g.b0 * Do) & ~1 : g.m0 - g.b0 * Do;
    g.b1 = c1_udiv(g.m_end - 1, Do);
    // window length in positions: (b1 - b0) D + x_last + d_filter - x_first
    g.span = (g.b1 - g.b0) * D + (g.m_end - 1 - g.b1 * Do) + g.df - g.x_first;
    g.wch = T.co_wg() * g.df * 2;  // floats per channel of filters
    g.w_lds = a.ccp * a.span2;     // filters' float offset in a stage buffer
    return g;
}

// Stage buffer (floats): ccp channel windows [ccp][span2], then ccp channels
// of filters [ccp][co][tap][2].  Input slot t of lane tid covers window floats
// FX * (t * NT + tid) onwards (FX = 4 loads two positions at once when
// d_image is even, span2 then a multiple of 4; FX = 1 one float).  Returns the
// byte offset of its source from the stage's input base.
__host__ __device__ inline uint32_t c1_xoffb(const C1Tile& T, const C1Args& a, const C1Block& g,
                                             int f)
{
    const int NB = 2, D = a.D;
    const int c_l = c1_udiv(f, a.span2);
    const int r = f - c_l * a.span2;
    if (T.FX == 4) {
        // an even position; past the window (unused) the last even one,
        // whose pair is still inside its batch entry (d_image even)
        const int lim = (g.span - 1) & ~1;
        const int v = g.x_first + (r / NB < lim ? r / NB : lim);
        const int bb = c1_udiv(v, D);
        return 4u * (uint32_t)((bb * a.C_in + c_l) * D * NB + (v - bb * D) * NB);
    }
    const int v = g.x_first + (r / NB < g.span - 1 ? r / NB : g.span - 1);  // past the window: unused
    const int bb = c1_udiv(v, D);
    return 4u * (uint32_t)((bb * a.C_in + c_l) * D * NB + (v - bb * D) * NB + (r % NB));
}

// Filter slot: floats FW * (t * NT + tid) onwards of the stage's filters.
// FW = 4 (16-byte loads, C_out even): rows past C_out are not loaded
// (C1_NOLOAD): their stale LDS values only reach accumulator rows of channels
// that are never stored.  FW = 1: channels past C_out read the last channel.
// Returns the byte offset of its source from the stage's filter base.
__host__ __device__ inline uint32_t c1_woffb(const C1Tile& T, const C1Args& a, const C1Block& g,
                                             int e)
{
    const int NB = 2, df = g.df;
    const int c_l = c1_udiv(e, g.wch);
    const int e2 = e - c_l * g.wch;
    if (T.FW == 4) {
        const int nco = T.co_wg() < a.C_out - g.co0 ? T.co_wg() : a.C_out - g.co0;
        return e2 < nco * df * NB ? 4u * (uint32_t)(c_l * a.C_out * df * NB + e2) : C1_NOLOAD;
    }
    const int co_l = c1_udiv(e2, df * NB);
    const int r = e2 - co_l * (df * NB);
    const int co = g.co0 + co_l < a.C_out - 1 ? g.co0 + co_l : a.C_out - 1;  // past C_out: unused
    return 4u * (uint32_t)(c_l * a.C_out * df * NB + (co - g.co0) * df * NB + r);
}

// Channels of stage s: [s * cc, s * cc + n_valid).
__host__ __device__ inline int c1_stage_channels(const C1Args& a, int s)
{
    return a.cc < a.C_in - s * a.cc ? a.cc : a.C_in - s * a.cc;
}

// Float offsets from a.x / a.w of the block's input and filter bases, and of
// stage s's bases from them.
__host__ __device__ inline int64_t c1_x_base(const C1Args& a, const C1Block& g)
{
    return (int64_t)g.b0 * a.C_in * a.D * 2;
}
__host__ __device__ inline int64_t c1_w_base(const C1Block& g) { return (int64_t)g.co0 * g.df * 2; }
__host__ __device__ inline int64_t c1_stage_x(const C1Args& a, int s)
{
    return (int64_t)s * a.cc * a.D * 2;
}
__host__ __device__ inline int64_t c1_stage_w(const C1Args& a, const C1Block& g, int s)
{
    return (int64_t)s * a.cc * a.C_out * g.df * 2;
}

// Whether input slot float f / filter slot float e is loaded in a stage of nv
// channels.
__host__ __device__ inline bool c1_x_loads(const C1Args& a, int f, int nv)
{
    return f < nv * a.span2;
}
__host__ __device__ inline bool c1_w_loads(const C1Tile& T, const C1Block& g, int e,
                                           uint32_t woffb, int nv)
{
    return e < nv * g.wch && (T.FW == 1 || woffb != C1_NOLOAD);
}

// LDS float offsets where wave `wave` lands input / filter slot t of buffer
// buf: a direct load of FX (FW) floats puts lane i FX i (FW i) floats further.
__host__ __device__ inline int c1_lds_x(const C1Tile& T, const C1Args& a, int buf, int t, int wave)
{
    return buf * a.stage_floats + wave * 64 * T.FX + t * T.nt() * T.FX;
}
__host__ __device__ inline int c1_lds_w(const C1Tile& T, const C1Args& a, const C1Block& g,
                                        int buf, int t, int wave)
{
    return buf * a.stage_floats + g.w_lds + wave * 64 * T.FW + t * T.nt() * T.FW;
}

// Per-lane fragment constants.  A (16 x 4): row mrow = (output channel
// co_a = mrow / 2, blade i_a = mrow % 2), column kk = (channel c_sub of the
// pair, input blade j); B (4 x 16): the same (c_sub, j) by output position
// column mrow.
struct C1Lane {
    int lane, wk, wrest, wco, wpos, mrow, kk, c_sub, j;
};

__host__ __device__ inline C1Lane c1_lane(const C1Tile& T, int tid)
{
    C1Lane l;
    l.lane = tid & 63;
    const int wave = tid >> 6;
    l.wk = wave / (T.WCO * T.WPOS);
    l.wrest = wave - l.wk * (T.WCO * T.WPOS);
    l.wco = l.wrest % T.WCO;
    l.wpos = l.wrest / T.WCO;
    l.mrow = l.lane & 15;
    l.kk = l.lane >> 4;
    l.c_sub = l.kk >> 1;
    l.j = l.kk & 1;
    return l;
}

// A fragment: buffer float offset of the lane's raw filter blade; per step
// add the pair's first channel c_l times wch (c1_a_pair) and c1_a_step.
__host__ __device__ inline int c1_a_ofs(const C1Tile& T, const C1Block& g, const C1Lane& l)
{
    const int co_a = l.mrow >> 1, i_a = l.mrow & 1;
    return g.w_lds + l.c_sub * g.wch + (l.wco * T.MW * 8 + co_a) * g.df * 2 +
           src_blade(2, i_a, l.j);
}
__host__ __device__ inline float c1_a_sign(const C1Args& a, const C1Lane& l)
{
    return sign_of(a.sign, (l.mrow & 1) * 2 + l.j);
}
__host__ __device__ inline int c1_a_pair(const C1Block& g, int c_l) { return c_l * g.wch; }
__host__ __device__ inline int c1_a_step(const C1Block& g, int wofs, int mw, int tap)
{
    return wofs + mw * 8 * g.df * 2 + tap * 2;
}

// B fragment: buffer float offset of the lane's input blade at output column
// nw (tail lanes read a valid position; their outputs are never stored); per
// step add c1_b_pair and 2 tap.
__host__ __device__ inline int c1_b_ofs(const C1Tile& T, const C1Args& a, const C1Block& g,
                                        const C1Lane& l, int nw)
{
    const int Do = a.Do;
    int m = g.m0 + (l.wpos * T.NW + nw) * 16 + l.mrow;
    m = m < g.m_end - 1 ? m : g.m_end - 1;
    const int bb = c1_udiv(m, Do);
    return l.c_sub * a.span2 + ((bb - g.b0) * a.D + (m - bb * Do) - g.x_first) * 2 + l.j;
}
__host__ __device__ inline int c1_b_pair(const C1Args& a, int c_l) { return c_l * a.span2; }

// K split: float4 index in LDS of K slice wk's partial sums of tile (mw, nw).
__host__ __device__ inline int c1_red_f4(const C1Tile& T, int wk, int wrest, int mw, int nw,
                                         int lane)
{
    return ((wk - 1) * (T.WCO * T.WPOS * T.MW * T.NW) + (wrest * T.MW + mw) * T.NW + nw) * 64 +
           lane;
}

// Epilogue: lane row 4 kk + r of a tile is channel 2 kk + r / 2, blade r % 2;
// each lane stores two blades (8 bytes) per channel half.
__host__ __device__ inline int c1_out_pos(const C1Tile& T, const C1Block& g, const C1Lane& l,
                                          int nw)
{
    return g.m0 + (l.wpos * T.NW + nw) * 16 + l.mrow;
}
__host__ __device__ inline int c1_out_channel(const C1Tile& T, const C1Block& g, const C1Lane& l,
                                              int mw, int half)
{
    return g.co0 + (l.wco * T.MW + mw) * 8 + 2 * l.kk + half;
}
// float offset of (position m, channel co)'s two blades: the position part
// (c1_out_base) plus co d_out 2
__host__ __device__ inline int64_t c1_out_base(const C1Args& a, int m)
{
    const int bb = c1_udiv(m, a.Do);
    return ((int64_t)bb * a.C_out * a.Do + (m - bb * a.Do)) * 2;
}
__host__ __device__ inline int64_t c1_out_chan(const C1Args& a, int co)
{
    return (int64_t)co * a.Do * 2;
}

}  // namespace cliff
